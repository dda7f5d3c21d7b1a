// Device side of the CGTP: one work-group computes one (j1, j2) block for a
// tile of pairs, i.e. one irrep-signal tensor product (Section 4.3) on the
// block's own sphere grid, entirely in LDS and registers:
//
//   per pass over a chunk of northern rings
//     1. lift (Definition 4.1 with s = 0 and s = 1, l = j): latitude stage
//        a_c[m] = coefficient * P^m_j(x_i), packed two real series per complex
//        transform;
//     2. longitude synthesis: inverse FFT in LDS (Stockham, radix 4/2/3);
//     3. pointwise products (Section 4.3 / 5.1): scalar-scalar and the
//        1 (x) 1 -> 1 Clebsch-Gordan coupling of the two toroidal fields, i.e.
//        the cross product;
//     4. longitude analysis: forward FFT in LDS, two real spectra per transform;
//     5. Legendre projection onto the block's rows l3 = d, d+2, ..., J, folding
//        the southern rings by parity, accumulated in LDS;
//   then recombination of the vector components with C^{j3 m3}_{j3-1, m3-q, 1, q},
//   scaling by 1/K (Theorem 4.2), and one contiguous store of the block.
//
// All quantities use the complex spherical basis with Condon-Shortley phase.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "cgtp_internal.h"

namespace cgtp {
namespace {

template <typename T> struct Cplx;
template <> struct Cplx<float> { using type = float2; };
template <> struct Cplx<double> { using type = double2; };

template <typename C> __device__ __forceinline__ C cmul(C a, C b) {
    C r;
    r.x = a.x * b.x - a.y * b.y;
    r.y = a.x * b.y + a.y * b.x;
    return r;
}
template <typename C> __device__ __forceinline__ C cadd(C a, C b) { C r; r.x = a.x + b.x; r.y = a.y + b.y; return r; }
template <typename C> __device__ __forceinline__ C csub(C a, C b) { C r; r.x = a.x - b.x; r.y = a.y - b.y; return r; }
template <typename C, typename T> __device__ __forceinline__ C cscale(C a, T s) { C r; r.x = a.x * s; r.y = a.y * s; return r; }
template <typename C> __device__ __forceinline__ C mul_i(C a, bool inv) {
    // multiply by -i (forward) or +i (inverse)
    C r;
    if (inv) { r.x = -a.y; r.y = a.x; } else { r.x = a.y; r.y = -a.x; }
    return r;
}

// In-place-free radix-R DFT of v[0..R-1]; forward uses exp(-2 pi i / R).
template <typename T, typename C>
__device__ __forceinline__ void butterfly(C* v, int R, bool inv) {
    if (R == 2) {
        C a = v[0], b = v[1];
        v[0] = cadd(a, b);
        v[1] = csub(a, b);
    } else if (R == 4) {
        C a = v[0], b = v[1], c = v[2], d = v[3];
        C s0 = cadd(a, c), s1 = csub(a, c), s2 = cadd(b, d), s3 = mul_i(csub(b, d), inv);
        v[0] = cadd(s0, s2);
        v[2] = csub(s0, s2);
        v[1] = cadd(s1, s3);
        v[3] = csub(s1, s3);
    } else if (R == 3) {
        const T h = (T)0.86602540378443864676;  // sqrt(3)/2
        C a = v[0], b = v[1], c = v[2];
        C t1 = cadd(b, c), t2 = csub(b, c);
        C m = csub(a, cscale(t1, (T)0.5));
        // forward: w = -1/2 - i h;  y1 = m - i h t2, y2 = m + i h t2
        C r = mul_i(cscale(t2, h), inv);   // -i h t2 (forward) / +i h t2 (inverse)
        v[0] = cadd(a, t1);
        v[1] = cadd(m, r);
        v[2] = csub(m, r);
    }
}

// Batched Stockham FFT over nb transforms of length Phi stored back to back.
// Reads src, ping-pongs with dst, returns the buffer holding the result.
template <typename T, typename C>
__device__ C* fft_batch(C* src, C* dst, int nb, int Phi, const int* rad, int nrad, const C* tw, bool inv) {
    int Ns = 1;
    for (int s = 0; s < nrad; ++s) {
        const int R = rad[s];
        const int nbf = Phi / R;
        const int total = nb * nbf;
        const int step = Phi / (Ns * R);
        for (int w = threadIdx.x; w < total; w += blockDim.x) {
            const int f = w / nbf, j = w - f * nbf;
            const int k = j % Ns;
            const C* in = src + f * Phi;
            C* out = dst + f * Phi;
            C v[4];
            for (int t = 0; t < R; ++t) v[t] = in[j + t * nbf];
            for (int t = 1; t < R; ++t) {
                C wv = tw[t * k * step];
                if (inv) wv.y = -wv.y;
                v[t] = cmul(v[t], wv);
            }
            butterfly<T, C>(v, R, inv);
            const int base = (j / Ns) * Ns * R + k;
            for (int t = 0; t < R; ++t) out[base + t * Ns] = v[t];
        }
        __syncthreads();
        C* tmp = src; src = dst; dst = tmp;
        Ns *= R;
    }
    return src;
}

// Row index n of a flat accumulator entry e, rows l3 = d + 2n of 2 l3 + 1 entries.
__device__ __forceinline__ int acc_row(int e, int d) {
    // rowoff(n) = 2 n^2 + (2d - 1) n ; largest n with rowoff(n) <= e
    const float b = 2.0f * d - 1.0f;
    int n = (int)((-b + sqrtf(b * b + 8.0f * (float)e)) * 0.25f);
    if (n < 0) n = 0;
    while (2 * n * n + (2 * d - 1) * n > e) --n;
    while (2 * (n + 1) * (n + 1) + (2 * d - 1) * (n + 1) <= e) ++n;
    return n;
}
__device__ __forceinline__ int acc_rowoff(int n, int d) { return 2 * n * n + (2 * d - 1) * n; }

template <typename T>
__global__ __launch_bounds__(kThreads) void block_kernel(Tables<T> tb, const int32_t* __restrict__ list,
                                                         LaunchMap map, const T* __restrict__ x1,
                                                         const T* __restrict__ x2, T* __restrict__ out, int64_t N,
                                                         int L) {
    using C = typename Cplx<T>::type;
    extern __shared__ __align__(16) unsigned char smem[];

    const int64_t wg = blockIdx.x;
    int cls = 0;
    while (cls + 1 < map.ncls && wg >= map.cum[cls + 1]) ++cls;
    const int pairs = map.pairs[cls];
    const int64_t ntiles = map.ntiles[cls];
    const int64_t local = wg - map.cum[cls];
    const int bi = (int)(local / ntiles);
    const int64_t tile = local - (int64_t)bi * ntiles;
    const BlockDesc bd = tb.blocks[list[map.list_off[cls] + bi]];
    const int j1 = bd.j1, j2 = bd.j2, J = bd.J, d = bd.d, R = bd.R, Phi = bd.Phi;
    const bool cross = bd.kind == kBlockCross;
    // synthesis transforms per (ring, pair).  Two real series share a complex
    // transform only when they come from the same input, so rounding crosstalk
    // stays proportional to that input's norm (the product is bilinear).
    const int nslot = cross ? 4 : 2;
    const int nz = cross ? 2 : 1;      // analysis transforms per (ring, pair)
    const int ncomp = cross ? 4 : 1;   // projected components
    const int n1 = 2 * j1 + 1, n2 = 2 * j2 + 1;
    const int nrows = (J - d) / 2 + 1;
    const int nel = nrows * (2 * d + 1) + 2 * nrows * (nrows - 1);
    const int64_t p0 = tile * pairs;
    const int np = (int)((N - p0) < pairs ? (N - p0) : pairs);
    const int nin = (L + 1) * (L + 1);
    const int64_t nout = (int64_t)nin * nin;

    T* xs1 = reinterpret_cast<T*>(smem);
    T* xs2 = xs1 + pairs * n1;
    T* acc = xs2 + pairs * n2;
    size_t head = sizeof(T) * ((size_t)pairs * (n1 + n2) + (size_t)pairs * ncomp * nel);
    head = (head + 15) & ~(size_t)15;
    C* bufA = reinterpret_cast<C*>(smem + head);
    C* bufB = bufA + (size_t)bd.chunk * pairs * nslot * Phi;

    int rad[kMaxRadix];
    for (int s = 0; s < kMaxRadix; ++s) rad[s] = bd.rad[s];
    const C* tw = reinterpret_cast<const C*>(tb.tw) + bd.tw_off;
    const T* pbar = tb.pbar + bd.pbar_off;
    const T* wt = tb.wt + bd.wt_off;
    const T* lcg1 = tb.lcg + 3 * j1 * j1;
    const T* lcg2 = tb.lcg + 3 * j2 * j2;

    // ---- inputs of the tile (rows past N read as zero)
    for (int e = threadIdx.x; e < pairs * n1; e += blockDim.x) {
        const int p = e / n1, m = e - p * n1;
        xs1[e] = p < np ? x1[(p0 + p) * nin + j1 * j1 + m] : (T)0;
    }
    for (int e = threadIdx.x; e < pairs * n2; e += blockDim.x) {
        const int p = e / n2, m = e - p * n2;
        xs2[e] = p < np ? x2[(p0 + p) * nin + j2 * j2 + m] : (T)0;
    }
    for (int e = threadIdx.x; e < pairs * ncomp * nel; e += blockDim.x) acc[e] = (T)0;
    __syncthreads();

    const T twopi_over_phi = (T)(6.283185307179586476925286766559 / (double)Phi);
    T ccg[9];
    for (int i = 0; i < 9; ++i) ccg[i] = tb.ccg[i];

    for (int r0 = 0; r0 < R; r0 += bd.chunk) {
        const int nr = (R - r0) < bd.chunk ? (R - r0) : bd.chunk;
        // ---- 1. lift, latitude stage: fill the packed synthesis inputs
        const int nsyn = nr * pairs * nslot;
        for (int e = threadIdx.x; e < nsyn * Phi; e += blockDim.x) {
            const int k = e % Phi;
            const int f = e / Phi;
            const int slot = f % nslot;
            const int rp = f / nslot;
            const int p = rp % pairs;
            const int ring = r0 + rp / pairs;
            const T* prow = pbar + (size_t)ring * bd.pbar_stride;
            T re = 0, im = 0;
            if (!cross) {
                // slot 0: scalar lift of x1, slot 1: scalar lift of x2 (real coefficients)
                const int j = slot == 0 ? j1 : j2;
                const T* xs = slot == 0 ? xs1 + p * n1 : xs2 + p * n2;
                const int m = k <= j ? k : (k >= Phi - j ? k - Phi : 1 << 20);
                if (m != (1 << 20)) {
                    const int am = m < 0 ? -m : m;
                    T pv = prow[j * (j + 1) / 2 + am];
                    if (m < 0 && (am & 1)) pv = -pv;
                    re = xs[m + j] * pv;
                }
            } else {
                const int j = slot < 2 ? j1 : j2;
                const T* xs = slot < 2 ? xs1 + p * n1 : xs2 + p * n2;
                const T* lc = slot < 2 ? lcg1 : lcg2;
                const int m = k <= j ? k : (k >= Phi - j ? k - Phi : 1 << 20);
                if (m != (1 << 20)) {
                    const int am = m < 0 ? -m : m;
                    T pv = prow[j * (j + 1) / 2 + am];
                    if (m < 0 && (am & 1)) pv = -pv;
                    const int nj = 2 * j + 1;
                    // component c of the lift at order m (orbital order m for vectors)
                    auto comp = [&](int q) -> T {   // q = 2: scalar
                        if (q == 2) return xs[m + j] * pv;
                        const int mj = m + q;
                        if (mj < -j || mj > j) return (T)0;
                        return lc[(q + 1) * nj + m + j] * xs[mj + j] * pv;
                    };
                    if ((slot & 1) == 0) { re = comp(2); im = comp(0); }
                    else { re = comp(-1); im = comp(1); }
                }
            }
            C v;
            v.x = re;
            v.y = im;
            bufA[(size_t)f * Phi + k] = v;
        }
        __syncthreads();
        // ---- 2. longitude synthesis (exp(+i m phi))
        C* syn = fft_batch<T, C>(bufA, bufB, nsyn, Phi, rad, bd.nrad, tw, true);
        C* zb = syn == bufA ? bufB : bufA;
        // ---- 3. pointwise products on the full circle
        const int nrp = nr * pairs;
        for (int e = threadIdx.x; e < nrp * Phi; e += blockDim.x) {
            const int k = e % Phi;
            const int rp = e / Phi;
            const int kk = k == 0 ? 0 : Phi - k;
            if (!cross) {
                // each slot already holds one Hermitian signal
                zb[(size_t)rp * Phi + k] = cmul(syn[((size_t)rp * 2) * Phi + k], syn[((size_t)rp * 2 + 1) * Phi + k]);
            } else {
                C f[8];   // f1 s, f1 q0, f1 q-1, f1 q+1, f2 s, f2 q0, f2 q-1, f2 q+1
                for (int s = 0; s < 4; ++s) {
                    const C F = syn[((size_t)rp * 4 + s) * Phi + k], Fr = syn[((size_t)rp * 4 + s) * Phi + kk];
                    f[2 * s].x = (F.x + Fr.x) * (T)0.5; f[2 * s].y = (F.y - Fr.y) * (T)0.5;
                    f[2 * s + 1].x = (F.y + Fr.y) * (T)0.5; f[2 * s + 1].y = (Fr.x - F.x) * (T)0.5;
                }
                const C a_s = f[0], a0 = f[1], am = f[2], ap = f[3];
                const C b_s = f[4], b0 = f[5], bm = f[6], bp = f[7];
                // ccg[(q1+1)*3 + q2+1] = C^{1, q1+q2}_{1 q1 1 q2}
                const C gs = cmul(a_s, b_s);
                const C gp = cadd(cscale(cmul(ap, b0), ccg[2 * 3 + 1]), cscale(cmul(a0, bp), ccg[1 * 3 + 2]));
                const C g0 = cadd(cadd(cscale(cmul(ap, bm), ccg[2 * 3 + 0]), cscale(cmul(a0, b0), ccg[1 * 3 + 1])),
                                  cscale(cmul(am, bp), ccg[0 * 3 + 2]));
                const C gm = cadd(cscale(cmul(a0, bm), ccg[1 * 3 + 0]), cscale(cmul(am, b0), ccg[0 * 3 + 1]));
                C z1, z2;   // z1 = gs + i g0, z2 = g-1 + i g+1
                z1.x = gs.x - g0.y; z1.y = gs.y + g0.x;
                z2.x = gm.x - gp.y; z2.y = gm.y + gp.x;
                zb[((size_t)rp * 2 + 0) * Phi + k] = z1;
                zb[((size_t)rp * 2 + 1) * Phi + k] = z2;
            }
        }
        __syncthreads();
        // ---- 4. longitude analysis (exp(-i m phi)); real spectra in re / im
        C* spec = fft_batch<T, C>(zb, syn, nrp * nz, Phi, rad, bd.nrad, tw, false);
        // ---- 5. Legendre projection of the chunk's rings, accumulated
        for (int e = threadIdx.x; e < pairs * ncomp * nel; e += blockDim.x) {
            const int el = e % nel;
            const int pc = e / nel;
            const int c = pc % ncomp;
            const int p = pc / ncomp;
            const int n = acc_row(el, d);
            const int l3 = d + 2 * n;
            const int m = el - acc_rowoff(n, d) - l3;
            const int am = m < 0 ? -m : m;
            const T sg = (m < 0 && (am & 1)) ? (T)-1 : (T)1;
            const int km = m < 0 ? m + Phi : m;
            const int lidx = l3 * (l3 + 1) / 2 + am;
            T s = 0;
            for (int r = 0; r < nr; ++r) {
                const int ring = r0 + r;
                const C G = spec[((size_t)(r * pairs + p) * nz + (c >> 1)) * Phi + km];
                const T g = (c & 1) ? G.y : G.x;
                s += wt[ring] * pbar[(size_t)ring * bd.pbar_stride + lidx] * g;
            }
            acc[e] += s * sg * twopi_over_phi;
        }
        __syncthreads();
    }

    // ---- recombination, 1/K, contiguous store of the block
    const int nblk = n1 * n2;
    const T* kinv = tb.kinv + bd.kinv_off;
    for (int e = threadIdx.x; e < np * nblk; e += blockDim.x) {
        const int p = e / nblk;
        const int o = e - p * nblk;
        int j3 = (int)sqrtf((float)(o + d * d));
        while (j3 * j3 - d * d > o) --j3;
        while ((j3 + 1) * (j3 + 1) - d * d <= o) ++j3;
        const int m3 = o - (j3 * j3 - d * d) - j3;
        T z;
        if (((J + j3) & 1) == 0) {
            z = acc[(p * ncomp + 0) * nel + acc_rowoff((j3 - d) / 2, d) + j3 + m3];
        } else {
            const int l3 = j3 - 1;
            const int rowoff = acc_rowoff((l3 - d) / 2, d);
            const T* rc = tb.rcg + 3 * j3 * j3;
            z = 0;
            // component slots: 1 -> q = 0, 2 -> q = -1, 3 -> q = +1
            const int slot_of_q[3] = {2, 1, 3};
            for (int q = -1; q <= 1; ++q) {
                const int m = m3 - q;
                if (m < -l3 || m > l3) continue;
                z += rc[(q + 1) * (2 * j3 + 1) + m3 + j3] *
                     acc[(p * ncomp + slot_of_q[q + 1]) * nel + rowoff + l3 + m];
            }
        }
        out[(p0 + p) * nout + bd.out_off + o] = z * kinv[j3 - d];
    }
}

template <typename T>
int launch(const Tables<T>& tb, const int32_t* list, const LaunchMap& map, int lds, const T* x1, const T* x2,
           T* out, int64_t N, int L, void* stream) {
    const int64_t grid = map.cum[map.ncls];
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(block_kernel<T>, dim3((unsigned)grid), dim3(kThreads), lds, (hipStream_t)stream, tb, list,
                       map, x1, x2, out, N, L);
    return (int)hipGetLastError();
}

}  // namespace

int launch_blocks_f32(const Tables<float>& tb, const int32_t* list, const LaunchMap& map, int lds, const float* x1,
                      const float* x2, float* out, int64_t N, int L, void* stream) {
    return launch<float>(tb, list, map, lds, x1, x2, out, N, L, stream);
}
int launch_blocks_f64(const Tables<double>& tb, const int32_t* list, const LaunchMap& map, int lds, const double* x1,
                      const double* x2, double* out, int64_t N, int L, void* stream) {
    return launch<double>(tb, list, map, lds, x1, x2, out, N, L, stream);
}

}  // namespace cgtp

// Device side of the multiple-input, multiple-output irrep-signal tensor
// products (the (0,0,0) Gaunt product and the (1,1,1) vector product,
// Section 4.3, Appendix D).  One work-group takes a tile of pairs through the
// whole product, in LDS and registers only.
//
// Per pair tile:
//   0. the input rows become scalar-harmonic coefficients of each spin
//      component (Definition 4.1: a[q][l][ml] = sum_j C^{j,ml+q}_{l,ml,1,q}
//      x^(j,l)_{ml+q}), stored as the B operand of the lift;
// then for each group of G north/south ring pairs:
//   1. lift on MFMA: per order am, a [16 rows (ring, parity of l - am)] x
//      [K = l] x [16 columns (sign of m, input, component, pair)] product with
//      P_l^am(x_ring) as the A operand; even and odd parts give the north and
//      south rings (P_l^m(-x) = (-1)^(l+m) P_l^m(x)), stored as one complex
//      transform input (north + i south) in the first pass's layout;
//   2. longitude synthesis, two in-register passes, in place;
//   3. pointwise products on half the circle: the north and south signals are
//      unpacked from each transform, multiplied (scalar product, or the
//      1 (x) 1 -> 1 coupling), and packed back as (north + i south);
//   4. longitude analysis, two passes;
//   5. Legendre projection on MFMA: per order am and parity, [rows l3] x
//      [4 rings] x [sign, component, pair], with w_ring P_l3^am(x_ring) as the
//      A operand and north +- south of each spectrum as the B operand,
//      accumulated in registers over all ring groups.
// Then the accumulators go to LDS, each output is recombined from up to three
// spectra (C^{j3,m3}_{l3,m3-q,1,q} for the vector product, with the
// longitude quadrature, unpacking and coupling constants and the sign of
// negative orders folded into the plan's weights), and stored contiguously.
//
// All quantities use the complex spherical basis with Condon-Shortley phase.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "istp_internal.h"

// This file builds the plain kernels (istp_kernel); with ISTP_CHANNEL_KERNELS
// set to 1 it builds the channel-wise, label-weighted forward kernels instead
// (istp_kernel_channels, istp_kernels_channels.hip), so that the plain ones
// carry none of the channel bookkeeping.
#ifndef ISTP_CHANNEL_KERNELS
#define ISTP_CHANNEL_KERNELS 0
#endif
// With ISTP_TENSOR_KERNELS set to 1 the same two kinds are built for spin 2
// only (istp_kernels_tensor.hip, istp_kernels_channels_tensor.hip): a
// translation unit of its own compiles in parallel with the others.
#ifndef ISTP_TENSOR_KERNELS
#define ISTP_TENSOR_KERNELS 0
#endif
// With ISTP_REAL_KERNELS set to 1 the Gaunt product for rows in the real
// spherical-harmonic basis is built (istp_kernels_real.hip): istp_kernel_real.
// Hermitian coefficients c_{l,-m} = (-1)^m conj(c_lm) make every ring's signal
// real, so north and south still share one transform; the lift operand holds
// Re c and Im c at +|m| (in place of the +|m| and -|m| columns), a lane and
// its partner column form the transforms' inputs at +|m| and -|m|, the
// products are taken on the whole circle (north = Re, south = Im), and the
// projection forms Re and Im of each order's spectrum from the analysis at
// +|m| and -|m|.  For |m| > 0 the part is the lowest bit of a lift column, so
// that a column's partner is the neighbouring lane of the same tile.
#ifndef ISTP_REAL_KERNELS
#define ISTP_REAL_KERNELS 0
#endif

namespace istp {
namespace {

using namespace ::cgtp::dev;

constexpr double kRsqrt2 = 0.70710678118654752440084436210485;

// Lift rows: MFMA row i carries ring ring(i) and the parity par(i) of l - am,
// chosen so that a lane's four accumulator elements hold (even, odd) for two
// rings (f32 rows are 4 (lane / 16) + v, f64 rows lane / 16 + 4 v).
template <typename T> __device__ __forceinline__ void lift_row(int i, int& ring, int& par);
template <> __device__ __forceinline__ void lift_row<float>(int i, int& ring, int& par) {
    ring = i >> 1;
    par = i & 1;
}
template <> __device__ __forceinline__ void lift_row<double>(int i, int& ring, int& par) {
    ring = (i & 3) + 4 * (i >> 3);
    par = (i >> 2) & 1;
}
// ring of accumulator elements 2 h (even) and 2 h + 1 (odd) of quarter q
template <typename T> __device__ __forceinline__ int lift_ring(int q, int h);
template <> __device__ __forceinline__ int lift_ring<float>(int q, int h) { return 2 * q + h; }
template <> __device__ __forceinline__ int lift_ring<double>(int q, int h) { return q + 4 * h; }

// Time reversal of a row: value c of the reversed row is (-1)^(m+j-l+S) times
// value src of the row, for the label (j, l) and order m that c holds.
template <int S>
__device__ __forceinline__ void reverse_index(int c, int* src, bool* neg) {
    if constexpr (S == 2) {   // label (j, l), j = |l - 2| .. l + 2, starts at 5 l^2 + j^2 - (l - 2)^2
        int l = (int)sqrtf((float)c / 5.0f);
        while (5 * (l + 1) * (l + 1) <= c) ++l;
        while (5 * l * l > c) --l;
        const int r = c - 5 * l * l, jmin = l >= 2 ? l - 2 : 2 - l;
        int j = jmin;
        while (j < l + 2 && (j + 1) * (j + 1) - jmin * jmin <= r) ++j;
        const int lo = j * j - jmin * jmin, m = r - lo - j;
        *src = 5 * l * l + lo + j - m;
        *neg = (m + j - l) & 1;
        return;
    }
    if (S == 0) {   // c = l^2 + l + m
        int l = (int)sqrtf((float)c);
        while ((l + 1) * (l + 1) <= c) ++l;
        while (l * l > c) --l;
        const int m = c - l * l - l;
        *src = l * l + l - m;
        *neg = m & 1;
    } else {        // label (j, l) of c starts at 3 l^2 + {0, 2l - 1, 4l}[j - l + 1]
        int l = (int)sqrtf((float)c / 3.0f);
        while (3 * (l + 1) * (l + 1) <= c) ++l;
        while (3 * l * l > c) --l;
        const int r = c - 3 * l * l;
        const int jj = r < 2 * l - 1 ? 0 : (r < 4 * l ? 1 : 2);
        const int lo = jj == 0 ? 0 : (jj == 1 ? 2 * l - 1 : 4 * l);
        const int j = l - 1 + jj, m = r - lo - j;
        *src = 3 * l * l + lo + j - m;
        *neg = (m + jj) & 1;
    }
}

// Step 0: the B operand of the lift for one pair tile (zero for pairs past N,
// rows past an input's degree bound and padding columns).  The tile's input
// rows and the lift couplings are first staged in LDS with one batch of loads
// per thread; then every entry is formed from LDS, per operand column (the
// plan's column table gives its order and offset; padding columns are zero).
// Column order: sign of m (+ first), input, component, pair; negative orders
// carry (-1)^am (P^{-m} = (-1)^m P^m).  With kReverseSecond the second input
// is staged time-reversed, x[(j,l), m] -> (-1)^(m+j-l+S) x[(j,l), -m].
// Channel bookkeeping of a work-group: its first row is channel c0 of pair n0.
struct ChanPos {
    int64_t n0;
    int c0;
};

template <typename T, int S, bool CH, bool RL>
__device__ __forceinline__ void build_coefficients(const IstpTables<T>& tb, const IstpDesc& d, int64_t p0, int np,
                                                   const T* __restrict__ x1, const T* __restrict__ x2, T* acoef,
                                                   T* stage, const IstpChan<T>& ch, ChanPos cp) {
    constexpr int NC = 2 * S + 1;
    const int P = d.pairs, nin = d.nin, nin2 = d.nin2;
    const int Lm = d.L > d.L2 ? d.L : d.L2;
    const int nx1 = P * nin, nx = nx1 + P * nin2, nxa = istp_stage_x(P, nin, nin2);
    const int ncg = S ? NC * NC * (Lm + 1) * (Lm + 1) : 0;
    const bool rev2 = d.flags & kReverseSecond;
    {
        T v[kStageLoads];
#pragma unroll
        for (int u = 0; u < kStageLoads; ++u) {
            const int e = threadIdx.x + u * kThreads;
            v[u] = (T)0;
            if (e < nx1) {
                const int p = e / nin, c = e - p * nin;
                if (p < np) {
                    T xv = x1[(p0 + p) * (int64_t)nin + c];
                    if constexpr (CH) {
                        if (ch.w1) {
                            const int64_t k = (ch.flags & kChanPerRow) ? p0 + p : (cp.c0 + p) % ch.channels;
                            xv *= ch.w1[k * ch.nl1 + tb.lab[c]];
                        }
                    }
                    v[u] = xv;
                }
            } else if (e < nx) {
                const int p = (e - nx1) / nin2, c = e - nx1 - p * nin2;
                int src = c;
                bool neg = false;
                if (rev2) reverse_index<S>(c, &src, &neg);
                if (p < np) {
                    int64_t r2 = p0 + p;
                    if constexpr (CH) {
                        if (ch.flags & kChanX2Shared) r2 = cp.n0 + (cp.c0 + p) / ch.channels;
                    }
                    T xv = x2[r2 * (int64_t)nin2 + src];
                    if constexpr (CH) {
                        if (ch.w2) {
                            const int64_t k = (ch.flags & kChanPerRow) ? p0 + p : (cp.c0 + p) % ch.channels;
                            xv *= ch.w2[k * ch.nl2 + tb.lab[nin + src]];
                        }
                    }
                    v[u] = neg ? -xv : xv;
                }
            } else if (e - nx < ncg) {
                v[u] = tb.liftcg[e - nx];
            }
        }
#pragma unroll
        for (int u = 0; u < kStageLoads; ++u) {
            const int e = threadIdx.x + u * kThreads;
            if (e < nx) stage[e] = v[u];
            else if (e - nx < ncg) stage[nxa + e - nx] = v[u];
        }
    }
    lds_barrier();
    // per operand column (order am, column col): its k rows, in chunks of 8
    const T* cgs = stage + nxa;
    const int per_sign = 2 * NC * P;
    const int nchunk = (Lm + 8) / 8;
    for (int it = threadIdx.x; it < d.n_bcol * nchunk; it += kThreads) {
        const int ci = it % d.n_bcol, k0 = 8 * (it / d.n_bcol);
        const int2 bc = tb.bcol[ci];
        const int am = bc.x & 255, col = bc.x >> 8;
        const bool two = RL ? (am || S == 1) : am;   // columns of both signs / parts at this order
        const int ncol = (two ? 2 : 1) * per_sign, cs = istp_cstride(ncol);
        const int kp = (Lm - am + 4) / 4 * 4;
        if (k0 >= kp) continue;
        const int k1 = min(k0 + 8, kp);
        T* dst = acoef + bc.y;
        if (col >= ncol) {
            for (int k = k0; k < k1; ++k) dst[k * cs] = (T)0;
            continue;
        }
        // RL, am > 0: the part is the lowest bit of the column (partners are neighbours)
        const int sg = (RL && two) ? (col & 1) : col / per_sign;
        const int rem = (RL && two) ? (col >> 1) : col - sg * per_sign;
        const int in = rem / (NC * P), c = (rem / P) % NC, p = rem % P;
        const int m = sg ? -am : am;
        // RL: column part sg = 0 holds Re c_{l,am}, 1 holds Im c_{l,am}, with
        // c_{l,am} = (-1)^am (r_{l,am} - i r_{l,-am}) / sqrt 2 (am > 0), c_{l,0} = r_{l,0}
        const T sign = RL ? (S == 1 ? (T)1 : (am ? (T)((am & 1) ? -kRsqrt2 : kRsqrt2) * (sg ? (T)-1 : (T)1) : (T)1))
                          : ((sg && (am & 1)) ? (T)-1 : (T)1);
        const int Lin = in ? d.L2 : d.L;
        const T* x = in ? stage + nx1 + p * nin2 : stage + p * nin;
#pragma unroll 4
        for (int k = k0; k < k1; ++k) {
            const int l = am + k;
            T v = (T)0;
            if (l <= Lin) {
                if (S == 0) {
                    v = x[l * l + l + m];   // RL: r_{l,am} (part 0) or r_{l,-am} (part 1)
                } else if constexpr (S == 2) {
                    // labels j = |l - 2| .. l + 2; label (j, l) starts at 5 l^2 + j^2 - (l - 2)^2
                    const int q = c - 2, mj = m + q, jmin = l >= 2 ? l - 2 : 2 - l;
                    const T* cg = cgs + 25 * l * l + m + l;
#pragma unroll
                    for (int jj = 0; jj < 5; ++jj) {
                        const int j = l - 2 + jj;
                        if (j < jmin || mj < -j || mj > j) continue;
                        const int lo = 5 * l * l + j * j - (l - 2) * (l - 2);
                        v += cg[(jj * 5 + c) * (2 * l + 1)] * x[lo + j + mj];
                    }
                } else if (RL) {
                    // spin 1, real-basis rows: Re (sg = 0) or Im (sg = 1) of a_q[l][am] =
                    // sum_j C^{j,am+q}_{l,am,1,q} c^(j,l)_{am+q}; the label's complex
                    // coefficient from its real-basis row, times -i where
                    // sigma = (-1)^(l+1-j) = -1
                    const int q = c - 1, mj = am + q;
                    const T* cg = cgs + 9 * l * l + am + l;
#pragma unroll
                    for (int jj = 0; jj < 3; ++jj) {
                        const int j = l - 1 + jj;
                        if (j < 0 || j + l < 1 || mj < -j || mj > j) continue;
                        const int lo = 3 * l * l + (jj == 0 ? 0 : (jj == 1 ? 2 * l - 1 : 4 * l));
                        const T* r0 = x + lo + j;
                        const int mu = mj < 0 ? -mj : mj;
                        T wr, wi;
                        if (mj == 0) {
                            wr = r0[0];
                            wi = (T)0;
                        } else if (mj > 0) {
                            const T h = (mu & 1) ? (T)-kRsqrt2 : (T)kRsqrt2;
                            wr = h * r0[mu];
                            wi = -h * r0[-mu];
                        } else {
                            wr = (T)kRsqrt2 * r0[mu];
                            wi = (T)kRsqrt2 * r0[-mu];
                        }
                        const bool flip = jj == 1;   // sigma = (-1)^(l+1-j) = -1 for j = l: c = -i w
                        const T cpart = sg ? (flip ? -wr : wi) : (flip ? wi : wr);
                        v += cg[(jj * 3 + c) * (2 * l + 1)] * cpart;
                    }
                } else {
                    const int q = c - 1, mj = m + q;
                    const T* cg = cgs + 9 * l * l + m + l;
#pragma unroll
                    for (int jj = 0; jj < 3; ++jj) {
                        const int j = l - 1 + jj;
                        if (j < 0 || j + l < 1 || mj < -j || mj > j) continue;
                        const int lo = 3 * l * l + (jj == 0 ? 0 : (jj == 1 ? 2 * l - 1 : 4 * l));
                        v += cg[(jj * 3 + c) * (2 * l + 1)] * x[lo + j + mj];
                    }
                }
            }
            dst[k * cs] = sign * v;
        }
    }
}

template <typename T, int A, int B, int S, bool LONG, bool CH, bool RL>
__device__ __forceinline__ void istp_body(const IstpTables<T>& tb, const IstpDesc& d, int64_t p0, int np,
                                          const T* __restrict__ x1, const T* __restrict__ x2, T* __restrict__ out,
                                          const IstpChan<T>& ch, unsigned char* smem) {
    using C2 = typename Cplx<T>::type;
    using Acc = typename Cplx<T>::acc4;
    constexpr int Phi = A * B;
    constexpr int H = Phi / 2 + 1;
    constexpr int BP = B + 1;
    constexpr int FS = A * BP;
    constexpr int NC = 2 * S + 1;   // spin components
    constexpr int NS = 2 * NC;      // synthesis transforms per unit
    constexpr int MT = max_tiles<T>(S);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, kq = lane >> 4;
    const int Lo = d.Lo, R = d.R, G = d.G, P = d.pairs;
    const int Lm = d.L > d.L2 ? d.L : d.L2;   // largest input degree
    const IstpLayout ly =
        istp_layout<T>(A, B, NC, G, P, d.acoef_len, d.hc_len, istp_stage_len(P, d.nin, d.nin2, Lm, S), d.n_proj);
    C2* tw2 = reinterpret_cast<C2*>(smem);
    int* ptab = reinterpret_cast<int*>(smem + ly.ptab);
    T* acoef = reinterpret_cast<T*>(smem + ly.acoef);
    C2* fbuf = reinterpret_cast<C2*>(smem + ly.fbuf);
    T* hc = reinterpret_cast<T*>(smem + ly.hc);
    auto ubuf = [&](int u) -> C2* { return fbuf + (size_t)u * ly.unit; };

    for (int e = tid; e < FS; e += kThreads) tw2[e] = reinterpret_cast<const C2*>(tb.tw)[e];
    for (int e = tid; e < d.n_proj; e += kThreads) {
        const ProjTile pt = tb.proj[e];
        ptab[e] = pt.a | (pt.am << 20) | (pt.par << 27);
    }
    ChanPos cp{p0, 0};
    if constexpr (CH) {
        cp.n0 = p0 / ch.channels;
        cp.c0 = (int)(p0 - cp.n0 * ch.channels);
    }
    build_coefficients<T, S, CH, RL>(tb, d, p0, np, x1, x2, acoef, reinterpret_cast<T*>(fbuf), ch, cp);

    // projection tiles of this wave: w, w + kWaves, ...  A lane's B operand is
    // column li (sign, component, pair; past the last column: column 0, whose
    // duplicate results are discarded) of ring kq of a ring quad; per tile
    // only the order's longitude position changes (order 0 has no negative
    // column: those lanes read position 0).  Each tile's (weight offset |
    // am << 20 | parity << 27) is in ptab.
    const int ntw = d.n_proj > wave ? (d.n_proj - 1 - wave) / kWaves + 1 : 0;
    const int col_l = li < 2 * NC * P ? li : 0;
    const int sg_l = col_l / (NC * P), c_l = (col_l / P) % NC, p_l = col_l % P;
    const int b_lane = ly.fbuf + (int)sizeof(C2) * ((kq * P + p_l) * ly.unit + c_l * FS);
    const int a_lane = (kq * d.wrow + li) * (int)sizeof(T);
    // weight tables as buffer resources: reads past the end return zero
    const __amdgpu_buffer_rsrc_t pw_rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)tb.pw, (short)0, d.pw_len * (int)sizeof(T), kBufferFlags);
    const __amdgpu_buffer_rsrc_t lw_rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)tb.lw, (short)0, d.lw_len * (int)sizeof(T), kBufferFlags);
    Acc acc[MT];
#pragma unroll
    for (int s = 0; s < MT; ++s) acc[s] = Acc(0);
    lds_barrier();

    for (int rg0 = 0; rg0 < R; rg0 += G) {
        // the transform phases take the units of the ring quads the projection
        // reads: whole quads up to the grid's last ring (the group's other units
        // are never read)
        const int Uq = min(G, (R - rg0 + 3) & ~3) * P;
        // ---- 1. lift on MFMA: per tile, K in batches of kMaxLiftSteps steps whose
        // weights are loaded at once
        {
            int ring0, par;
            lift_row<T>(li, ring0, par);
            for (int ti = wave; ti < d.n_lift; ti += kWaves) {
                const LiftTile lt = tb.lift[ti];
                const int ring = 8 * lt.rb + ring0;
                const bool rowok = ring < G && rg0 + ring < R;
                const int voff = ((rg0 + ring) * lt.kp + kq) * (int)sizeof(T);
                const T* bb = acoef + lt.acoef + kq * lt.cstride + li;
                Acc da = Acc(0);
                T a[kMaxLiftSteps];
                if constexpr (!LONG) {
                    // K <= 4 kMaxLiftSteps (every forward product): one batch of weights
#pragma unroll
                    for (int s = 0; s < kMaxLiftSteps; ++s) {
                        const int k = 4 * s + kq;
                        a[s] = (s < lt.steps && rowok && (k & 1) == par)
                                   ? buffer_load<T>(lw_rsrc, voff + 4 * s * (int)sizeof(T), lt.lw * (int)sizeof(T))
                                   : (T)0;
                    }
#pragma unroll
                    for (int s = 0; s < kMaxLiftSteps; ++s)
                        if (s < lt.steps) da = mfma16(a[s], bb[4 * s * lt.cstride], da);
                } else {
                    // the gradient product's degree-2L lift: K in batches
                    for (int s0 = 0; s0 < lt.steps; s0 += kMaxLiftSteps) {
#pragma unroll
                        for (int s = 0; s < kMaxLiftSteps; ++s) {
                            const int k = 4 * (s0 + s) + kq;
                            a[s] = (s0 + s < lt.steps && rowok && (k & 1) == par)
                                       ? buffer_load<T>(lw_rsrc, voff + 4 * (s0 + s) * (int)sizeof(T),
                                                        lt.lw * (int)sizeof(T))
                                       : (T)0;
                        }
#pragma unroll
                        for (int s = 0; s < kMaxLiftSteps; ++s)
                            if (s0 + s < lt.steps) da = mfma16(a[s], bb[4 * (s0 + s) * lt.cstride], da);
                    }
                }
                const int col = 16 * lt.ct + li;
                // RL: the partner column (other part, same input and pair) is lane li ^ 1
                Acc pa = Acc(0);
                if constexpr (RL) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) pa[v] = __shfl_xor(da[v], 1, 64);
                }
                if (col < lt.ncol) {
                    const int per_sign = 2 * NC * P;
                    const bool two = RL && (lt.am || S == 1);   // both parts at this order
                    const int sg = two ? (col & 1) : col / per_sign;
                    const int rem = two ? (col >> 1) : col - sg * per_sign;
                    const int in = rem / (NC * P), c = (rem / P) % NC, p = rem % P;
                    // RL spin 1: f_0 (c = 1) is real per ring and is stored like spin 0;
                    // f_+1 is complex: its north and south take slots 0 and 2 of the
                    // input (c = 2 gives them at +am, c = 0 at -am as f_+1[-m] =
                    // -conj f_-1[m]); at am = 0 only c = 2 and f_0's part Re store
                    int slot = c, n = sg ? Phi - lt.am : lt.am;
                    bool skip = false;
                    if constexpr (RL && S == 1) {
                        if (c == 1) skip = sg && lt.am == 0;
                        else {
                            slot = sg ? 2 : 0;
                            n = c == 2 ? lt.am : Phi - lt.am;
                            skip = c == 0 && lt.am == 0;
                        }
                    }
                    C2* dst = fbuf + (size_t)p * ly.unit + (in * NC + slot) * FS + (n % A) * BP + n / A;
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int r = 8 * lt.rb + lift_ring<T>(kq, h);
                        if (r >= G || skip) continue;
                        const T e = da[2 * h], o = da[2 * h + 1];
                        if constexpr (RL) {
                            const T pe = two ? pa[2 * h] : (T)0, po = two ? pa[2 * h + 1] : (T)0;
                            if (S == 1 && c != 1) {
                                // part Re: N = (e + o) + i (pe + po); part Im: S = (pe - po) + i (e - o);
                                // c = 0 stores -conj of them
                                const C2 v = sg ? cmk<C2>(pe - po, e - o) : cmk<C2>(e + o, pe + po);
                                dst[(size_t)r * P * ly.unit] = c == 2 ? v : cmk<C2>(-v.x, v.y);
                            } else {
                                // north N = (E + O) over both parts, south S = (E - O); the
                                // input at +am is N + i S, at -am conj N + i conj S
                                dst[(size_t)r * P * ly.unit] =
                                    sg ? cmk<C2>(pe + po + (e - o), (pe - po) - (e + o))
                                       : cmk<C2>(e + o - (pe - po), pe + po + (e - o));
                            }
                        } else {
                            dst[(size_t)r * P * ly.unit] = cmk<C2>(e + o, e - o);
                        }
                    }
                }
            }
        }
        lds_barrier();
        // ---- 2. synthesis: pass 1 on rows (orders |m| > Lm are zero), pass 2 on columns
        {
            const int ntask = Uq * NS * A;
            for (int task = tid; task < ntask; task += kThreads) {
                const int t = task % A, f = task / A;
                C2* row = ubuf(f / NS) + (f % NS) * FS + t * BP;
                C2 v[B];
#pragma unroll
                for (int n2i = 0; n2i < B; ++n2i) {
                    const int n = t + A * n2i;
                    const int am = n <= Phi - n ? n : Phi - n;
                    v[n2i] = am <= Lm ? row[n2i] : cmk<C2>((T)0, (T)0);
                }
                Dft<B, true, C2>::run(v);
                const C2* twr = tw2 + t * BP;
                C2 w[B];
#pragma unroll
                for (int k2 = 1; k2 < B; ++k2) w[k2] = twr[k2];
#pragma unroll
                for (int k2 = 0; k2 < B; ++k2) row[k2] = k2 == 0 ? v[k2] : cmulc(v[k2], w[k2]);
            }
        }
        lds_barrier();
        {
            const int ntask = Uq * NS * B;
            for (int task = tid; task < ntask; task += kThreads) {
                const int k2 = task % B, f = task / B;
                C2* fb = ubuf(f / NS) + (f % NS) * FS + k2;
                C2 u[A];
#pragma unroll
                for (int t = 0; t < A; ++t) u[t] = fb[t * BP];
                Dft<A, true, C2>::run(u);
#pragma unroll
                for (int k1 = 0; k1 < A; ++k1) fb[k1 * BP] = u[k1];
            }
        }
        lds_barrier();
        // ---- 3. products on half the circle; the product of component c goes to
        // slot NC + c (positions n and -n are read and written by one task)
        if constexpr (RL && S == 0) {
            // real signals: north = Re, south = Im of each transform, on the whole circle
            const int ntask = Uq * Phi;
            for (int task = tid; task < ntask; task += kThreads) {
                const int n = task % Phi, pn = n + n / B;
                C2* fb = ubuf(task / Phi);
                const C2 f1 = fb[pn], f2 = fb[FS + pn];
                fb[FS + pn] = cmk<C2>(f1.x * f2.x, f1.y * f2.y);
            }
        } else if constexpr (RL) {
            // spin 1, real fields: per hemisphere f_+1 (slot 0 north, slot 2 south), f_0 =
            // Re / Im of slot 1, f_-1 = -conj f_+1; the coupling gives g_+1 = b0 a+ - a0 b+
            // and g_0 = a+ b- - a- b+ = -2 i Im(a+ conj b+) (g_-1 = conj g_+1): slot 3 and 5
            // take g_+1's north and south, slot 4 Im g_0 (north + i south)
            const int ntask = Uq * Phi;
            for (int task = tid; task < ntask; task += kThreads) {
                const int n = task % Phi, pn = n + n / B;
                C2* fb = ubuf(task / Phi);
                const C2 an = fb[pn], a0 = fb[FS + pn], as = fb[2 * FS + pn];
                const C2 bn = fb[3 * FS + pn], b0 = fb[4 * FS + pn], bs = fb[5 * FS + pn];
                fb[3 * FS + pn] = cmk<C2>(b0.x * an.x - a0.x * bn.x, b0.x * an.y - a0.x * bn.y);
                fb[5 * FS + pn] = cmk<C2>(b0.y * as.x - a0.y * bs.x, b0.y * as.y - a0.y * bs.y);
                fb[4 * FS + pn] = cmk<C2>((T)-2 * (an.y * bn.x - an.x * bn.y), (T)-2 * (as.y * bs.x - as.x * bs.y));
            }
        } else {
            const int ntask = Uq * H;
            for (int task = tid; task < ntask; task += kThreads) {
                const int n = task % H;
                C2* fb = ubuf(task / H);
                const int kk = n == 0 ? 0 : Phi - n;
                const int pn = n + n / B, pk = kk + kk / B;
                // unpacked (times 2): north = F(n) + conj F(-n), south = -i (F(n) - conj F(-n))
                C2 gn[NC], gs[NC];
                if constexpr (S == 2) {
                    // 2 (x) 2 -> 2 coupling of components q = -2..2 (slots c = q + 2 of input 0, then of
                    // input 1), one hemisphere at a time (its ten unpacked components only).
                    // C^{2 q}_{2 q1 2 q2} is +-1, +-2 or +-sqrt(6) times 1 / sqrt(14); the common factor
                    // is in the plan's recombination weights (which checks this pattern)
                    const T r6 = (T)2.449489742783178098197284;   // sqrt(6)
#pragma unroll
                    for (int hs = 0; hs < 2; ++hs) {
                        C2 f[NS];
#pragma unroll
                        for (int s2 = 0; s2 < NS; ++s2) {
                            const C2 Fn = fb[s2 * FS + pn], Fk = fb[s2 * FS + pk];
                            f[s2] = hs ? cmk<C2>(Fn.y + Fk.y, Fk.x - Fn.x) : cmk<C2>(Fn.x + Fk.x, Fn.y - Fk.y);
                        }
                        const C2* a = f;        // a[q + 2]
                        const C2* b = f + NC;   // b[q + 2]
                        C2* g = hs ? gs : gn;
                        auto lin = [](T u, C2 x, T v, C2 y) { return cmk<C2>(u * x.x + v * y.x, u * x.y + v * y.y); };
                        // q = +2: 2 (a0 b2 + a2 b0) - sqrt6 a1 b1
                        g[4] = lin((T)2, cadd(cmul(a[2], b[4]), cmul(a[4], b[2])), -r6, cmul(a[3], b[3]));
                        // q = +1: sqrt6 (a-1 b2 + a2 b-1) - (a0 b1 + a1 b0)
                        g[3] = lin(r6, cadd(cmul(a[1], b[4]), cmul(a[4], b[1])), (T)-1,
                                   cadd(cmul(a[2], b[3]), cmul(a[3], b[2])));
                        // q = 0: 2 (a-2 b2 + a2 b-2) + (a-1 b1 + a1 b-1) - 2 a0 b0
                        g[2] = cadd(lin((T)2, cadd(cmul(a[0], b[4]), cmul(a[4], b[0])), (T)-2, cmul(a[2], b[2])),
                                    cadd(cmul(a[1], b[3]), cmul(a[3], b[1])));
                        // q = -1: sqrt6 (a-2 b1 + a1 b-2) - (a-1 b0 + a0 b-1)
                        g[1] = lin(r6, cadd(cmul(a[0], b[3]), cmul(a[3], b[0])), (T)-1,
                                   cadd(cmul(a[1], b[2]), cmul(a[2], b[1])));
                        // q = -2: 2 (a-2 b0 + a0 b-2) - sqrt6 a-1 b-1
                        g[0] = lin((T)2, cadd(cmul(a[0], b[2]), cmul(a[2], b[0])), -r6, cmul(a[1], b[1]));
                    }
                } else {
                C2 fn[NS], fs[NS];
#pragma unroll
                for (int s = 0; s < NS; ++s) {
                    const C2 Fn = fb[s * FS + pn], Fk = fb[s * FS + pk];
                    fn[s] = cmk<C2>(Fn.x + Fk.x, Fn.y - Fk.y);
                    fs[s] = cmk<C2>(Fn.y + Fk.y, Fk.x - Fn.x);
                }
                if (S == 0) {
                    gn[0] = cmul(fn[0], fn[1]);
                    gs[0] = cmul(fs[0], fs[1]);
                } else {
                    // antisymmetric 1 (x) 1 -> 1 coupling of components q = -1, 0, +1
                    // (slots c = q + 1 of input 0, then of input 1); its constant is in the plan's weights
#pragma unroll
                    for (int hs = 0; hs < 2; ++hs) {
                        const C2* a = hs ? fs : fn;
                        const C2* b = a + NC;
                        C2* g = hs ? gs : gn;
                        g[2] = csub(cmul(a[2], b[1]), cmul(a[1], b[2]));
                        g[1] = csub(cmul(a[2], b[0]), cmul(a[0], b[2]));
                        g[0] = csub(cmul(a[1], b[0]), cmul(a[0], b[1]));
                    }
                }
                }
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    C2* z = fb + (NC + c) * FS;
                    z[pn] = cmk<C2>(gn[c].x - gs[c].y, gn[c].y + gs[c].x);
                    if (kk != n) z[pk] = cmk<C2>(gn[c].x + gs[c].y, gs[c].x - gn[c].y);
                }
            }
        }
        lds_barrier();
        // ---- 4. analysis: pass 1 reads slot NC + z and writes rows of slot z, pass 2 in place
        {
            const int ntask = Uq * NC * A;
            for (int task = tid; task < ntask; task += kThreads) {
                const int t = task % A, f = task / A;
                const int z = f % NC;
                C2* ub = ubuf(f / NC);
                const C2* zb = ub + (NC + z) * FS;
                C2 v[B];
#pragma unroll
                for (int n2i = 0; n2i < B; ++n2i) {
                    const int n = t + A * n2i;
                    v[n2i] = zb[n + n / B];
                }
                Dft<B, false, C2>::run(v);
                C2* row = ub + z * FS + t * BP;
                const C2* twr = tw2 + t * BP;
                C2 w[B];
#pragma unroll
                for (int k2 = 1; k2 < B; ++k2) w[k2] = twr[k2];
#pragma unroll
                for (int k2 = 0; k2 < B; ++k2) row[k2] = k2 == 0 ? v[k2] : cmul(v[k2], w[k2]);
            }
        }
        lds_barrier();
        {
            const int ntask = Uq * NC * B;
            for (int task = tid; task < ntask; task += kThreads) {
                const int k2 = task % B, f = task / B;
                C2* fb = ubuf(f / NC) + (f % NC) * FS + k2;
                C2 u[A];
#pragma unroll
                for (int t = 0; t < A; ++t) u[t] = fb[t * BP];
                Dft<A, false, C2>::run(u);
#pragma unroll
                for (int k1 = 0; k1 < A; ++k1) fb[k1 * BP] = u[k1];
            }
        }
        lds_barrier();
        // ---- 5. Legendre projection on MFMA, four rings per step: the step's
        // weights (buffer loads) and spectra (LDS) are all requested before the
        // products issue
        for (int h = 0; h < G / 4; ++h) {
            if (rg0 + 4 * h >= R) break;
            const int hofs = h * 4 * P * ly.unit * (int)sizeof(C2);
            const int ringofs = (rg0 + 4 * h) * d.wrow;
            int tw[MT];
#pragma unroll
            for (int s = 0; s < MT; ++s) tw[s] = s < ntw ? __builtin_amdgcn_readfirstlane(ptab[wave + kWaves * s]) : 0;
            T av[MT];
#pragma unroll
            for (int s = 0; s < MT; ++s)
                av[s] = s < ntw ? buffer_load<T>(pw_rsrc, a_lane, ((tw[s] & 0xfffff) + ringofs) * (int)sizeof(T)) : (T)0;
#pragma unroll
            for (int s = 0; s < MT; ++s) {
                if (s < ntw) {
                    const int am = (tw[s] >> 20) & 127;
                    T bv;
                    if constexpr (RL) {
                        const int km = am ? Phi - am : 0;
                        const T eps = (tw[s] >> 27) ? (T)-1 : (T)1;
                        if (S == 0 || c_l == 1) {
                            // Re (part 0) and Im (part 1) of (analysis at +am + conj(at -am)) / 2 and of
                            // (at +am - conj(at -am)) / 2i, north + eps south, doubled (the plan halves it)
                            const C2 zp = *reinterpret_cast<const C2*>(smem + b_lane + (am + am / B) * (int)sizeof(C2) + hofs);
                            const C2 zm = *reinterpret_cast<const C2*>(smem + b_lane + (km + km / B) * (int)sizeof(C2) + hofs);
                            bv = sg_l ? (zp.y - zm.y) - eps * (zp.x - zm.x) : (zp.x + zm.x) + eps * (zp.y + zm.y);
                        } else {
                            // spin 1, g_+1 (c = 2) at +am, g_-1 = conj g_+1(-m) (c = 0): north in
                            // slot 0, south in slot 2 of the unit (b_lane points at slot c_l)
                            const int k = c_l == 2 ? am : km;
                            const int u0 = b_lane - c_l * FS * (int)sizeof(C2) + (k + k / B) * (int)sizeof(C2) + hofs;
                            const C2 zn = *reinterpret_cast<const C2*>(smem + u0);
                            const C2 zs = *reinterpret_cast<const C2*>(smem + u0 + 2 * FS * (int)sizeof(C2));
                            const T re = zn.x + eps * zs.x, im = zn.y + eps * zs.y;
                            bv = sg_l ? (c_l == 2 ? im : -im) : re;
                        }
                    } else {
                        const int k = sg_l ? (am ? Phi - am : 0) : am;
                        const C2 zv = *reinterpret_cast<const C2*>(smem + b_lane + (k + k / B) * (int)sizeof(C2) + hofs);
                        bv = (tw[s] >> 27) ? zv.x - zv.y : zv.x + zv.y;
                    }
                    acc[s] = mfma16(av[s], bv, acc[s]);
                }
            }
        }
        lds_barrier();
    }

    // ---- spectra of every pair to LDS: [pair][component][l3^2 + l3 + m]; the
    // real-basis spin-1 kernel keeps its order-0 imaginary parts after them
    // ([(Lo + 1)^2 + l3])
    const int no = (Lo + 1) * (Lo + 1);
    const int nos = (RL && S == 1) ? no + Lo + 1 : no;   // per-component stride
#pragma unroll
    for (int s = 0; s < MT; ++s) {
        if (s < ntw) {
            const ProjTile pt = tb.proj[wave + kWaves * s];
            const int ncp = ((pt.am || (RL && S == 1)) ? 2 : 1) * NC * P;
            if (li < ncp) {
                const int sg = li / (NC * P), c = (li / P) % NC, p = li % P;
                const bool im0 = RL && S == 1 && sg && pt.am == 0;
                const int m = sg ? -pt.am : pt.am;
                T* hp = hc + (size_t)(p * NC + c) * nos + (im0 ? no : m);
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int l3 = pt.am + pt.par + 2 * (acc_row<T>(kq, v) + 16 * pt.rt);
                    if (l3 <= Lo) hp[im0 ? l3 : l3 * l3 + l3] = acc[s][v];
                }
            }
        }
    }
    lds_barrier();
    // ---- recombination and contiguous stores
    if constexpr (S == 2) {
        // five terms per output: weights and end-phase entries in two words each
        const Acc* cf4 = reinterpret_cast<const Acc*>(tb.coef);
        const int4* ci4 = reinterpret_cast<const int4*>(tb.coefi);
        const int nout = d.nout, hs = NC * no;
        // (outputs are stored non-temporally: they are not read again here)
        for (int o = tid; o < nout; o += kThreads) {
            const Acc ca = cf4[2 * o], cb = cf4[2 * o + 1];
            const int4 ia = ci4[2 * o], ib = ci4[2 * o + 1];
            int cc = cp.c0;
            const int lo = (CH && ch.wo) ? tb.lab[d.nin + d.nin2 + o] : 0;
            for (int p = 0; p < np; ++p) {
                const T* hp = hc + (size_t)p * hs;
                T v = ca.x * hp[ia.x] + ca.y * hp[ia.y] + ca.z * hp[ia.z] + ca.w * hp[ia.w] + cb.x * hp[ib.x];
                if constexpr (CH) {
                    if (ch.wo) {
                        const int64_t k = (ch.flags & kChanPerRow) ? p0 + p : cc;
                        v *= ch.wo[k * ch.nlo + lo];
                    }
                    cc = cc + 1 == ch.channels ? 0 : cc + 1;
                }
                if (d.flags & kNegate) v = -v;
                __builtin_nontemporal_store(v, out + (p0 + p) * (int64_t)nout + o);
            }
        }
    } else {
        const Acc* cf4 = reinterpret_cast<const Acc*>(tb.coef);
        const int4* ci4 = reinterpret_cast<const int4*>(tb.coefi);
        const int nout = d.nout, hs = NC * nos;
        for (int o0 = tid; o0 < nout; o0 += 4 * kThreads) {
            Acc cf[4];
            int4 ix[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int o = min(o0 + u * kThreads, nout - 1);
                cf[u] = cf4[o];
                ix[u] = ci4[o];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int o = o0 + u * kThreads;
                if (o >= nout) break;
                if constexpr (!CH) {
                    for (int p = 0; p < np; ++p) {
                        const T* hp = hc + (size_t)p * hs;
                        T v = cf[u].x * hp[ix[u].x];
                        if (S == 1) v += cf[u].y * hp[ix[u].y] + cf[u].z * hp[ix[u].z];
                        if (d.flags & kNegate) v = -v;
                        __builtin_nontemporal_store(v, out + (p0 + p) * (int64_t)nout + o);
                    }
                } else {
                    // output label weight of row p: row k of wo, k = the row or its channel
                    const int lo = ch.wo ? tb.lab[d.nin + d.nin2 + o] : 0;
                    int cc = cp.c0;
                    for (int p = 0; p < np; ++p) {
                        const T* hp = hc + (size_t)p * hs;
                        T v = cf[u].x * hp[ix[u].x];
                        if (S == 1) v += cf[u].y * hp[ix[u].y] + cf[u].z * hp[ix[u].z];
                        if (ch.wo) {
                            const int64_t k = (ch.flags & kChanPerRow) ? p0 + p : cc;
                            v *= ch.wo[k * ch.nlo + lo];
                        }
                        cc = cc + 1 == ch.channels ? 0 : cc + 1;
                        if (d.flags & kNegate) v = -v;
                        __builtin_nontemporal_store(v, out + (p0 + p) * (int64_t)nout + o);
                    }
                }
            }
        }
    }
}

// LONG: lifts of more than 4 kMaxLiftSteps degrees (only the gradient
// product's degree-2L input, fp32, Phi >= 72); a kernel of its own, so that
// the forward kernels keep their register allocation.
template <typename T, int S, bool LONG, bool CH, bool RL = false>
__device__ __forceinline__ void run_istp(const IstpTables<T>& tb, const IstpDesc& d, const T* __restrict__ x1,
                                         const T* __restrict__ x2, T* __restrict__ out, int64_t N,
                                         const IstpChan<T>& ch) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int64_t p0 = (int64_t)blockIdx.x * d.pairs;
    const int np = (int)((N - p0) < d.pairs ? (N - p0) : d.pairs);
#define ISTP_CASE(PHI, A_, B_)                                                                      \
    case PHI:                                                                                       \
        if constexpr ((sizeof(T) == 4 || PHI <= 54) && (!LONG || (sizeof(T) == 4 && PHI >= 72)) &&  \
                      (S != 2 || PHI <= 81))                                                        \
            istp_body<T, A_, B_, S, LONG, CH, RL>(tb, d, p0, np, x1, x2, out, ch, smem);            \
        break;
    switch (d.Phi) {
        ISTP_CASE(1, 1, 1)
        ISTP_CASE(6, 3, 2)
        ISTP_CASE(9, 3, 3)
        ISTP_CASE(16, 4, 4)
        ISTP_CASE(18, 6, 3)
        ISTP_CASE(24, 6, 4)
        ISTP_CASE(27, 9, 3)
        ISTP_CASE(32, 8, 4)
        ISTP_CASE(36, 6, 6)
        ISTP_CASE(48, 8, 6)
        ISTP_CASE(54, 9, 6)
        ISTP_CASE(64, 8, 8)
        ISTP_CASE(72, 9, 8)
        ISTP_CASE(81, 9, 9)
        ISTP_CASE(96, 12, 8)
        ISTP_CASE(108, 12, 9)
        ISTP_CASE(128, 16, 8)
        ISTP_CASE(144, 12, 12)
        default: break;
    }
#undef ISTP_CASE
}

#if ISTP_REAL_KERNELS
template <typename T, int S, bool LONG>
__global__ __launch_bounds__(kThreads, 1) void istp_kernel_real(IstpTables<T> tb, IstpDesc d,
                                                                const T* __restrict__ x1, const T* __restrict__ x2,
                                                                T* __restrict__ out, int64_t N) {
    run_istp<T, S, LONG, false, true>(tb, d, x1, x2, out, N, IstpChan<T>{nullptr, nullptr, nullptr, 1, 0, 0, 0, 0});
}

template <typename T>
int launch_real(const IstpTables<T>& tb, const IstpDesc& d, const T* x1, const T* x2, T* out, int64_t N,
                void* stream) {
    const int64_t grid = (N + d.pairs - 1) / d.pairs;
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    const int Lm = d.L > d.L2 ? d.L : d.L2;
    const bool long_lift = Lm + 1 > 4 * kMaxLiftSteps;
    if ((d.spin != 0 && d.spin != 1) || d.flags != kRealBasis) return (int)hipErrorInvalidConfiguration;
    if (long_lift && (sizeof(T) != 4 || d.Phi < 72 || d.spin != 0)) return (int)hipErrorInvalidConfiguration;
    void (*kern)(IstpTables<T>, IstpDesc, const T*, const T*, T*, int64_t) =
        d.spin ? istp_kernel_real<T, 1, false>
               : (long_lift ? istp_kernel_real<T, 0, true> : istp_kernel_real<T, 0, false>);
    if (d.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
        if (e != hipSuccess) return (int)e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), d.lds_bytes, (hipStream_t)stream, tb, d, x1, x2,
                       out, N);
    return (int)hipGetLastError();
}
#elif !ISTP_CHANNEL_KERNELS
template <typename T, int S, bool LONG>
__global__ __launch_bounds__(kThreads, 1) void istp_kernel(IstpTables<T> tb, IstpDesc d, const T* __restrict__ x1,
                                                           const T* __restrict__ x2, T* __restrict__ out, int64_t N) {
    run_istp<T, S, LONG, false>(tb, d, x1, x2, out, N, IstpChan<T>{nullptr, nullptr, nullptr, 1, 0, 0, 0, 0});
}

template <typename T>
int launch(const IstpTables<T>& tb, const IstpDesc& d, const T* x1, const T* x2, T* out, int64_t N, void* stream) {
    const int64_t grid = (N + d.pairs - 1) / d.pairs;
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    const int Lm = d.L > d.L2 ? d.L : d.L2;
    const bool long_lift = Lm + 1 > 4 * kMaxLiftSteps;
    if (long_lift && (sizeof(T) != 4 || d.Phi < 72)) return (int)hipErrorInvalidConfiguration;
    void (*kern)(IstpTables<T>, IstpDesc, const T*, const T*, T*, int64_t);
#if !ISTP_TENSOR_KERNELS
    if (d.spin != 0 && d.spin != 1) return (int)hipErrorInvalidConfiguration;
    if (long_lift) kern = d.spin ? istp_kernel<T, 1, true> : istp_kernel<T, 0, true>;
    else kern = d.spin ? istp_kernel<T, 1, false> : istp_kernel<T, 0, false>;
#else
    if (d.spin != 2 || long_lift || d.Phi > 81) return (int)hipErrorInvalidConfiguration;
    kern = istp_kernel<T, 2, false>;
#endif
    if (d.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
        if (e != hipSuccess) return (int)e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), d.lds_bytes, (hipStream_t)stream, tb, d, x1, x2,
                       out, N);
    return (int)hipGetLastError();
}
#else
// forward products only (input degrees <= 32: no long lifts)
template <typename T, int S>
__global__ __launch_bounds__(kThreads, 1) void istp_kernel_channels(IstpTables<T> tb, IstpDesc d,
                                                                    const T* __restrict__ x1,
                                                                    const T* __restrict__ x2, T* __restrict__ out,
                                                                    int64_t N, IstpChan<T> ch) {
    run_istp<T, S, false, true>(tb, d, x1, x2, out, N, ch);
}

template <typename T>
int launch_channels(const IstpTables<T>& tb, const IstpDesc& d, const T* x1, const T* x2, T* out, int64_t N,
                    const IstpChan<T>& ch, void* stream) {
    const int64_t grid = (N + d.pairs - 1) / d.pairs;
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    const int Lm = d.L > d.L2 ? d.L : d.L2;
    if (Lm + 1 > 4 * kMaxLiftSteps || ch.channels < 1) return (int)hipErrorInvalidConfiguration;
    void (*kern)(IstpTables<T>, IstpDesc, const T*, const T*, T*, int64_t, IstpChan<T>);
#if !ISTP_TENSOR_KERNELS
    if (d.spin != 0 && d.spin != 1) return (int)hipErrorInvalidConfiguration;
    kern = d.spin ? istp_kernel_channels<T, 1> : istp_kernel_channels<T, 0>;
#else
    if (d.spin != 2 || d.Phi > 81) return (int)hipErrorInvalidConfiguration;
    kern = istp_kernel_channels<T, 2>;
#endif
    if (d.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
        if (e != hipSuccess) return (int)e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), d.lds_bytes, (hipStream_t)stream, tb, d, x1, x2,
                       out, N, ch);
    return (int)hipGetLastError();
}
#endif

}  // namespace

// Exported launchers: spins 0 and 1 from istp_kernels.hip and
// istp_kernels_channels.hip; spin 2 from istp_kernels_tensor.hip and
// istp_kernels_channels_tensor.hip.
#if ISTP_REAL_KERNELS
int launch_istp_real_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2,
                         float* out, int64_t N, void* stream) {
    return launch_real<float>(tb, d, x1, x2, out, N, stream);
}
int launch_istp_real_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                         double* out, int64_t N, void* stream) {
    return launch_real<double>(tb, d, x1, x2, out, N, stream);
}
#elif !ISTP_CHANNEL_KERNELS && !ISTP_TENSOR_KERNELS
int launch_istp_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2, float* out,
                    int64_t N, void* stream) {
    return launch<float>(tb, d, x1, x2, out, N, stream);
}
int launch_istp_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                    double* out, int64_t N, void* stream) {
    return launch<double>(tb, d, x1, x2, out, N, stream);
}
#elif !ISTP_CHANNEL_KERNELS
int launch_istp_tensor_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2,
                           float* out, int64_t N, void* stream) {
    return launch<float>(tb, d, x1, x2, out, N, stream);
}
int launch_istp_tensor_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                           double* out, int64_t N, void* stream) {
    return launch<double>(tb, d, x1, x2, out, N, stream);
}
#elif !ISTP_TENSOR_KERNELS
int launch_istp_channels_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2,
                             float* out, int64_t N, const IstpChan<float>& ch, void* stream) {
    return launch_channels<float>(tb, d, x1, x2, out, N, ch, stream);
}
int launch_istp_channels_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                             double* out, int64_t N, const IstpChan<double>& ch, void* stream) {
    return launch_channels<double>(tb, d, x1, x2, out, N, ch, stream);
}
#else
int launch_istp_channels_tensor_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1,
                                    const float* x2, float* out, int64_t N, const IstpChan<float>& ch,
                                    void* stream) {
    return launch_channels<float>(tb, d, x1, x2, out, N, ch, stream);
}
int launch_istp_channels_tensor_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1,
                                    const double* x2, double* out, int64_t N, const IstpChan<double>& ch,
                                    void* stream) {
    return launch_channels<double>(tb, d, x1, x2, out, N, ch, stream);
}
#endif

}  // namespace istp

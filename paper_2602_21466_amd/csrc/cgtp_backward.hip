// Gradients of the full CGTP: the adjoint of the block kernel's procedure
// (Section 4.3), block by block.  The CGTP is bilinear, so for an upstream
// gradient g of the outputs, the gradient for x1 (x2) is the transpose of the
// linear map x1 -> z (x2 -> z) applied to g.  Every stage of the forward
// kernel (cgtp_kernels.hip) is linear in the input it carries, and each is
// transposed here in reverse order, with the forward plan's own tables:
//
//   end phase (recombination, 1/K, scales) -> g scattered onto the
//       projection's accumulator entries with the same weights;
//   Legendre projection (MFMA)             -> Legendre synthesis: per ring and
//       order, the sum over l3 of the same weights times those entries;
//   longitude analysis (forward DFT)       -> inverse DFT, conjugate twiddles;
//   pointwise products (bilinear)          -> the incoming gradient times the
//       conjugate of the other factor;
//   longitude synthesis (inverse DFT)      -> forward DFT;
//   lift (Definition 4.1, real weights)    -> the lift's weights applied to
//       the gradient, summed over the rings.
//
// Transposes are taken for the real inner product of complex arrays, under
// which a complex-linear map's adjoint is its conjugate transpose.  The
// forward forms each product on half the circle and writes the other half as
// its conjugate (the signals have real coefficients); the scalar blocks'
// transpose below uses the equivalent full-circle form z(k) = F0(k) F1(k),
// which is the same function of the inputs and so has the same gradient.
//
// One work-group computes one (j1, j2) block for a tile of two pairs: the
// block's contribution to the pairs' gradient rows of degree j1 (x1) and j2
// (x2), written to a workspace; a last kernel sums the contributions over the
// other degree in a fixed order.  The phases are work-group-wide task pools
// separated by barriers; rings go bd.bwd_rings at a time.  Small blocks run
// on 256-thread work-groups, large ones on 768 threads; in both the
// accumulator-entry gradients are held in registers as the B operands of the
// transposed projection (wave w owns |m| = w, w + waves, ...), and the two
// pairs share the staged Legendre values, the weight loads and the barriers.

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "cgtp_internal.h"
#include "device_common.h"

namespace cgtp {
namespace {

using namespace ::cgtp::dev;

template <typename T, int A, int B, bool SMALL>
__device__ __forceinline__ void bwd_body(const Tables<T>& tb, const BlockDesc& bd, int64_t n0, int64_t N,
                                         const T* __restrict__ x1, const T* __restrict__ x2,
                                         const T* __restrict__ gin, T* __restrict__ wbase, int L,
                                         unsigned char* smem) {
    using C = typename Cplx<T>::type;
    constexpr int Phi = A * B;
    constexpr int H = Phi / 2 + 1;
    constexpr int BP = B + 1;
    constexpr int FS = slot_stride(A, B);
    constexpr int NT = SMALL ? kBwdSmallThreads : kBwdThreads;
    constexpr int NW = NT / 64;                       // waves
    constexpr int P = SMALL ? kBwdSmallPairs : kBwdLargePairs;   // pairs of the work-group
    constexpr int MPW = BwdGeom<T, SMALL>::mpw;       // |m| values per wave
    constexpr int KS = bwd_ks<T, SMALL>(0);           // MFMA K steps (4 rows each) of the first |m|
    using Acc = typename Cplx<T>::acc4;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, lk = lane >> 4;       // MFMA lane: column / A-row index, K index
    const int j1 = bd.j1, j2 = bd.j2, J = bd.J, R = bd.R, d = bd.d, G = bd.bwd_rings;
    const bool cross = bd.kind == kBlockCross;
    const int nslot = cross ? 4 : 2;
    const int nz = cross ? 2 : 1;          // analysis transforms
    const int ncomp = cross ? 4 : 1;       // projected components
    const int n1 = 2 * j1 + 1, n2 = 2 * j2 + 1;
    const int nin = (L + 1) * (L + 1);
    const int64_t nout = (int64_t)nin * nin;
    const int nrows = (J - d) / 2 + 1;
    const int np = (int)((N - n0) < P ? (N - n0) : P);   // pairs of this work-group that exist
    auto tmin = [&](int mp) { return mp > d ? (mp - d + 1) / 2 : 0; };

    const BwdLayout ly = bwd_layout(bd, (int)sizeof(T), G, P);
    T* lc = reinterpret_cast<T*>(smem + ly.lc);          // [3][n1] then [3][n2]
    C* tw2 = reinterpret_cast<C*>(smem + ly.tw2);        // [t][k2] = exp(-2 pi i t k2 / Phi), pass layout
    C* cvn = reinterpret_cast<C*>(smem + ly.cvn);        // [pair][slot][longitude n]: lifted coefficients
    C* cacc = reinterpret_cast<C*>(smem + ly.cacc);      // [pair][slot][longitude n]: their gradients, summed over rings
    T* prs = reinterpret_cast<T*>(smem + ly.prs);        // [ring of the group][input][longitude n]: P_j^|m(n)|
    C* fbuf = reinterpret_cast<C*>(smem + ly.fbuf);      // [unit = ring of the group * P + pair][kBwdSlots]
    auto slot = [&](int u, int s) -> C* { return fbuf + (size_t)(u * kBwdSlots + s) * FS; };
    const int zs0 = nslot;              // slots of the analysis gradients (spectra)
    const int zg0 = kBwdSlots - 2;      // slots of the product gradients (circle)

    // ---- set-up: couplings, twiddles, cleared sums
    for (int e = tid; e < 3 * n1; e += NT) lc[e] = tb.lcg[3 * j1 * j1 + e];
    for (int e = tid; e < 3 * n2; e += NT) lc[3 * n1 + e] = tb.lcg[3 * j2 * j2 + e];
    {
        const C* tw = reinterpret_cast<const C*>(tb.tw) + bd.tw_off;
        for (int e = tid; e < A * BP; e += NT) tw2[e] = tw[e];
    }
    for (int e = tid; e < P * nslot * Phi; e += NT) cacc[e] = cmk<C>((T)0, (T)0);
    // ---- the pairs' lifted coefficients, as the forward forms them (zero for
    // pairs past N):
    //   even slot: (x_m, C^{j, m}_{j, m, 1, 0} x_m), odd slot: (C^{j,m-1}_{j,m,1,-1}
    //   x_{m-1}, C^{j,m+1}_{j,m,1,1} x_{m+1}), times (-1)^m for negative m;
    //   scalar blocks (x_m, 0)
    for (int e = tid; e < P * nslot * Phi; e += NT) {
        const int ps = e / Phi, nn = e - ps * Phi, pp = ps / nslot, s = ps - pp * nslot;
        const bool first = cross ? (s < 2) : (s == 0);
        const int j = first ? j1 : j2, nj = 2 * j + 1;
        const int m = nn <= Phi / 2 ? nn : nn - Phi, am = m < 0 ? -m : m;
        C val = cmk<C>((T)0, (T)0);
        if (am <= j && pp < np) {
            const int mj = m + j;
            const T* xrow = (first ? x1 : x2) + (n0 + pp) * nin + j * j;
            const T* lcj = first ? tb.lcg + 3 * j1 * j1 : tb.lcg + 3 * j2 * j2;
            const T sg = (m < 0 && (am & 1)) ? (T)-1 : (T)1;
            if (!cross || (s & 1) == 0) {
                const T xm = sg * xrow[mj];
                val = cmk<C>(xm, cross ? lcj[nj + mj] * xm : (T)0);
            } else {
                const T xlo = mj >= 1 ? xrow[mj - 1] : (T)0;
                const T xhi = mj + 1 < nj ? xrow[mj + 1] : (T)0;
                val = cmk<C>(sg * lcj[mj] * xlo, sg * lcj[2 * nj + mj] * xhi);
            }
        }
        cvn[e] = val;
    }
    // ---- transpose of the end phase, into MFMA B operands.  Output (j3, m3) of
    // the block is a weighted sum of accumulator entries: an even path reads
    // component 0 at (l3 = j3, m3); an odd path reads, for q = -1, 0, +1,
    // component 2, 1, 3 at (l3 = j3 - 1, m3 - q) with the plan's term q + 1.
    // Each entry thus feeds one output, and its gradient is that term's weight
    // times the output's gradient.  For |m| = wave + NW t with nr rows and
    // ks = ceil(nr / 4) MFMA K steps, lane (k, j) holds the entries of rows
    // l3 = d + 2 (tmin(|m|) + ks k + s) in column j = (pair, sign, component):
    // B[t][s].  (Each lane's rows are consecutive, so its weights, operand A of
    // the same rows, come in a few wide loads.)
    const T* coefs = tb.coef + (size_t)bd.coef_off * 4;
    const int ncolp = 2 * ncomp;                        // columns of one pair
    const int cpair = li / ncolp, cc = li - cpair * ncolp;
    const int csign = cc / ncomp, ccomp = cc - csign * ncomp;
    const T* grow = gin + (n0 + cpair) * nout + bd.out_off;
    auto entry_grad = [&](int comp, int m, int l3) -> T {
        const int q = comp == 2 ? -1 : (comp == 3 ? 1 : 0);
        const int j3 = comp == 0 ? l3 : l3 + 1, m3 = m + q;
        if (j3 > J) return (T)0;
        const int o = j3 * j3 - d * d + j3 + m3;
        return coefs[4 * o + (comp == 0 ? 0 : q + 1)] * grow[o];
    };
    // the lane's column exists for the |m| at hand (and its pair for this work-group)
    auto col_ok = [&](int mp) { return cpair < P && csign < (mp == 0 ? 1 : 2); };
    T bq[MPW][KS];
#pragma unroll
    for (int t = 0; t < MPW; ++t) {
        const int mp = wave + NW * t;
        const int nr = mp <= J ? nrows - tmin(mp) : 0;
        const int l30 = d + 2 * tmin(mp);
        const bool ok = mp <= J && col_ok(mp) && cpair < np;
#pragma unroll
        for (int s = 0; s < bwd_ks<T, SMALL>(t); ++s) {
            const int ksm = (nr + 3) / 4, row = ksm * lk + s;
            bq[t][s] = (ok && s < ksm && row < nr) ? entry_grad(ccomp, csign ? -mp : mp, l30 + 2 * row) : (T)0;
        }
    }
    __syncthreads();

    // the block's weight table as a buffer resource (reads past it return zero)
    const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(tb.wtab + bd.wtab_off), (short)0, (tb.wtab_len - bd.wtab_off) * (int)sizeof(T), kBufferFlags);

    for (int rg0 = 0; rg0 < R; rg0 += G) {
        const int nrg = (R - rg0) < G ? (R - rg0) : G;
        const int nu = nrg * P;   // units (ring, pair) of the group
        // ---- 0. the group's Legendre values, staged
        for (int e = tid; e < nrg * 2 * Phi; e += NT) {
            const int nn = e % Phi, f = e / Phi, r = f >> 1;
            const int j = (f & 1) ? j2 : j1;
            const int m = nn <= Phi / 2 ? nn : nn - Phi, am = m < 0 ? -m : m;
            prs[e] = am <= j ? tb.pbar[bd.pbar_off + (size_t)(rg0 + r) * bd.pbar_stride + j * (j + 1) / 2 + am]
                             : (T)0;
        }
        // the analysis-gradient slots are cleared (orders past J stay zero)
        for (int e = tid; e < nu * nz * FS; e += NT) {
            const int u = e / (nz * FS), rest = e - u * nz * FS;
            slot(u, zs0)[rest] = cmk<C>((T)0, (T)0);   // nz consecutive slots
        }
        __syncthreads();
        // ---- 1. synthesis pass 1 of the lifts (as the forward)
        for (int task = tid; task < nu * nslot * A; task += NT) {
            const int t = task % A, f = task / A, s = f % nslot, u = f / nslot;
            const int r = u / P, pp = u - r * P;
            const bool first = cross ? (s < 2) : (s == 0);
            const C* cv = cvn + (size_t)(pp * nslot + s) * Phi + t;
            const T* pr = prs + (size_t)(2 * r + (first ? 0 : 1)) * Phi + t;
            C v[B];
#pragma unroll
            for (int i = 0; i < B; ++i) {
                const C c = cv[A * i];
                const T pv = pr[A * i];
                v[i] = cmk<C>(c.x * pv, c.y * pv);
            }
            Dft<B, true, C>::run(v);
            C* row = slot(u, s) + t * BP;
            const C* twr = tw2 + t * BP;
#pragma unroll
            for (int k2 = 0; k2 < B; ++k2) row[k2] = k2 == 0 ? v[0] : cmulc(v[k2], twr[k2]);
        }
        // ---- 3. transpose of the projection (other slots than the synthesis'),
        // on MFMA: per |m|, D[ring][column] = sum over rows l3 of A[ring][row] =
        // 2 w_r P^|m|_l3(x_r) (the forward's weight table, read in place) times
        // B[row][column] (the entry gradients); D goes to the real (even
        // component) or imaginary (odd) part of the spectrum gradient at the
        // pass-layout position of m
#pragma unroll
        for (int t = 0; t < MPW; ++t) {
            const int mp = wave + NW * t;
            if (mp <= J) {
                const int nr = nrows - tmin(mp), ksm = (nr + 3) / 4;
                const int r0 = (d + 2 * tmin(mp) - (J & 1)) / 2 + ksm * lk;   // the lane's first table row
                T a[KS];
                load_run(wrsrc, ((mp * bd.rpad + rg0 + li) * bd.wrow + r0) * (int)sizeof(T),
                         li < nrg ? min(ksm, bwd_ks<T, SMALL>(t)) : 0, a);
                Acc acc = Acc(0);
#pragma unroll
                for (int s = 0; s < bwd_ks<T, SMALL>(t); ++s)
                    if (s < ksm) acc = mfma16(ksm * lk + s < nr ? a[s] : (T)0, bq[t][s], acc);
                if (col_ok(mp)) {
                    const int k = csign ? Phi - mp : mp;
                    const int pos = 2 * (k + k / B) + (ccomp & 1);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r = acc_row<T>(lk, q);
                        if (r < nrg)
                            reinterpret_cast<T*>(slot(r * P + cpair, zs0 + (ccomp >> 1)))[pos] = acc[q];
                    }
                }
            }
        }
        __syncthreads();
        // ---- 2 and 4. synthesis pass 2 of the lifts and the transpose of analysis
        // pass 2 of the spectrum gradients: both inverse DFTs down the columns, in
        // place, over the consecutive slots 0 .. nslot + nz - 1
        for (int task = tid; task < nu * (nslot + nz) * B; task += NT) {
            const int k2 = task % B, f = task / B, s = f % (nslot + nz), u = f / (nslot + nz);
            C* fb = slot(u, s) + k2;
            C w[A];
#pragma unroll
            for (int t = 0; t < A; ++t) w[t] = fb[t * BP];
            Dft<A, true, C>::run(w);
#pragma unroll
            for (int k1 = 0; k1 < A; ++k1) fb[k1 * BP] = w[k1];
        }
        __syncthreads();
        // ---- 5. transpose of analysis pass 1: conjugate twiddles, inverse DFT
        // along the row, back to the longitudes n = t + A n2 (product gradients)
        for (int task = tid; task < nu * nz * A; task += NT) {
            const int t = task % A, f = task / A, z = f % nz, u = f / nz;
            const C* row = slot(u, zs0 + z) + t * BP;
            const C* twr = tw2 + t * BP;
            C v[B];
#pragma unroll
            for (int k2 = 0; k2 < B; ++k2) v[k2] = k2 == 0 ? row[0] : cmulc(row[k2], twr[k2]);
            Dft<B, true, C>::run(v);
            C* zg = slot(u, zg0 + z);
#pragma unroll
            for (int i = 0; i < B; ++i) {
                const int nn = t + A * i;
                zg[nn + nn / B] = v[i];
            }
        }
        __syncthreads();
        // ---- 6. transpose of the products at longitudes n and -n; the lifts'
        // transforms are overwritten in place with their gradients
        for (int task = tid; task < nu * H; task += NT) {
            const int nn = task % H, r = task / H;   // r: unit
            const int kk = nn == 0 ? 0 : Phi - nn;
            const int pn = nn + nn / B, pk = kk + kk / B;
            const bool self = kk == nn;
            const C* zg1 = slot(r, zg0);
            if (!cross) {
                C* f0 = slot(r, 0);
                C* f1 = slot(r, 1);
                const C a = f0[pn], b = f1[pn], za = zg1[pn];
                f0[pn] = cmulc(za, b);
                f1[pn] = cmulc(za, a);
                if (!self) {
                    const C ak = f0[pk], bk = f1[pk], zk = zg1[pk];
                    f0[pk] = cmulc(zk, bk);
                    f1[pk] = cmulc(zk, ak);
                }
                continue;
            }
            const C* zg2 = slot(r, zg0 + 1);
            // the forward writes z1 = gs + i g0 at n and conj(gs) + i conj(g0) at -n
            // (z2 likewise from g-1, g+1); transposed:
            C ggs, gg0, ggm, ggp;
            {
                const C z1n = zg1[pn], z2n = zg2[pn];
                const C z1k = self ? cmk<C>((T)0, (T)0) : cconj(zg1[pk]);
                const C z2k = self ? cmk<C>((T)0, (T)0) : cconj(zg2[pk]);
                ggs = cadd(z1n, z1k);
                gg0 = mul_mi<false>(csub(z1n, z1k));
                ggm = cadd(z2n, z2k);
                ggp = mul_mi<false>(csub(z2n, z2k));
            }
            // the unpacked signals (times 2), as the forward forms them
            C f[8];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const C* fs = slot(r, s);
                const C Fn = fs[pn], Fk = fs[pk];
                f[2 * s] = cmk<C>(Fn.x + Fk.x, Fn.y - Fk.y);
                f[2 * s + 1] = cmk<C>(Fn.y + Fk.y, Fk.x - Fn.x);
            }
            const C as = f[0], a0 = f[1], am = f[2], ap = f[3];
            const C bs = f[4], b0 = f[5], bm = f[6], bp = f[7];
            const bool even_dot = bd.products & kEvenDot, odd_sv = bd.products & kOddSV;
            C fg[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) fg[i] = cmk<C>((T)0, (T)0);
            // the gradient of a factor of a product is the product's gradient times
            // the conjugate of the other factor
            if (even_dot) {   // gs = ap bm - a0 b0 + am bp
                fg[3] = cadd(fg[3], cmulc(ggs, bm));
                fg[6] = cadd(fg[6], cmulc(ggs, ap));
                fg[1] = csub(fg[1], cmulc(ggs, b0));
                fg[5] = csub(fg[5], cmulc(ggs, a0));
                fg[2] = cadd(fg[2], cmulc(ggs, bp));
                fg[7] = cadd(fg[7], cmulc(ggs, am));
            } else {          // gs = as bs
                fg[0] = cadd(fg[0], cmulc(ggs, bs));
                fg[4] = cadd(fg[4], cmulc(ggs, as));
            }
            if (odd_sv) {     // g+1 = as bp, g0 = as b0, g-1 = as bm
                fg[0] = cadd(fg[0], cadd(cadd(cmulc(ggp, bp), cmulc(gg0, b0)), cmulc(ggm, bm)));
                fg[7] = cadd(fg[7], cmulc(ggp, as));
                fg[5] = cadd(fg[5], cmulc(gg0, as));
                fg[6] = cadd(fg[6], cmulc(ggm, as));
            } else {          // g+1 = ap b0 - a0 bp, g0 = ap bm - am bp, g-1 = a0 bm - am b0
                fg[3] = cadd(fg[3], cadd(cmulc(ggp, b0), cmulc(gg0, bm)));
                fg[1] = cadd(fg[1], csub(cmulc(ggm, bm), cmulc(ggp, bp)));
                fg[2] = csub(fg[2], cadd(cmulc(gg0, bp), cmulc(ggm, b0)));
                fg[5] = cadd(fg[5], csub(cmulc(ggp, ap), cmulc(ggm, am)));
                fg[6] = cadd(fg[6], cadd(cmulc(gg0, ap), cmulc(ggm, a0)));
                fg[7] = csub(fg[7], cadd(cmulc(ggp, a0), cmulc(gg0, am)));
            }
            // transpose of the unpacking fA = F(n) + conj F(-n), fB = -i (F(n) - conj F(-n)):
            // F(n) receives fA' + i fB', F(-n) receives conj(fA' - i fB')
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const C ga = fg[2 * s], ign = mul_mi<true>(fg[2 * s + 1]);
                const C dn = cadd(ga, ign), dk = cconj(csub(ga, ign));
                C* fs = slot(r, s);
                if (self) {
                    fs[pn] = cadd(dn, dk);
                } else {
                    fs[pn] = dn;
                    fs[pk] = dk;
                }
            }
        }
        __syncthreads();
        // ---- 7. transpose of synthesis pass 2: forward DFT down the columns
        for (int task = tid; task < nu * nslot * B; task += NT) {
            const int k2 = task % B, f = task / B, s = f % nslot, r = f / nslot;   // r: unit
            C* fb = slot(r, s) + k2;
            C u[A];
#pragma unroll
            for (int t = 0; t < A; ++t) u[t] = fb[t * BP];
            Dft<A, false, C>::run(u);
#pragma unroll
            for (int k1 = 0; k1 < A; ++k1) fb[k1 * BP] = u[k1];
        }
        __syncthreads();
        // ---- 8. transpose of synthesis pass 1: twiddles, forward DFT along the
        // row; the coefficient gradient at longitude n = t + A n2 is that times
        // the Legendre value, kept in natural order in slot nslot + s
        for (int task = tid; task < nu * nslot * A; task += NT) {
            const int t = task % A, f = task / A, s = f % nslot, u = f / nslot;
            const int r = u / P;
            const bool first = cross ? (s < 2) : (s == 0);
            const C* row = slot(u, s) + t * BP;
            const C* twr = tw2 + t * BP;
            C v[B];
#pragma unroll
            for (int k2 = 0; k2 < B; ++k2) v[k2] = k2 == 0 ? row[0] : cmul(row[k2], twr[k2]);
            Dft<B, false, C>::run(v);
            const T* pr = prs + (size_t)(2 * r + (first ? 0 : 1)) * Phi + t;
            C* out = slot(u, nslot + s);
#pragma unroll
            for (int i = 0; i < B; ++i) {
                const T pv = pr[A * i];
                out[t + A * i] = cmk<C>(v[i].x * pv, v[i].y * pv);
            }
        }
        __syncthreads();
        // ---- 9. sum over the group's rings, in ring order, per pair
        for (int e = tid; e < P * nslot * Phi; e += NT) {
            const int ps = e / Phi, nn = e - ps * Phi, pp = ps / nslot, s = ps - pp * nslot;
            C sum = cacc[e];
            for (int r = 0; r < nrg; ++r) sum = cadd(sum, slot(r * P + pp, nslot + s)[nn]);
            cacc[e] = sum;
        }
        __syncthreads();
    }

    // ---- transpose of the lift: each input component collects the gradients of
    // the lifted coefficients it was placed in, with the same weights
    auto sgn = [&](int m) -> T { return (m < 0 && ((-m) & 1)) ? (T)-1 : (T)1; };
    const int nrow = n1 + n2;
    for (int e = tid; e < np * nrow; e += NT) {
        const int pp = e / nrow, ee = e - pp * nrow;
        auto at = [&](int s, int m) -> C { return cacc[(pp * nslot + s) * Phi + (m < 0 ? Phi + m : m)]; };
        const bool first = ee < n1;
        const int j = first ? j1 : j2, nj = 2 * j + 1, mj = first ? ee : ee - n1, mc = mj - j;
        const T* lcj = first ? lc : lc + 3 * n1;
        const int s0 = first ? 0 : (cross ? 2 : 1);   // the input's even slot
        // even slot, order mc: (x, C0 x)
        const C c = at(s0, mc);
        T acc = sgn(mc) * (c.x + (cross ? lcj[nj + mj] * c.y : (T)0));
        if (cross) {
            // odd slot: real part of order mc + 1 holds C- x_mc, imaginary part of
            // order mc - 1 holds C+ x_mc
            if (mc + 1 <= j) acc += sgn(mc + 1) * lcj[mj + 1] * at(s0 + 1, mc + 1).x;
            if (mc - 1 >= -j) acc += sgn(mc - 1) * lcj[2 * nj + mj - 1] * at(s0 + 1, mc - 1).y;
        }
        wbase[(n0 + pp) * nrow + ee] = acc;
    }
}

// Work-group -> (block, tile of pairs); the block body for the block's longitude size.
template <typename T, bool SMALL>
__global__ __launch_bounds__(SMALL ? kBwdSmallThreads : kBwdThreads) void bwd_kernel(
        Tables<T> tb, const int32_t* __restrict__ list, const T* __restrict__ x1, const T* __restrict__ x2,
        const T* __restrict__ g, T* __restrict__ ws, int64_t N, int L) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int P = SMALL ? kBwdSmallPairs : kBwdLargePairs;
    const int64_t ntile = (N + P - 1) / P;
    const int64_t wg = blockIdx.x;
    const int li = (int)(wg / ntile);
    const int64_t n0 = (wg - (int64_t)li * ntile) * P;
    const BlockDesc bd = tb.blocks[list[li]];
    T* wbase = ws + bwd_block_off(L, bd.j1, bd.j2) * N;
#define CGTP_BCASE(PHI, A_, B_) \
    case PHI: bwd_body<T, A_, B_, SMALL>(tb, bd, n0, N, x1, x2, g, wbase, L, smem); break;
    switch (bd.Phi) {
        CGTP_BCASE(1, 1, 1)
        CGTP_BCASE(2, 2, 1)
        CGTP_BCASE(3, 3, 1)
        CGTP_BCASE(4, 2, 2)
        CGTP_BCASE(6, 3, 2)
        CGTP_BCASE(8, 4, 2)
        CGTP_BCASE(9, 3, 3)
        CGTP_BCASE(12, 4, 3)
        CGTP_BCASE(16, 4, 4)
        CGTP_BCASE(18, 6, 3)
        CGTP_BCASE(24, 6, 4)
        CGTP_BCASE(27, 9, 3)
        CGTP_BCASE(32, 8, 4)
        CGTP_BCASE(36, 6, 6)
        CGTP_BCASE(48, 8, 6)
        CGTP_BCASE(54, 9, 6)
        CGTP_BCASE(64, 8, 8)
        CGTP_BCASE(72, 9, 8)
        CGTP_BCASE(81, 9, 9)
        CGTP_BCASE(96, 12, 8)
        CGTP_BCASE(108, 12, 9)
        CGTP_BCASE(128, 16, 8)
        CGTP_BCASE(144, 12, 12)
        default: break;
    }
#undef CGTP_BCASE
}

// Sums of the blocks' contributions in a fixed order: gx1[n, (l, m)] over the
// blocks (l, j2), gx2[n, (l, m)] over the blocks (j1, l).  One thread per
// (input, pair, component).
template <typename T>
__global__ __launch_bounds__(256) void bwd_reduce_kernel(const T* __restrict__ ws, T* __restrict__ gx1,
                                                         T* __restrict__ gx2, int64_t N, int L) {
    const int nin = (L + 1) * (L + 1);
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= 2 * N * nin) return;
    const int which = (int)(e / (N * nin));
    const int64_t rest = e - (int64_t)which * N * nin;
    const int64_t n = rest / nin;
    const int c = (int)(rest - n * nin);
    T* dst = which == 0 ? gx1 : gx2;
    if (!dst) return;
    int l = 0;
    while ((l + 1) * (l + 1) <= c) ++l;
    const int i = c - l * l;   // component within degree l
    T sum = (T)0;
    for (int o = 0; o <= L; ++o) {
        const int j1 = which == 0 ? l : o, j2 = which == 0 ? o : l;
        const int w = 2 * (j1 + j2) + 2;
        sum += ws[bwd_block_off(L, j1, j2) * N + n * w + (which == 0 ? i : 2 * j1 + 1 + i)];
    }
    dst[n * nin + c] = sum;
}

template <typename T, bool SMALL>
int launch_variant(const Tables<T>& tb, const int32_t* list, int64_t nblocks, int lds, const T* x1, const T* x2,
                   const T* g, T* ws, int64_t N, int L, void* stream) {
    constexpr int P = SMALL ? kBwdSmallPairs : kBwdLargePairs;
    const int64_t grid = nblocks * ((N + P - 1) / P);
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    if (lds > 64 * 1024) {
        hipError_t e =
            hipFuncSetAttribute((const void*)bwd_kernel<T, SMALL>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        if (e != hipSuccess) return (int)e;
    }
    hipLaunchKernelGGL((bwd_kernel<T, SMALL>), dim3((unsigned)grid), dim3(SMALL ? kBwdSmallThreads : kBwdThreads),
                       lds, (hipStream_t)stream, tb, list, x1, x2, g, ws, N, L);
    return (int)hipGetLastError();
}

template <typename T>
int launch_bwd(const Tables<T>& tb, const BwdLaunch& bl, const T* x1, const T* x2, const T* g, T* gx1, T* gx2,
               T* ws, int64_t N, int L, void* stream) {
    int err = launch_variant<T, true>(tb, bl.block_list, bl.nsmall, bl.lds_small, x1, x2, g, ws, N, L, stream);
    if (err) return err;
    err = launch_variant<T, false>(tb, bl.block_list + bl.nsmall, bl.nlarge, bl.lds_large, x1, x2, g, ws, N, L,
                                   stream);
    if (err) return err;
    const int64_t rgrid = (2 * N * (int64_t)(L + 1) * (L + 1) + 255) / 256;
    if (rgrid <= 0) return 0;
    if (rgrid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(bwd_reduce_kernel<T>, dim3((unsigned)rgrid), dim3(256), 0, (hipStream_t)stream, ws, gx1, gx2,
                       N, L);
    return (int)hipGetLastError();
}

}  // namespace

int launch_backward_f32(const Tables<float>& tb, const BwdLaunch& bl, const float* x1, const float* x2,
                        const float* g, float* gx1, float* gx2, float* ws, int64_t N, int L, void* stream) {
    return launch_bwd<float>(tb, bl, x1, x2, g, gx1, gx2, ws, N, L, stream);
}
int launch_backward_f64(const Tables<double>& tb, const BwdLaunch& bl, const double* x1, const double* x2,
                        const double* g, double* gx1, double* gx2, double* ws, int64_t N, int L, void* stream) {
    return launch_bwd<double>(tb, bl, x1, x2, g, gx1, gx2, ws, N, L, stream);
}

}  // namespace cgtp

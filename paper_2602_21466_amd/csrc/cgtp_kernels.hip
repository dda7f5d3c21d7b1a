// Device side of the CGTP: one work-group computes one (j1, j2) block for a
// tile of pairs, i.e. one irrep-signal tensor product (Section 4.3) on the
// block's own sphere grid, in LDS and registers only.
//
// For each group of four northern rings:
//   1. lift (Definition 4.1, l = j, s = 0 and s = 1) fused into the first
//      pass of the longitude synthesis: the coefficient a_c[m] =
//      (coupling) * x_m * P^m_j(x_i) is formed as the pass loads it; two real
//      series of one input share a complex transform;
//   2. second synthesis pass (in place);
//   3. pointwise products on half the circle (the other half is the complex
//      conjugate): scalar-scalar, and the 1 (x) 1 -> 1 coupling of the two
//      toroidal fields, i.e. the cross product (Section 5.1);
//   4. longitude analysis in two passes, in place; each complex transform
//      carries two real spectra;
//   5. Legendre projection on MFMA: per |m| a [rows l3] x [4 rings] x
//      [sign, component, pair] product accumulated in registers, with the
//      Gauss weights, the north-south folding and P^m_l in the A operand.
// Then, per pair, the accumulators go through LDS once: the vector
// components are recombined with C^{j3 m3}_{j3-1, m3-q, 1, q}, every path is
// scaled by 1/K (Theorem 4.2), and the block is stored contiguously.
//
// All quantities use the complex spherical basis with Condon-Shortley phase.

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "cgtp_internal.h"
#include "device_common.h"

// This file builds the plain kernel (block_kernel); with CGTP_CHANNEL_KERNELS
// set to 1 it builds the channel-wise, path-weighted one instead
// (block_kernel_channels, cgtp_kernels_channels.hip), and with
// CGTP_REAL_KERNELS set to 1 the one for inputs and outputs in the real
// spherical-harmonic basis (block_kernel_real, cgtp_kernels_real.hip).  The
// plain kernel carries none of their bookkeeping, which would cost it
// registers in the ring loop.
#ifndef CGTP_CHANNEL_KERNELS
#define CGTP_CHANNEL_KERNELS 0
#endif
#ifndef CGTP_REAL_KERNELS
#define CGTP_REAL_KERNELS 0
#endif
#ifndef CGTP_APRE_AT
#define CGTP_APRE_AT 2
#endif

namespace cgtp {
namespace {

using namespace ::cgtp::dev;

constexpr double kRsqrt2 = 0.70710678118654752440084436210485;

__device__ __forceinline__ BlockDesc uniform_desc(const BlockDesc& g) {
    BlockDesc b;
    const int32_t* src = reinterpret_cast<const int32_t*>(&g);
    int32_t* dst = reinterpret_cast<int32_t*>(&b);
#pragma unroll
    for (int k = 0; k < (int)(offsetof(BlockDesc, out_off) / 4); ++k) dst[k] = __builtin_amdgcn_readfirstlane(src[k]);
    b.out_off = rfl64(g.out_off);
    return b;
}

// ---------------------------------------------------------------- LDS layout
//
// A longitude transform lives in "pass layout": A rows of B + 1 complex
// entries (one pad per row), element k = k2 + B k1 at k1 (B + 1) + k2.  The
// first pass writes rows, the second reads and rewrites columns in place, and
// the padding keeps both access patterns free of bank conflicts.  Slots,
// (ring, pair) units and rings are padded (slot_stride, unit_stride,
// ring_stride) so that the transforms one wave works on, and the MFMA
// operands read in place, spread over the banks.

struct Layout {
    int lc, prn, tw2, tdl, cvn, x2b, fbuf, bbuf;   // byte offsets
    int per_rp;                                      // complex entries per (ring, pair)
    int per_r;                                       // complex entries per ring
};

__device__ __forceinline__ int align16(int v) { return (v + 15) & ~15; }

// Block-level data first (couplings, Legendre rows of every ring, twiddles,
// MFMA tile table), then the tile's lifted coefficients, then the per-ring
// working set; the end phase reuses the working set for the accumulators.
template <typename T, int A, int B>
__device__ __forceinline__ Layout make_layout(const BlockDesc& b, int nslot, bool x2buf) {
    using C = typename Cplx<T>::type;
    constexpr int FS = A * (B + 1);
    constexpr int FSS = slot_stride(A, B);
    Layout l;
    const int P = b.pairs, n1 = 2 * b.j1 + 1, n2 = 2 * b.j2 + 1;
    int o = 0;
    l.lc = o; o = align16(o + (int)sizeof(T) * 3 * (n1 + n2));
    l.prn = o; o = align16(o + (int)sizeof(T) * b.R * 2 * pr_stride(A * B));
    l.tw2 = o; o = align16(o + (int)sizeof(C) * FS);
    l.tdl = o; o = align16(o + 4 * b.ntiles);
    l.cvn = o; o = align16(o + (int)sizeof(C) * P * nslot * cv_stride(A * B));
    l.x2b = o;
    if (x2buf) o = align16(o + (int)sizeof(C) * x2buf_entries(nslot, FSS, kRingGroup));
    l.per_rp = unit_stride(nslot, FSS);
    l.per_r = ring_stride(P, l.per_rp);
    l.fbuf = o;
    l.bbuf = l.fbuf;
    return l;
}

// ---------------------------------------------------------------- the block body

// RL: real-basis rows.  A real function's complex coefficients are Hermitian,
// c_-m = (-1)^m conj(c_m), and then (cross blocks) its scalar lift f_s is
// real, its q = 0 lift f_0 is i times a real signal and f_-1 = conj(f_+1), so
// one transform carries f_s + f_0 (series s_m + a0_m) and one f_+1 (series
// a+_m); the products give the real gs, i times a real g0 and g+1 (g-1 =
// conj(g+1)), carried as z1 = gs + g0 and z2 = g+1.  The MFMA columns are the
// same (real and imaginary parts of z1 and z2 at +|m| and -|m|); the end
// phase combines up to four of them per real-basis output (plan-made).
// Blocks with a degree-0 input are a scaling, the same in either basis: they
// run as in the complex basis.
template <typename T, int A, int B, bool CH, bool RL>
__device__ __forceinline__ void block_body(const Tables<T>& tb, const TileDesc* __restrict__ tdesc,
                                           const BlockDesc& bd, int64_t pt0, int64_t pt1, int64_t N,
                                           const T* __restrict__ x1, const T* __restrict__ x2,
                                           T* __restrict__ out, int L, const ChanArgs<T>& ch,
                                           unsigned char* smem) {
    using C = typename Cplx<T>::type;
    using Acc = typename Cplx<T>::acc4;
    constexpr int Phi = A * B;
    constexpr int H = Phi / 2 + 1;
    constexpr int BP = B + 1;          // padded row of the pass layout
    constexpr int FS = slot_stride(A, B);   // padded transform plus the slot padding
    constexpr int MT = MaxTiles<T>::value;
    constexpr int CVS = cv_stride(Phi), PRS = pr_stride(Phi);   // row strides of cvn and prn

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j1 = bd.j1, j2 = bd.j2, J = bd.J, R = bd.R, P = bd.pairs, lgP = bd.lg_pairs;
    const bool cross = bd.kind == kBlockCross;
    const int lgS = cross ? 2 : 1;     // nslot = 4 or 2 synthesis transforms per (ring, pair)
    const int lgZ = cross ? 1 : 0;     // nz = 2 or 1 analysis transforms per (ring, pair)
    const int nslot = 1 << lgS, nz = 1 << lgZ;
    const int ncomp = cross ? 4 : 1;   // projected components
    const int n1 = 2 * j1 + 1, n2 = 2 * j2 + 1;
    const int nin = (L + 1) * (L + 1);
    const int64_t nout = (int64_t)nin * nin;

    const Layout ly = make_layout<T, A, B>(bd, nslot, CH && bd.x2share);
    // channel-wise launch whose rows of a tile all share one second input: its
    // lift is synthesised once per ring, into a buffer of its own
    const bool xsh = CH && bd.x2share && (ch.flags & kX2Shared) && ch.channels % P == 0;
    C* x2buf = reinterpret_cast<C*>(smem + ly.x2b);      // [ring][second-input slot], pass layout
    T* lc = reinterpret_cast<T*>(smem + ly.lc);          // [3][n1] then [3][n2]
    T* prn = reinterpret_cast<T*>(smem + ly.prn);        // [ring][input][longitude n], rows PRS apart: P_j^|m(n)|, zero for |m| > j
    C* tw2 = reinterpret_cast<C*>(smem + ly.tw2);        // [t][k2] = exp(-2 pi i t k2 / Phi), pass layout
    int* tdl = reinterpret_cast<int*>(smem + ly.tdl);    // per MFMA tile: weight offset in bytes

    C* cvn = reinterpret_cast<C*>(smem + ly.cvn);        // [pair][slot][longitude n], rows CVS apart: lifted coefficients, two series
    C* fbuf = reinterpret_cast<C*>(smem + ly.fbuf);      // per (ring, pair): nslot transforms, pass layout
    T* bbuf = reinterpret_cast<T*>(smem + ly.bbuf);      // MFMA tiles, end phase only
    // transforms of (ring, pair) rp = ring * P + pair
    auto rpbuf = [&](int rp) -> C* {
        return fbuf + (size_t)(rp >> lgP) * ly.per_r + (size_t)(rp & (P - 1)) * ly.per_rp;
    };
    const TileDesc* __restrict__ td = tdesc + bd.tdesc_off;
    using Coef4 = typename Cplx<T>::acc4;
    const Coef4* coef4 = reinterpret_cast<const Coef4*>(RL ? tb.coefr : tb.coef) + bd.coef_off;
    const int4* coefi = reinterpret_cast<const int4*>(RL ? tb.coefir : tb.coefi) + bd.coef_off;

    // ---- block-level set-up: couplings, Legendre rows of every ring, twiddles
    for (int e = tid; e < 3 * n1; e += kThreads) lc[e] = tb.lcg[3 * j1 * j1 + e];
    for (int e = tid; e < 3 * n2; e += kThreads) lc[3 * n1 + e] = tb.lcg[3 * j2 * j2 + e];
    {
        const C* tw = reinterpret_cast<const C*>(tb.tw) + bd.tw_off;
        for (int e = tid; e < A * BP; e += kThreads) tw2[e] = tw[e];
    }
    // Legendre rows of every ring in longitude order: entry n of (ring, input j)
    // is P_j^|m| at the order m = n or n - Phi that longitude index n carries in
    // the synthesis, zero for |m| > j (Phi > 2 j, so n <= Phi / 2 gives m = n)
    // (four entries per thread at a time: their loads are in flight together)
    for (int e0 = tid; e0 < R * 2 * Phi; e0 += 4 * kThreads) {
        T v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * kThreads;
            const int ri = e / Phi, n = e - ri * Phi;
            const int j = (ri & 1) ? j2 : j1;
            const int m = n <= Phi / 2 ? n : n - Phi, am = m < 0 ? -m : m;
            const T* prow = tb.pbar + bd.pbar_off + (size_t)(ri >> 1) * bd.pbar_stride;
            v[u] = (e < R * 2 * Phi && am <= j) ? prow[j * (j + 1) / 2 + am] : (T)0;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * kThreads, ri = e / Phi;
            if (e < R * 2 * Phi) prn[ri * PRS + (e - ri * Phi)] = v[u];
        }
    }

    for (int u = tid; u < bd.ntiles; u += kThreads) {
        const TileDesc t = td[u];
        tdl[u] = t.a_off * (int)sizeof(T);
    }


    // MFMA operands: the block's weight table as a buffer resource (reads past it
    // return zero), and this lane's byte offsets of row / column i, ring kq
    const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(tb.wtab + bd.wtab_off), (short)0, (tb.wtab_len - bd.wtab_off) * (int)sizeof(T), kBufferFlags);
    const int lane_a = ((lane >> 4) * bd.wrow + (lane & 15)) * (int)sizeof(T);
    // B operand: the in-place analysis output of the lane's column
    // c = 16 ct + i = (sign, component, pair) of the tile's column tile ct at
    // the longitude position of +|m| or -|m| (columns past the last read
    // column 0; their results are discarded)
    const int lgC = lgP + (cross ? 2 : 0);   // log2(ncomp * pairs): columns per sign
    // this wave's MFMA tiles: wave w owns w, w + kWaves, ...; per tile the LDS
    // byte address of the lane's B operand at ring 4 h + kq, h = 0
    const int ntw = bd.ntiles > wave ? (bd.ntiles - 1 - wave) / kWaves + 1 : 0;
    // the tile whose operands slot s loads: the wave's own, or for slots past its
    // last tile (and waves without tiles) a tile of the block, never out of range
    auto tile_of = [&](int s) { return min(wave + kWaves * min(s, max(ntw - 1, 0)), bd.ntiles - 1); };
    // the MFMA weights (operand A) of this wave's tiles for the ring group at rg0
    auto prefetch_weights_at = [&](T (&ap)[kRingGroup / 4][MT], int rg) {
#pragma unroll
        for (int s = 0; s < MT; ++s) {
            if (s < ntw) {
                const int ax = tdl[tile_of(s)] + lane_a;
#pragma unroll
                for (int h = 0; h < kRingGroup / 4; ++h)
                    ap[h][s] = buffer_load<T>(wrsrc, ax, (rg + 4 * h) * bd.wrow * (int)sizeof(T));
            }
        }
    };
    int bx[MT];
#pragma unroll
    for (int s = 0; s < MT; ++s) {
        const TileDesc t = td[tile_of(s)];
        const int mp = t.code >> 16, ct = t.code & 0xff;
        int c = 16 * ct + (lane & 15);
        if (c >= ((mp == 0 ? 1 : 2) << lgC)) c = 0;
        const int comp = (c >> lgP) & (ncomp - 1), p = c & (P - 1);
        const int pos = (c >> lgC) ? (t.b_off >> 16) : (t.b_off & 0xffff);
        bx[s] = ly.fbuf +
                ((((lane >> 4) * ly.per_r + p * ly.per_rp + (comp >> 1) * FS) * 2 + (comp & 1)) + pos) *
                    (int)sizeof(T);
    }
    const bool even_dot = bd.products & kEvenDot, odd_sv = bd.products & kOddSV;
    // (the longitude quadrature and unpacking scales, the products' coupling
    // constants and the sign of negative orders are folded into the output
    // coefficients)

    // rings past the last one of the grid are read by the projection (with zero
    // weight); give them finite contents once
    {
        T* fz = reinterpret_cast<T*>(fbuf);
        for (int e = tid; e < kRingGroup * ly.per_r * 2; e += kThreads) fz[e] = (T)0;
    }
    const bool x2s = CH && (ch.flags & kX2Shared);
    // the couplings (lc) are read by other waves in the first tile's lift fill
    lds_barrier();

    for (int64_t pt = pt0; pt < pt1; ++pt) {
    const int64_t p0 = pt * P;
    const int np = (int)((N - p0) < P ? (N - p0) : P);
    // channel of the tile's first row and the pair it belongs to (rows are
    // (pair, channel), channel fastest)
    int64_t n0 = p0;
    int c0 = 0;
    if constexpr (CH) {
        n0 = p0 / ch.channels;
        c0 = (int)(p0 - n0 * ch.channels);
    }
    // ---- ring-independent lifted coefficients of the tile in longitude order
    // (zero for |m| > j and for rows past N), per slot:
    //   even slot: (x_m, C^{j, m}_{j, m, 1, 0} x_m)                          scalar and q = 0
    //   odd slot:  (C^{j,m-1}_{j,m,1,-1} x_{m-1}, C^{j,m+1}_{j,m,1,1} x_{m+1})   q = -1, +1
    // for orbital order m, times (-1)^m for negative m (P^{-m} = (-1)^m P^m);
    // scalar blocks use (x_m, 0) only.
    for (int e = tid; e < (P << lgS) * Phi; e += kThreads) {
        const int ps = e / Phi, n = e - ps * Phi;
        const int p = ps >> lgS, s = ps & (nslot - 1);
        const bool first = cross ? (s < 2) : (s == 0);
        const int j = first ? j1 : j2, nj = 2 * j + 1;
        const int m = n <= Phi / 2 ? n : n - Phi, am = m < 0 ? -m : m;
        C val = cmk<C>((T)0, (T)0);
        if (am <= j && p < np) {
            const int mj = m + j;
            const T* xg = first ? x1 : x2;
            const int64_t xr = (first || !x2s) ? p0 + p : n0 + (c0 + p) / ch.channels;
            const int64_t row = xr * nin + j * j;
            const T* lcj = first ? lc : lc + 3 * n1;
            const T sg = (m < 0 && (am & 1)) ? (T)-1 : (T)1;
            if (RL && cross) {
                // complex coefficient of order k from the real-basis row:
                // c_0 = r_0, c_k = (-1)^k (r_k - i r_-k) / sqrt 2, c_-k = (r_k + i r_-k) / sqrt 2
                const T* r0 = xg + row + j;
                auto coefc = [&](int k) -> C {
                    const int ak = k < 0 ? -k : k;
                    if (ak > j) return cmk<C>((T)0, (T)0);
                    if (k == 0) return cmk<C>(r0[0], (T)0);
                    const T rp = r0[ak] * (T)kRsqrt2, rm = r0[-ak] * (T)kRsqrt2;
                    if (k < 0) return cmk<C>(rp, rm);
                    return (ak & 1) ? cmk<C>(-rp, rm) : cmk<C>(rp, -rm);
                };
                if ((s & 1) == 0) {   // f_s + f_0: (1 + C^{j,m}_{j,m,1,0}) c_m
                    const C c = coefc(m);
                    const T f = sg * ((T)1 + lcj[nj + mj]);
                    val = cmk<C>(f * c.x, f * c.y);
                } else {              // f_+1: C^{j,m+1}_{j,m,1,1} c_{m+1}
                    const C c = coefc(m + 1);
                    const T f = sg * lcj[2 * nj + mj];
                    val = cmk<C>(f * c.x, f * c.y);
                }
            } else if (!cross || (s & 1) == 0) {
                const T xm = sg * xg[row + mj];
                val = cmk<C>(xm, cross ? lcj[nj + mj] * xm : (T)0);
            } else {
                const T xlo = mj >= 1 ? xg[row + mj - 1] : (T)0;
                const T xhi = mj + 1 < nj ? xg[row + mj + 1] : (T)0;
                val = cmk<C>(sg * lcj[mj] * xlo, sg * lcj[2 * nj + mj] * xhi);
            }
        }
        cvn[ps * CVS + n] = val;
    }

    Acc acc[MT];
#pragma unroll
    for (int s = 0; s < MT; ++s) acc[s] = Acc(0);
    lds_barrier();

    for (int rg0 = 0; rg0 < R; rg0 += kRingGroup) {
        const int nrg = (R - rg0) < kRingGroup ? (R - rg0) : kRingGroup;
        // Phases 1 to 4 work on (ring, pair) units; wave w owns units w, w + kWaves,
        // ... and takes each of them through synthesis, products and analysis, so
        // between these phases only its own LDS accesses need ordering.
        const int nunit = nrg << lgP;
        auto prefetch_weights = [&](T (&ap)[kRingGroup / 4][MT]) { prefetch_weights_at(ap, rg0); };
        const int uw = nunit > wave ? (nunit - 1 - wave) / kWaves + 1 : 0;   // units of this wave

        // Transforms of this wave: every slot of its units or, with a shared second
        // input, its units' first-input slots and its share of the group's
        // second-input transforms (one per ring and slot, from pair 0's lift),
        // dealt from the last wave down: waves with the most units come first in
        // the unit order, so the totals even out.
        const int lgH = lgS - 1;   // log2 of the slots per input
        const int nx2 = xsh ? nrg << lgH : 0;
        const int q0 = kWaves - 1 - wave;
        const int nx2w = nx2 > q0 ? (nx2 - 1 - q0) / kWaves + 1 : 0;
        const int ntr = xsh ? (uw << lgH) + nx2w : uw << lgS;
        auto tr_of = [&](int f, int& rp, int& s) {
            if (!xsh) {
                rp = wave + kWaves * (f >> lgS);
                s = f & (nslot - 1);
            } else if (f < (uw << lgH)) {
                rp = wave + kWaves * (f >> lgH);
                s = f & ((1 << lgH) - 1);
            } else {
                const int q = q0 + kWaves * (f - (uw << lgH));
                rp = (q >> lgH) << lgP;
                s = (1 << lgH) + (q & ((1 << lgH) - 1));
            }
        };
        // slot s of unit rp (the shared buffer holds the second input's slots)
        auto slotp = [&](int rp, int s) -> C* {
            if (xsh && s >= (1 << lgH)) return x2buf + (size_t)(((rp >> lgP) << lgH) + s - (1 << lgH)) * FS;
            return rpbuf(rp) + (size_t)s * FS;
        };
        // ---- 1. lift + synthesis pass 1: task (transform, t) -> row t
        {
            const int ntask = ntr * A;
            for (int task = lane; task < ntask; task += 64) {
                const int t = task % A;
                const int f = task / A;
                int rp, s;
                tr_of(f, rp, s);
                const int p = rp & (P - 1), r = rp >> lgP;
                const bool first = cross ? (s < 2) : (s == 0);
                // inputs n = t + A n2i: both factors in longitude order, read at
                // constant offsets from the task's first element
                const C* cv = cvn + (size_t)((p << lgS) + s) * CVS + t;
                const T* pr = prn + (size_t)(((rg0 + r) << 1) + (first ? 0 : 1)) * PRS + t;
                C v[B];
#pragma unroll
                for (int n2i = 0; n2i < B; ++n2i) {
                    const C c = cv[A * n2i];
                    const T pv = pr[A * n2i];
                    v[n2i] = cmk<C>(c.x * pv, c.y * pv);
                }
                Dft<B, true, C>::run(v);
                C* row = slotp(rp, s) + t * BP;
                // all twiddles first: the row stores may not be moved above them
                const C* twr = tw2 + t * BP;
                C w[B];
#pragma unroll
                for (int k2 = 1; k2 < B; ++k2) w[k2] = twr[k2];
#pragma unroll
                for (int k2 = 0; k2 < B; ++k2) row[k2] = k2 == 0 ? v[k2] : cmulc(v[k2], w[k2]);
            }
        }
        wave_lds_sync();
        // ---- 2. synthesis pass 2 (in place): task (transform, column k2)
        {
            const int ntask = ntr * B;
            for (int task = lane; task < ntask; task += 64) {
                const int k2 = task % B;
                const int f = task / B;
                int rp, s;
                tr_of(f, rp, s);
                C* fb = slotp(rp, s) + k2;
                C u[A];
#pragma unroll
                for (int t = 0; t < A; ++t) u[t] = fb[t * BP];
                Dft<A, true, C>::run(u);
#pragma unroll
                for (int k1 = 0; k1 < A; ++k1) fb[k1 * BP] = u[k1];
            }
        }
        // the shared transforms were made by other waves
        if (xsh)
            lds_barrier();
        else
            wave_lds_sync();
#if CGTP_APRE_AT == 2
        T apre[kRingGroup / 4][MT];
        prefetch_weights(apre);
#endif
        // ---- 3. pointwise products on half the circle, mirrored (real basis: on
        // the whole circle, in place)
        if (RL && cross) {
            const int ntask = uw * Phi;
            for (int task = lane; task < ntask; task += 64) {
                const int n = task % Phi, rp = wave + kWaves * (task / Phi);
                const int pn = n + n / B;
                C* fb = rpbuf(rp);
                // as = Re T1, a0 = i al (al = Im T1), a+ = T2, a- = conj(T2); b likewise
                const C t1a = fb[pn], ap = fb[FS + pn], t1b = fb[2 * FS + pn], bp = fb[3 * FS + pn];
                const T al = t1a.y, be = t1b.y;
                const T ddot = ap.x * bp.x + ap.y * bp.y;   // Re(a+ conj b+)
                // gs: as bs, or (dot) a+ b- - a0 b0 + a- b+ = 2 Re(a+ conj b+) + al be
                const T gs = even_dot ? (T)2 * ddot + al * be : t1a.x * t1b.x;
                T g0, gpx, gpy;
                if (odd_sv) {   // g+ = as b+, g0 = as b0
                    g0 = t1a.x * be;
                    gpx = t1a.x * bp.x;
                    gpy = t1a.x * bp.y;
                } else {        // g+ = a+ b0 - a0 b+ = i (be a+ - al b+), g0 = a+ b- - a- b+ = 2 i Im(a+ conj b+)
                    g0 = (T)2 * (ap.y * bp.x - ap.x * bp.y);
                    gpx = -(be * ap.y - al * bp.y);
                    gpy = be * ap.x - al * bp.x;
                }
                fb[2 * FS + pn] = cmk<C>(gs, g0);    // z1 = gs + g0 (g0 imaginary)
                fb[3 * FS + pn] = cmk<C>(gpx, gpy);  // z2 = g+1
            }
        } else {
            const int ntask = uw * H;
            for (int task = lane; task < ntask; task += 64) {
                const int n = task % H, rp = wave + kWaves * (task / H);
                const int kk = n == 0 ? 0 : Phi - n;
                const int pn = n + n / B, pk = kk + kk / B;   // pass-layout positions
                // the products overwrite the second input's transforms: positions
                // n and -n are read and written by this task only
                C* fb = rpbuf(rp);
                if (!cross) {
                    const C g = cmul(fb[pn], slotp(rp, 1)[pn]);
                    fb[FS + pn] = g;
                    fb[FS + pk] = cconj(g);
                } else {
                    // unpacked (times 2): fA = F(n) + conj F(-n), fB = -i (F(n) - conj F(-n))
                    C f[8];
#pragma unroll
                    for (int s = 0; s < 4; ++s) {
                        const C* fs = slotp(rp, s);
                        const C Fn = fs[pn], Fk = fs[pk];
                        f[2 * s] = cmk<C>(Fn.x + Fk.x, Fn.y - Fk.y);
                        f[2 * s + 1] = cmk<C>(Fn.y + Fk.y, Fk.x - Fn.x);
                    }
                    const C as = f[0], a0 = f[1], am = f[2], ap = f[3];
                    const C bs = f[4], b0 = f[5], bm = f[6], bp = f[7];
                    C gs, gp, g0, gm;
                    if (even_dot) {
                        // C^{0 0}_{1 q 1 -q} is c (+1, -1, +1) for q = 1, 0, -1; c applied at staging
                        gs = cadd(csub(cmul(ap, bm), cmul(a0, b0)), cmul(am, bp));
                    } else {
                        gs = cmul(as, bs);
                    }
                    if (odd_sv) {
                        gp = cmul(as, bp);
                        g0 = cmul(as, b0);
                        gm = cmul(as, bm);
                    } else {
                        // antisymmetric 1 (x) 1 -> 1 coupling, constant applied at staging
                        gp = csub(cmul(ap, b0), cmul(a0, bp));
                        g0 = csub(cmul(ap, bm), cmul(am, bp));
                        gm = csub(cmul(a0, bm), cmul(am, b0));
                    }
                    // z1 = gs + i g0, z2 = g-1 + i g+1; at -n the conjugated signals
                    C* z1 = fb + 2 * FS;
                    C* z2 = fb + 3 * FS;
                    z1[pn] = cmk<C>(gs.x - g0.y, gs.y + g0.x);
                    z2[pn] = cmk<C>(gm.x - gp.y, gm.y + gp.x);
                    if (kk != n) {
                        z1[pk] = cmk<C>(gs.x + g0.y, g0.x - gs.y);
                        z2[pk] = cmk<C>(gm.x + gp.y, gp.x - gm.y);
                    }
                }
            }
        }
        wave_lds_sync();
#if CGTP_APRE_AT == 1
        T apre[kRingGroup / 4][MT];
        prefetch_weights(apre);
#endif
        // ---- 4a. analysis pass 1: task ((unit, z), t); rows into slot z
        {
            const int ntask = (uw << lgZ) * A;
            for (int task = lane; task < ntask; task += 64) {
                const int t = task % A;
                const int f = task / A;
                const int z = f & (nz - 1), rp = wave + kWaves * (f >> lgZ);
                const C* zb = rpbuf(rp) + (size_t)(nslot - nz + z) * FS;
                C v[B];
#pragma unroll
                for (int n2i = 0; n2i < B; ++n2i) {
                    const int n = t + A * n2i;
                    v[n2i] = zb[n + n / B];
                }
                Dft<B, false, C>::run(v);
                C* row = rpbuf(rp) + (size_t)z * FS + t * BP;
                const C* twr = tw2 + t * BP;
                C w[B];
#pragma unroll
                for (int k2 = 1; k2 < B; ++k2) w[k2] = twr[k2];
#pragma unroll
                for (int k2 = 0; k2 < B; ++k2) row[k2] = k2 == 0 ? v[k2] : cmul(v[k2], w[k2]);
            }
        }
        wave_lds_sync();
#if CGTP_APRE_AT == 0
        // the group's MFMA weights (operand A) are fetched now and land during the
        // last transform pass (fetched earlier they would hold registers through
        // the register peak of the row passes)
        T apre[kRingGroup / 4][MT];
        prefetch_weights(apre);
#endif
        // ---- 4b. analysis pass 2, in place
        {
            const int ntask = (uw << lgZ) * B;
            for (int task = lane; task < ntask; task += 64) {
                const int k2 = task % B;
                const int f = task / B;
                const int z = f & (nz - 1), rp = wave + kWaves * (f >> lgZ);
                C* yb = rpbuf(rp) + (size_t)z * FS + k2;
                C u[A];
#pragma unroll
                for (int t = 0; t < A; ++t) u[t] = yb[t * BP];
                Dft<A, false, C>::run(u);
#pragma unroll
                for (int k1 = 0; k1 < A; ++k1) yb[k1 * BP] = u[k1];
            }
        }
        lds_barrier();
        // ---- 5. Legendre projection on MFMA, accumulated over ring groups.  Lane
        // (i, kq) feeds row i / column i of ring 4 h + kq: its weight sits at
        // a_off + ring wrow + i of the block's table (a buffer load whose ring
        // offset is scalar), its spectrum value at the lane's B offset plus the
        // tile's.
        {
#pragma unroll
            for (int h = 0; h < kRingGroup / 4; ++h) {
                const int hofs = h * 4 * ly.per_r * (int)sizeof(C);
                T bv[MT];
#pragma unroll
                for (int s = 0; s < MT; ++s) bv[s] = *reinterpret_cast<const T*>(smem + bx[s] + hofs);
                // a quad of rings wholly past the grid's last ring adds nothing
                if (h == 0 || rg0 + 4 * h < R) {
#pragma unroll
                    for (int s = 0; s < MT; ++s)
                        if (s < ntw) acc[s] = mfma16(apre[h][s], bv[s], acc[s]);
                }
            }
        }
        lds_barrier();
    }

    // ---- accumulators -> LDS verbatim (tile u at u * tile_stride), then each
    // output as up to three weighted entries (plan-made), contiguous stores
#pragma unroll
    for (int s = 0; s < MT; ++s)
        if (s < ntw) *reinterpret_cast<Acc*>(bbuf + (size_t)(wave + kWaves * s) * tile_stride<T>() + lane * 4) = acc[s];
    // path weights of the tile's rows, [row][path of the block], staged over the
    // lifted coefficients (no longer needed for this tile; they hold at least
    // pairs * (2 (j1 + j2) + 1) >= rows * paths entries)
    T* wl = reinterpret_cast<T*>(cvn);
    const int nbp = J - bd.d + 1;   // paths of the block
    if constexpr (CH) {
        if (ch.w)
            for (int e = tid; e < np * nbp; e += kThreads) {
                const int p = e / nbp, q = e - p * nbp;
                const int64_t k = (ch.flags & kWeightsPerRow) ? p0 + p : (int64_t)((c0 + p) % ch.channels);
                wl[e] = ch.w[k * ch.npaths + bd.path_off + q];
            }
    }
    lds_barrier();
    {
        const int nblk = n1 * n2;
        T* const ob = out + p0 * nout + bd.out_off;
        // the next output's coefficients are loaded while this one is stored
        Coef4 cfn{};
        int4 ixn{};
        if (tid < nblk) {
            cfn = coef4[tid];
            ixn = coefi[tid];
        }
        for (int o = tid; o < nblk; o += kThreads) {
            const Coef4 cf = cfn;
            const int4 ix = ixn;
            if (o + kThreads < nblk) {
                cfn = coef4[o + kThreads];
                ixn = coefi[o + kThreads];
            }
            const bool one = !RL && (ix.w & 1);   // scalar-scalar or dot path: one term
            const T* e0 = bbuf + ix.x;    // the terms' entries for row 0; row p's are 4 p further on
            const T* e1 = bbuf + ix.y;
            const T* e2 = bbuf + ix.z;
            const T* wq = wl + (ix.w >> 1);   // weight of this output's path, row p at nbp p
            // two rows at a time; each row's store goes through a wave-uniform row
            // pointer, non-temporal (the outputs are not read again here)
#pragma unroll 2
            for (int p = 0; p < np; ++p) {
                T z = cf.x * e0[4 * p];
                if (!one) z += cf.y * e1[4 * p] + cf.z * e2[4 * p];
                if constexpr (RL) z += cf.w * bbuf[ix.w + 4 * p];   // the real basis' fourth term
                if constexpr (CH) {
                    if (ch.w) z *= wq[p * nbp];
                }
                T* orow = ob + (int64_t)p * nout;
                __builtin_nontemporal_store(z, orow + o);
            }
        }
    }
    lds_barrier();
    }   // pair tiles
}

// Work-group -> (class, block, pair tiles) and the block body for its grid.
template <typename T, bool CH, bool RL>
__device__ __forceinline__ void run_blocks(const Tables<T>& tb, const BlockDesc* __restrict__ blocks,
                                           const TileDesc* __restrict__ tdesc, const int32_t* __restrict__ list,
                                           const LaunchMap& map, const T* __restrict__ x1,
                                           const T* __restrict__ x2, T* __restrict__ out, int64_t N, int L,
                                           const ChanArgs<T>& ch) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int64_t wg = blockIdx.x;
    int cls = 0;
    while (cls + 1 < map.ncls && wg >= map.cum[cls + 1]) ++cls;
    const int64_t wpb = map.wpb[cls];
    const int64_t local = wg - map.cum[cls];
    const int bi = (int)(local / wpb);
    const int64_t g = local - (int64_t)bi * wpb;
    // every descriptor field is wave-uniform: keep it in scalar registers
    const BlockDesc bd = uniform_desc(blocks[list[map.list_off[cls] + bi]]);
    const int64_t pt0 = g * map.tpw[cls];
    const int64_t pt1 = (pt0 + map.tpw[cls]) < map.ntiles[cls] ? (pt0 + map.tpw[cls]) : map.ntiles[cls];

#define CGTP_CASE(PHI, A_, B_) \
    case PHI: block_body<T, A_, B_, CH, RL>(tb, tdesc, bd, pt0, pt1, N, x1, x2, out, L, ch, smem); break;
    switch (bd.Phi) {
        CGTP_CASE(1, 1, 1)
        CGTP_CASE(2, 2, 1)
        CGTP_CASE(3, 3, 1)
        CGTP_CASE(4, 2, 2)
        CGTP_CASE(6, 3, 2)
        CGTP_CASE(8, 4, 2)
        CGTP_CASE(9, 3, 3)
        CGTP_CASE(12, 4, 3)
        CGTP_CASE(16, 4, 4)
        CGTP_CASE(18, 6, 3)
        CGTP_CASE(24, 6, 4)
        CGTP_CASE(27, 9, 3)
        CGTP_CASE(32, 8, 4)
        CGTP_CASE(36, 6, 6)
        CGTP_CASE(48, 8, 6)
        CGTP_CASE(54, 9, 6)
        CGTP_CASE(64, 8, 8)
        CGTP_CASE(72, 9, 8)
        CGTP_CASE(81, 9, 9)
        CGTP_CASE(96, 12, 8)
        CGTP_CASE(108, 12, 9)
        CGTP_CASE(128, 16, 8)
        CGTP_CASE(144, 12, 12)
        default: break;
    }
#undef CGTP_CASE
}

#if CGTP_REAL_KERNELS
template <typename T>
__global__ __launch_bounds__(kThreads, 1) void block_kernel_real(Tables<T> tb, const BlockDesc* __restrict__ blocks,
                                                                 const TileDesc* __restrict__ tdesc,
                                                                 const int32_t* __restrict__ list, LaunchMap map,
                                                                 const T* __restrict__ x1, const T* __restrict__ x2,
                                                                 T* __restrict__ out, int64_t N, int L) {
    run_blocks<T, false, true>(tb, blocks, tdesc, list, map, x1, x2, out, N, L, ChanArgs<T>{nullptr, 1, 0, 0});
}
#elif !CGTP_CHANNEL_KERNELS
template <typename T>
__global__ __launch_bounds__(kThreads, 1) void block_kernel(Tables<T> tb, const BlockDesc* __restrict__ blocks,
                                                            const TileDesc* __restrict__ tdesc,
                                                            const int32_t* __restrict__ list, LaunchMap map,
                                                            const T* __restrict__ x1, const T* __restrict__ x2,
                                                            T* __restrict__ out, int64_t N, int L) {
    run_blocks<T, false, false>(tb, blocks, tdesc, list, map, x1, x2, out, N, L, ChanArgs<T>{nullptr, 1, 0, 0});
}
#else
template <typename T>
__global__ __launch_bounds__(kThreads, 1) void block_kernel_channels(
        Tables<T> tb, const BlockDesc* __restrict__ blocks, const TileDesc* __restrict__ tdesc,
        const int32_t* __restrict__ list, LaunchMap map, const T* __restrict__ x1, const T* __restrict__ x2,
        T* __restrict__ out, int64_t N, int L, ChanArgs<T> ch) {
    run_blocks<T, true, false>(tb, blocks, tdesc, list, map, x1, x2, out, N, L, ch);
}
#endif

template <typename T>
int launch(const Tables<T>& tb, const int32_t* list, const LaunchMap& map, int lds, const T* x1, const T* x2,
           T* out, int64_t N, int L, const ChanArgs<T>& ch, void* stream) {
    const int64_t grid = map.cum[map.ncls];
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
#if CGTP_REAL_KERNELS
    const void* kern = (const void*)block_kernel_real<T>;
#elif !CGTP_CHANNEL_KERNELS
    const void* kern = (const void*)block_kernel<T>;
#else
    const void* kern = (const void*)block_kernel_channels<T>;
#endif
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        if (e != hipSuccess) return (int)e;
    }
#if CGTP_REAL_KERNELS
    (void)ch;
    hipLaunchKernelGGL(block_kernel_real<T>, dim3((unsigned)grid), dim3(kThreads), lds, (hipStream_t)stream, tb,
                       tb.blocks, tb.tdesc, list, map, x1, x2, out, N, L);
#elif !CGTP_CHANNEL_KERNELS
    (void)ch;
    hipLaunchKernelGGL(block_kernel<T>, dim3((unsigned)grid), dim3(kThreads), lds, (hipStream_t)stream, tb,
                       tb.blocks, tb.tdesc, list, map, x1, x2, out, N, L);
#else
    hipLaunchKernelGGL(block_kernel_channels<T>, dim3((unsigned)grid), dim3(kThreads), lds, (hipStream_t)stream,
                       tb, tb.blocks, tb.tdesc, list, map, x1, x2, out, N, L, ch);
#endif
    return (int)hipGetLastError();
}

}  // namespace

#if CGTP_REAL_KERNELS
int launch_blocks_real_f32(const Tables<float>& tb, const int32_t* list, const LaunchMap& map, int lds,
                           const float* x1, const float* x2, float* out, int64_t N, int L, void* stream) {
    return launch<float>(tb, list, map, lds, x1, x2, out, N, L, ChanArgs<float>{nullptr, 1, 0, 0}, stream);
}
int launch_blocks_real_f64(const Tables<double>& tb, const int32_t* list, const LaunchMap& map, int lds,
                           const double* x1, const double* x2, double* out, int64_t N, int L, void* stream) {
    return launch<double>(tb, list, map, lds, x1, x2, out, N, L, ChanArgs<double>{nullptr, 1, 0, 0}, stream);
}
#elif !CGTP_CHANNEL_KERNELS
int launch_blocks_f32(const Tables<float>& tb, const int32_t* list, const LaunchMap& map, int lds, const float* x1,
                      const float* x2, float* out, int64_t N, int L, void* stream) {
    return launch<float>(tb, list, map, lds, x1, x2, out, N, L, ChanArgs<float>{nullptr, 1, 0, 0}, stream);
}
int launch_blocks_f64(const Tables<double>& tb, const int32_t* list, const LaunchMap& map, int lds, const double* x1,
                      const double* x2, double* out, int64_t N, int L, void* stream) {
    return launch<double>(tb, list, map, lds, x1, x2, out, N, L, ChanArgs<double>{nullptr, 1, 0, 0}, stream);
}
#else
int launch_blocks_channels_f32(const Tables<float>& tb, const int32_t* list, const LaunchMap& map, int lds,
                               const float* x1, const float* x2, float* out, int64_t N, int L,
                               const ChanArgs<float>& ch, void* stream) {
    return launch<float>(tb, list, map, lds, x1, x2, out, N, L, ch, stream);
}
int launch_blocks_channels_f64(const Tables<double>& tb, const int32_t* list, const LaunchMap& map, int lds,
                               const double* x1, const double* x2, double* out, int64_t N, int L,
                               const ChanArgs<double>& ch, void* stream) {
    return launch<double>(tb, list, map, lds, x1, x2, out, N, L, ch, stream);
}
#endif

}  // namespace cgtp

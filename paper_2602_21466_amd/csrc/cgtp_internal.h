// Internal layout shared by the host plan (cgtp_plan.cpp) and the kernels
// (cgtp_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace cgtp {

#ifndef CGTP_THREADS
#define CGTP_THREADS 768
#endif
#ifndef CGTP_RING_GROUP
#define CGTP_RING_GROUP 8
#endif
// MFMA accumulator tiles per wave (fp32): 9 x 12 waves = 108 tiles hold the
// largest block of degree 32 (99 tiles at one pair); fewer registers than 10
// per wave, and faster in measurement although some blocks take fewer pairs
#ifndef CGTP_MAX_TILES_F32
#define CGTP_MAX_TILES_F32 9
#endif
constexpr int kThreads = CGTP_THREADS;   // work-group size of the block kernel (wave64s, one work-group per CU)
constexpr int kWaves = kThreads / 64;
constexpr int kRingGroup = CGTP_RING_GROUP;   // rings per pass: K = 4 steps of a 16x16x4 MFMA
constexpr int kLdsBudget = 160 * 1024;   // all of a gfx950 CU's LDS (one work-group per CU)
constexpr int kMaxPairs = 16;

// MFMA accumulator tiles (16 x 16) each wave may hold, per precision.
template <typename T> struct MaxTiles;
template <> struct MaxTiles<float> { static constexpr int value = CGTP_MAX_TILES_F32; };
template <> struct MaxTiles<double> { static constexpr int value = 4; };

// Product kinds per path (mirrors cgtp_path_norm's *kind).
enum PathKind : int32_t { kSS = 0, kCross = 1, kSV = 2, kDot = 3 };

// Which lifts and products a block needs.
enum BlockKind : int32_t {
    kBlockScalar = 0,   // only scalar-scalar paths (a degree-0 input)
    kBlockCross = 1,    // scalar and toroidal lifts of both inputs; four projected components
};

// Products of a kBlockCross block (BlockDesc::products); zero bits give the
// default cover's scalar-scalar (even paths) and cross (odd paths) products.
enum BlockProducts : int32_t {
    kEvenDot = 1,   // even paths: dot product of the toroidal lifts
    kOddSV = 2,     // odd paths: scalar lift of x1 times toroidal lift of x2
};

// One (j1, j2) block: one irrep-signal tensor product on its own grid.
//
// The Phi-point longitude transforms run as two in-register passes: pass 1
// does A transforms of length B over stride-A inputs, pass 2 does B transforms
// of length A (Phi = A * B, natural-order output, in place in LDS).
//
// The Legendre projection is a batch of small GEMMs, one per |m|: rows
// l3 = d, d+2, ..., J (those >= |m|), K = rings, columns (sign of m,
// component, pair).  It runs on 16x16x4 MFMA tiles whose accumulators stay in
// registers across all rings; its B operand is read in place in the analysis
// output.
struct alignas(16) BlockDesc {
    int32_t j1, j2, J, d;      // d = |j1 - j2|
    int32_t R;                 // northern rings of the block's grid
    int32_t Phi, A, B;         // longitudes, Phi = A * B
    int32_t kind;              // BlockKind
    int32_t pairs;             // pairs per work-group
    int32_t ntiles;            // MFMA accumulator tiles per work-group
    int32_t lds_bytes;         // dynamic LDS of one work-group
    int32_t tw_off;            // offset of the Phi-point twiddle table (complex entries)
    int32_t pbar_off;          // offset of the grid's Legendre table (elements)
    int32_t pbar_stride;       // Legendre entries per ring: (lmax+1)(lmax+2)/2
    int32_t wtab_off;          // offset of the MFMA weights of the grid, parity of J (elements)
    int32_t lmax;              // largest degree of the grid's tables
    int32_t coef_off;          // index of the block's first output in coef / coefi
    int32_t tdesc_off;         // offset of the block's MFMA tile descriptors
    int32_t lg_pairs;          // log2(pairs)
    int32_t products;          // BlockProducts bits
    int32_t rpad;              // rings of the weight table: R rounded up to the ring group
    int32_t wrow;              // entries per ring row of the weight table
    int32_t path_off;          // index of path (j1, j2, |j1 - j2|) in the (l1, l2, l3) order of all paths
    int32_t x2share;           // channel kernel: LDS holds a shared second-input buffer (x2_bytes) beside the working set
    int32_t bwd_rings;         // gradient kernel: rings per group (bwd_layout)
    int64_t out_off;           // offset of the block inside one pair's output
};

// One 16x16 accumulator tile of the Legendre projection, in the order the
// waves take them (wave w owns tiles w, w + 4, ...).
//   a_off: offset of (|m|, ring 0, first row l3_0) in the block's weight table
//          ([|m|][ring][row], wrow rows per ring; rows past the tile's last
//          valid one are read but their results are discarded)
//   rs_nv: valid rows of the tile << 16
//   b_off: element offsets of longitudes +|m| (bits 0..15) and -|m| (bits
//          16..31) in a transform's pass layout
//   code:  |m| << 16 | row tile << 8 | column tile
struct alignas(16) TileDesc {
    int32_t a_off, rs_nv, b_off, code;
};

// Device tables, one allocation per plan; offsets in elements of T.
//   wtab[grid]: for m' = 0..lmax, ring r, l = m'..lmax:
//     2 w_r P^{m'}_l(x_r) at  R * (m' (lmax+1) - m' (m'-1) / 2) + r (lmax - m' + 1) + (l - m')
template <typename T>
struct Tables {
    const T* pbar;      // [grid][ring][l (l+1)/2 + m]
    const T* wtab;      // see above
    const T* tw;        // per Phi, complex pairs in pass layout: [t < A][k2 < B+1] = exp(-2 pi i t k2 / Phi)
    const T* lcg;       // [j][q+1][m + j] = C^{j, m+q}_{j, m, 1, q}
    const T* coef;      // per block and output (j3, m3): up to three term weights (4 per output)
    const int32_t* coefi;   // per block and output: end-phase entries of the terms for pair 0; bit 0 of the
                            // fourth word flags a single term, the bits above it hold j3 - |j1 - j2|
    const T* coefr;         // the same for outputs in the real basis: four term weights per output
    const int32_t* coefir;  // and their four entries (no flags)
    const TileDesc* tdesc;
    int32_t wtab_len;   // elements of wtab
    const BlockDesc* blocks;
};

// Blocks grouped by pairs-per-work-group.  One launch covers every class:
// work-groups [cum[c], cum[c+1]) belong to class c, wpb[c] consecutive
// work-groups per block, heaviest classes first; each work-group walks tpw[c]
// consecutive tiles of pairs of its block.
constexpr int kMaxClasses = 8;
struct LaunchMap {
    int32_t ncls;
    int32_t pairs[kMaxClasses];
    int32_t list_off[kMaxClasses];
    int32_t tpw[kMaxClasses];       // pair tiles per work-group
    int64_t ntiles[kMaxClasses];    // pair tiles per block: ceil(N / pairs)
    int64_t wpb[kMaxClasses];       // work-groups per block: ceil(ntiles / tpw)
    int64_t cum[kMaxClasses + 1];
};

// Longitude sizes the kernel supports and their two-pass factorisation.
// Returns false when Phi is not supported.
inline bool fft_factors(int phi, int* A, int* B) {
    static const int tab[][3] = {{1, 1, 1},    {2, 2, 1},    {3, 3, 1},    {4, 2, 2},    {6, 3, 2},
                                 {8, 4, 2},    {9, 3, 3},    {12, 4, 3},   {16, 4, 4},   {18, 6, 3},
                                 {24, 6, 4},   {27, 9, 3},   {32, 8, 4},   {36, 6, 6},   {48, 8, 6},
                                 {54, 9, 6},   {64, 8, 8},   {72, 9, 8},   {81, 9, 9},   {96, 12, 8},
                                 {108, 12, 9}, {128, 16, 8}, {144, 12, 12}};
    for (const auto& r : tab)
        if (r[0] == phi) {
            *A = r[1];
            *B = r[2];
            return true;
        }
    return false;
}

// Strides of the per-ring working set, in complex entries: one transform in
// pass layout (slot), one (ring, pair) unit, one ring.  The transform passes
// put the rows or columns of several transforms of a unit in one wave's
// lanes; a slot stride of 8 (mod 16) entries starts neighbouring transforms
// 16 four-byte banks apart, so their accesses overlap on fewer banks than
// with the stride of 1 (mod 16) that suits the MFMA operand reads alone.
// Per grid (a model of the passes' bank conflicts, each entry checked by
// measurement): 12 (no padding) for 144 points, 9 for 81 and 108; the 24-
// and 54-point grids keep 1, since there the larger padding costs their
// blocks half their pairs per work-group at the LDS budget.  Units are 2
// and rings 1 (mod 16) entries apart.  (fp32; fp64 plans use the same
// strides.)
#ifndef CGTP_PAD
#define CGTP_PAD 1
#endif
__host__ __device__ constexpr int slot_mod(int A, int B) {
    return (A * B == 24 || A * B == 54) ? 1 : A * B == 144 ? 12 : (A * B == 81 || A * B == 108) ? 9 : 8;
}
__host__ __device__ constexpr int slot_stride(int A, int B) {
    return CGTP_PAD ? A * (B + 1) + ((slot_mod(A, B) - A * (B + 1)) & 15) : A * (B + 1);
}
// Row strides of the lifted coefficients ([pair][slot][row], complex) and of
// the Legendre values ([ring][input][row], real), which the first synthesis
// pass reads for several transforms at once: a row of Phi entries padded per
// grid (from the same bank-conflict model, checked by measurement) so that
// power-of-two and other multiple-of-16 lengths do not start every row on the
// same bank.
__host__ __device__ constexpr int cv_mod(int phi) {
    return phi == 96 ? 12 : phi == 72 ? 9 : (phi == 64 || phi == 48) ? 8 : phi == 36 ? 3 : -1;
}
__host__ __device__ constexpr int pr_mod(int phi) {
    return phi == 128 ? 16 : (phi == 96 || phi == 72) ? 2 : (phi == 64 || phi == 48 || phi == 36) ? 8
         : phi == 54 ? 9 : phi == 144 ? 1 : -1;
}
__host__ __device__ constexpr int cv_stride(int phi) {
    return cv_mod(phi) < 0 ? phi : phi + ((cv_mod(phi) - phi) & 15);
}
__host__ __device__ constexpr int pr_stride(int phi) {
    return pr_mod(phi) < 0 ? phi : phi + ((pr_mod(phi) - phi) & 31);
}
__host__ __device__ constexpr int unit_stride(int nslot, int fs) {
    return CGTP_PAD ? nslot * fs + ((2 - nslot * fs) & 15) : nslot * fs;
}
__host__ __device__ constexpr int ring_stride(int pairs, int per_rp) {
    return CGTP_PAD ? pairs * per_rp + ((1 - pairs * per_rp) & 15) : pairs * per_rp + 8;
}

// Channel-wise launches with a shared second input synthesise it once per
// ring into a buffer of its own: half the transforms of a unit, per ring of
// the ring group (complex entries).
__host__ __device__ constexpr int x2buf_entries(int nslot, int fs, int rings) { return rings * (nslot / 2) * fs; }

// End phase: MFMA tile u of a block is dumped at u * tile_stride<T>() elements;
// the padding keeps consecutive tiles on different LDS banks.
template <typename T> __host__ __device__ constexpr int tile_stride() { return sizeof(T) == 4 ? 260 : 258; }

// Accumulator geometry shared by host and device.
struct TileGeom {
    int nrows;   // rows l3 = d, d+2, ..., J
    int ncomp;   // projected components (1 scalar, 4 scalar + vector)
    int pairs;
    __host__ __device__ int tmin(int mp, int d) const { return mp > d ? (mp - d + 1) / 2 : 0; }
    __host__ __device__ int rows(int mp, int d) const { return nrows - tmin(mp, d); }
    __host__ __device__ int ncols(int mp) const { return (mp == 0 ? 1 : 2) * ncomp * pairs; }
    __host__ __device__ int nrt(int mp, int d) const { return (rows(mp, d) + 15) / 16; }
    __host__ __device__ int nct(int mp) const { return (ncols(mp) + 15) / 16; }
};

// ---------------------------------------------------------------- gradients
//
// The gradient kernel (cgtp_backward.hip) runs one work-group per (block,
// tile of pairs), in two sizes: 256 threads and kBwdSmallPairs pairs for
// blocks with (2 J + 1) * components <= kBwdSmallThreads, 768 threads and
// kBwdLargePairs pairs for the others.  The transposed Legendre projection
// runs on 16x16x4 MFMA per |m|: wave w owns |m| = w, w + waves, ..., and holds
// the gradients of those accumulator entries in registers as B operands
// (lane: column lane % 16 = (pair, sign, component); with ks = ceil(rows / 4)
// K steps, step s takes row ks * (lane / 16) + s, so a lane's rows are
// consecutive).  LDS, in
// byte offsets: couplings [3][n1 + n2], twiddles in pass layout, the pair's
// lifted coefficients and their gradients ([pair][slot][Phi] each), then per
// ring group the Legendre values [ring][input][Phi] and kBwdSlots transforms
// per (ring, pair).
constexpr int kBwdThreads = 768;         // large blocks
constexpr int kBwdSmallThreads = 256;    // small blocks
constexpr int kBwdSmallLds = 52 * 1024;  // small blocks: ring groups sized for three work-groups per CU
constexpr int kBwdSmallPairs = 2;        // small blocks: pairs per work-group (a cross block's 8 columns each)
constexpr int kBwdLargePairs = 2;        // large blocks: pairs per work-group
constexpr int kBwdSlots = 8;   // 4 lifts, 2 analysis gradients, 2 product gradients
constexpr int kBwdMaxRings = 16;   // rings per group: the 16 rows of the transposed projection's MFMA tile
// Register budget of the B operands: |m| values per wave (mpw) and, for the
// t-th of them (|m| >= waves * t), K steps of 4 rows.  A block's |m| has at
// most floor((J - |m|) / 2) + 1 <= rmax - floor(|m| / 2) rows (rmax = Jmax / 2
// + 1), so the t-th needs at most ceil((rmax - waves * t / 2) / 4) steps.
template <typename T, bool SMALL> struct BwdGeom;
template <> struct BwdGeom<float, false> { static constexpr int mpw = 6, rmax = 33; };   // J <= 64
template <> struct BwdGeom<float, true> { static constexpr int mpw = 9, rmax = 17; };    // J <= 32
template <> struct BwdGeom<double, false> { static constexpr int mpw = 4, rmax = 20; };  // J <= 38
template <> struct BwdGeom<double, true> { static constexpr int mpw = 9, rmax = 17; };
template <typename T, bool SMALL>
__host__ __device__ constexpr int bwd_ks(int t) {
    const int nw = (SMALL ? kBwdSmallThreads : kBwdThreads) / 64;
    const int rows = BwdGeom<T, SMALL>::rmax - nw * t / 2;
    return rows < 1 ? 1 : (rows + 3) / 4;
}
struct BwdLayout {
    int lc, tw2, cvn, cacc, prs, fbuf, end;
};
__host__ __device__ inline int bwd_columns(const BlockDesc& b) {
    return (2 * b.J + 1) * (b.kind == kBlockCross ? 4 : 1);
}
__host__ __device__ inline bool bwd_small(const BlockDesc& b) { return bwd_columns(b) <= kBwdSmallThreads; }
__host__ __device__ inline int bwd_align16(int v) { return (v + 15) & ~15; }
__host__ __device__ inline BwdLayout bwd_layout(const BlockDesc& b, int esz, int rings, int pairs) {
    const int csz = 2 * esz;
    const bool cross = b.kind == kBlockCross;
    const int nslot = cross ? 4 : 2;
    const int n1 = 2 * b.j1 + 1, n2 = 2 * b.j2 + 1;
    BwdLayout l;
    int o = 0;
    l.lc = o; o = bwd_align16(o + esz * 3 * (n1 + n2));
    l.tw2 = o; o = bwd_align16(o + csz * b.A * (b.B + 1));
    l.cvn = o; o = bwd_align16(o + csz * pairs * nslot * b.Phi);
    l.cacc = o; o = bwd_align16(o + csz * pairs * nslot * b.Phi);
    l.prs = o; o = bwd_align16(o + esz * rings * 2 * b.Phi);
    l.fbuf = o; o += csz * rings * pairs * kBwdSlots * slot_stride(b.A, b.B);
    l.end = o;
    return l;
}
// Whether a block fits its variant's B-operand registers.
template <typename T>
inline bool bwd_fits(const BlockDesc& b) {
    const bool small = bwd_small(b);
    const int nw = (small ? kBwdSmallThreads : kBwdThreads) / 64;
    const int mpw = small ? BwdGeom<T, true>::mpw : BwdGeom<T, false>::mpw;
    if (b.J + 1 > mpw * nw) return false;
    const int nrows = (b.J - b.d) / 2 + 1;
    for (int mp = 0; mp <= b.J; ++mp) {
        const int rows = nrows - (mp > b.d ? (mp - b.d + 1) / 2 : 0);
        const int ks = small ? bwd_ks<T, true>(mp / nw) : bwd_ks<T, false>(mp / nw);
        if (rows > 4 * ks) return false;
    }
    return true;
}

// Offset (elements per pair) of block (j1, j2)'s gradient rows in the
// workspace: blocks in (j1, j2) order, each [pair][n1 + n2].
__host__ __device__ inline int64_t bwd_block_off(int L, int j1, int j2) {
    const int64_t M = L + 1;
    return M * j1 * j1 + (int64_t)j1 * M * M + (int64_t)(2 * j1 + 1) * j2 + (int64_t)j2 * j2;
}

// Records the HIP code behind a CGTP_EHIP status (cgtp_last_hip_error reads it).
void set_last_hip_error(int code);

// Launches the block kernel over the whole map; returns a hipError_t value.
// Multiplicity channels and path weights of a launch.  The N rows of x1 and
// out are (pair, channel) rows, channel fastest.  x2 holds one row per row of
// x1, or with kX2Shared one row per pair (row r / channels).  With w set, path
// (l1, l2, l3) of row r is scaled by w[k * npaths + path], k = r
// (kWeightsPerRow) or r mod channels.
enum ChanFlags : int32_t { kX2Shared = 1, kWeightsPerRow = 2 };
template <typename T>
struct ChanArgs {
    const T* w;        // NULL: unweighted
    int32_t channels;  // >= 1
    int32_t flags;     // ChanFlags
    int32_t npaths;
};

int launch_blocks_f32(const Tables<float>& tb, const int32_t* block_list, const LaunchMap& map,
                      int lds_bytes, const float* x1, const float* x2, float* out, int64_t N,
                      int L, void* stream);
int launch_blocks_f64(const Tables<double>& tb, const int32_t* block_list, const LaunchMap& map,
                      int lds_bytes, const double* x1, const double* x2, double* out, int64_t N,
                      int L, void* stream);
int launch_blocks_channels_f32(const Tables<float>& tb, const int32_t* block_list, const LaunchMap& map,
                               int lds_bytes, const float* x1, const float* x2, float* out, int64_t N,
                               int L, const ChanArgs<float>& ch, void* stream);
int launch_blocks_channels_f64(const Tables<double>& tb, const int32_t* block_list, const LaunchMap& map,
                               int lds_bytes, const double* x1, const double* x2, double* out, int64_t N,
                               int L, const ChanArgs<double>& ch, void* stream);

// Real basis: the block kernel with real-basis rows in and out
// (cgtp_kernels_real.hip), tables coefr / coefir for the end phase.
int launch_blocks_real_f32(const Tables<float>& tb, const int32_t* block_list, const LaunchMap& map,
                           int lds_bytes, const float* x1, const float* x2, float* out, int64_t N,
                           int L, void* stream);
int launch_blocks_real_f64(const Tables<double>& tb, const int32_t* block_list, const LaunchMap& map,
                           int lds_bytes, const double* x1, const double* x2, double* out, int64_t N,
                           int L, void* stream);

// Gradients: the per-block kernels (block_list: the nsmall small-variant
// blocks, then the nlarge others) over their blocks x N pairs into ws, then
// the sums over the other degree into gx1 / gx2 (either may be NULL).
struct BwdLaunch {
    const int32_t* block_list;
    int32_t nsmall, nlarge;
    int32_t lds_small, lds_large;
};
int launch_backward_f32(const Tables<float>& tb, const BwdLaunch& bl, const float* x1, const float* x2,
                        const float* g, float* gx1, float* gx2, float* ws, int64_t N, int L, void* stream);
int launch_backward_f64(const Tables<double>& tb, const BwdLaunch& bl, const double* x1, const double* x2,
                        const double* g, double* gx1, double* gx2, double* ws, int64_t N, int L, void* stream);

}  // namespace cgtp

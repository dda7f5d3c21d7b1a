// Internal layout shared by the host plan (istp_plan.cpp) and the kernel
// (istp_kernels.hip) of the multiple-input, multiple-output irrep-signal
// tensor products.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace istp {

constexpr int kThreads = 1024;   // work-group size (16 wave64s, one work-group per CU)
constexpr int kWaves = kThreads / 64;
constexpr int kLdsBudget = 160 * 1024;   // all of a gfx950 CU's LDS (one work-group per CU)
constexpr int kMaxLiftSteps = 9;   // K = 4 lift steps whose weights a wave loads at once

// Projection accumulator tiles (16 x 16) a wave may hold, per precision.
template <typename T> struct MaxTiles;
template <> struct MaxTiles<float> { static constexpr int value = 13; };
template <> struct MaxTiles<double> { static constexpr int value = 4; };
// Spin 2 holds its products' ten components in registers: at most 7 tiles a
// wave (its projections need at most 98 tiles, L <= 20).
template <typename T>
__host__ __device__ constexpr int max_tiles(int S) {
    return S == 2 && MaxTiles<T>::value > 7 ? 7 : MaxTiles<T>::value;
}

// One product: a first input of degree <= L and a second of degree <= L2
// lifted to spin-S signals, the pointwise product projected on degrees <= Lo
// (the forward product: L2 = L, Lo = 2 L).
//
// Grid: n_theta = 2 R Gauss-Legendre rings (R north rings, the south ones
// their mirror images), Phi = A * B equispaced longitudes.  A work-group takes
// `pairs` pairs through `G` north/south ring pairs at a time.
//
// Per ring pair and pair, every signal (input i, spin component c) is one
// complex transform carrying the north ring in its real and the south ring in
// its imaginary part; the C product components are packed the same way.
enum IstpFlags : int32_t {
    kReverseSecond = 1,   // the second input enters time-reversed: x[(j,l), m] -> (-1)^(m+j-l+S) x[(j,l), -m]
    kNegate = 2,          // outputs are negated
    kRealBasis = 4,       // rows in the real basis (spin 0 and 1, their own kernel: launch_istp_real_*)
};
struct alignas(16) IstpDesc {
    int32_t L, L2, Lo, spin, C;  // input degree bounds, output bound, spin, C = 2 spin + 1 components
    int32_t R, G, Phi, A, B;     // rings, ring pairs per group (a multiple of 4), longitudes = A * B
    int32_t pairs, nin, nin2, nout;   // pairs per work-group, values per input row (first, second), output row
    int32_t n_lift, n_proj;      // lift / projection MFMA tiles
    int32_t acoef_len;           // elements of the lift coefficient operand in LDS
    int32_t hc_len;              // elements of the end-phase spectra of one pair
    int32_t lw_len, pw_len;      // elements of the lift / projection weight tables
    int32_t wrow;                // projection weight entries per ring (row tiles * 16)
    int32_t lds_bytes;
    int32_t n_bcol;              // columns of the lift coefficient operand over all orders
    int32_t flags;               // IstpFlags
};

// Lift tile: spectra of order +-am of 16 rows (ring, l - am parity; rings
// 8 rb .. 8 rb + 7 of the group) x 16 columns (sign of m, input, component,
// pair) over K = l - am.
//   acoef: LDS element offset of (am, k = 0, column 16 ct) in the coefficient operand
//   cstride: elements per k row of that operand
//   lw: offset of (am, ring 0, k = 0) in the lift weights; kp entries per ring
//   ncol: valid columns of the order (all tiles of it); steps: K / 4
struct alignas(16) LiftTile {
    int32_t am, ct, acoef, cstride, lw, kp, ncol, steps, rb;
};

// Projection tile: rows l3 = am + par + 2 (16 rt + i), K = rings, columns
// (sign of m, component, pair); its weights start at `a` (ring 0, row 16 rt).
struct alignas(16) ProjTile {
    int32_t am, par, rt, a;
};

// Device tables, one allocation per plan.
template <typename T>
struct IstpTables {
    const T* lw;          // [am][ring < rpad][k < kp(am)]: P_{am+k}^{am}(x_ring), zero past max(L, L2) or R
    const T* pw;          // [am][par][ring < rpad][row < wrow]: w_ring P_{am+par+2 row}^{am}(x_ring), zero past Lo or R
    const T* tw;          // [t < A][k2 < B + 1]: exp(-2 pi i t k2 / Phi), pass layout
    const T* liftcg;      // [l][j - l + s][q + s][ml + l]: C^{j, ml+q}_{l, ml, s, q} (spin s > 0), l <= max(L, L2)
    const T* coef;        // per output: term weights, 4 (spin 0, 1: three terms and a pad) or 8 (spin 2: five terms)
    const int32_t* coefi; // per output: end-phase spectrum index of each term (pair 0), as coef
    const LiftTile* lift;
    const ProjTile* proj;
    const int2* bcol;     // per operand column: (am | column << 8, element offset of (am, k = 0, column))
    const IstpDesc* desc;
    const int32_t* lab;   // label index of every column: input 1 [nin], input 2 [nin2], output [nout]
};

// Multiplicity channels and label weights of a launch (the channel-wise
// kernels only).  Rows of x1 and out are (pair, channel), channel fastest; x2
// has one row per row, or with kChanX2Shared one per pair (row / channels).
// Weight rows k = the row (kChanPerRow) or its channel: w1[k nl1 + label] scales
// input 1, w2[k nl2 + label] input 2, wo[k nlo + label] the output; NULL: 1.
enum IstpChanFlags : int32_t { kChanX2Shared = 1, kChanPerRow = 2 };
template <typename T>
struct IstpChan {
    const T* w1;
    const T* w2;
    const T* wo;
    int32_t channels, flags;
    int32_t nl1, nl2, nlo;
};

// LDS of one work-group (byte offsets): twiddles at 0; one packed word per
// projection tile (ptab); the lift coefficient operand; then G * P (ring pair, pair) units of 2 C transforms each, `unit`
// complex entries apart (kUnitSkew entries of padding spread the units over
// the banks).  Before the first lift the tile's input rows and the lift
// couplings are staged at the units (stage_len elements).  The end phase puts
// the spectra of every pair at `hc`, over the coefficient operand and the units.
constexpr int kUnitSkew = 8;
constexpr int kStageLoads = 18;         // staged elements per thread (one batch of loads)
struct IstpLayout {
    int ptab, acoef, fbuf, hc;   // byte offsets
    int unit;              // complex entries per unit
    int bytes;             // total
};
__host__ __device__ inline int istp_align16(int v) { return (v + 15) & ~15; }
// staged elements: both inputs of every pair (rounded to 4), then C^{j,ml+q}_{l,ml,s,q}
// up to the larger input degree Lm (spin s > 0)
__host__ __device__ inline int istp_stage_x(int P, int nin, int nin2) { return (P * (nin + nin2) + 3) & ~3; }
__host__ __device__ inline int istp_stage_len(int P, int nin, int nin2, int Lm, int spin) {
    return istp_stage_x(P, nin, nin2) + (spin ? (2 * spin + 1) * (2 * spin + 1) * (Lm + 1) * (Lm + 1) : 0);
}
template <typename T>
__host__ __device__ inline IstpLayout istp_layout(int A, int B, int C, int G, int P, int acoef_len, int hc_len,
                                                  int stage_len, int n_proj) {
    const int FS = A * (B + 1), cs = 2 * (int)sizeof(T);
    IstpLayout l;
    l.unit = 2 * C * FS + kUnitSkew;
    l.ptab = istp_align16(FS * cs);
    l.acoef = istp_align16(l.ptab + 4 * n_proj);
    l.fbuf = istp_align16(l.acoef + acoef_len * (int)sizeof(T));
    l.hc = l.acoef;
    const int main_end = l.fbuf + G * P * l.unit * cs;
    const int end_end = l.hc + P * hc_len * (int)sizeof(T);
    const int stage_end = l.fbuf + stage_len * (int)sizeof(T);
    l.bytes = main_end > end_end ? main_end : end_end;
    if (stage_end > l.bytes) l.bytes = stage_end;
    return l;
}

// Lift coefficient operand: k rows of an order am are `cstride` elements apart,
// 16 per column tile.  (Padding the stride to an odd number of 16-element
// halves would keep rows k and k + 1 of one MFMA operand on opposite bank
// halves, but the space it takes costs more pairs per work-group than the
// conflicts it saves.)
__host__ __device__ inline int istp_cstride(int ncol) {
    const int nct = (ncol + 15) / 16;
    return 16 * nct;
}

int launch_istp_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2, float* out,
                    int64_t N, void* stream);
int launch_istp_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                    double* out, int64_t N, void* stream);
int launch_real_to_complex_f32(const float* r, float* re, float* im, float* sum, int64_t rows, int nin,
                               void* stream);
int launch_real_to_complex_f64(const double* r, double* re, double* im, double* sum, int64_t rows, int nin,
                               void* stream);
int launch_real_from_complex_f32(float* out, const float* pbb, const float* pss, int64_t rows, int Lo,
                                 void* stream);
int launch_real_from_complex_f64(double* out, const double* pbb, const double* pss, int64_t rows, int Lo,
                                 void* stream);
int launch_real_to_complex_spin_f32(const float* r, float* re, float* im, float* sum, int64_t rows, int nin, int s,
                                    void* stream);
int launch_real_to_complex_spin_f64(const double* r, double* re, double* im, double* sum, int64_t rows, int nin,
                                    int s, void* stream);
int launch_real_from_complex_spin_f32(float* out, const float* paa, const float* pbb, const float* pss,
                                      int64_t rows, int nout, int s, void* stream);
int launch_real_from_complex_spin_f64(double* out, const double* paa, const double* pbb, const double* pss,
                                      int64_t rows, int nout, int s, void* stream);
int launch_istp_real_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2,
                         float* out, int64_t N, void* stream);
int launch_istp_real_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                         double* out, int64_t N, void* stream);
int launch_istp_tensor_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2,
                           float* out, int64_t N, void* stream);
int launch_istp_tensor_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                           double* out, int64_t N, void* stream);
int launch_istp_channels_tensor_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1,
                                    const float* x2, float* out, int64_t N, const IstpChan<float>& ch,
                                    void* stream);
int launch_istp_channels_tensor_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1,
                                    const double* x2, double* out, int64_t N, const IstpChan<double>& ch,
                                    void* stream);
int launch_istp_channels_f32(const IstpTables<float>& tb, const IstpDesc& d, const float* x1, const float* x2,
                             float* out, int64_t N, const IstpChan<float>& ch, void* stream);
int launch_istp_channels_f64(const IstpTables<double>& tb, const IstpDesc& d, const double* x1, const double* x2,
                             double* out, int64_t N, const IstpChan<double>& ch, void* stream);

}  // namespace istp

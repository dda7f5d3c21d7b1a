// Device helpers shared by the kernels of this library: complex arithmetic,
// small in-register DFTs with compile-time twiddles, raw buffer loads, the
// 16x16x4 MFMA and its accumulator layout, and LDS ordering primitives.
// Internal; included by the .hip sources only.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace cgtp {
namespace dev {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Cplx;
template <> struct Cplx<float> { using type = float2; using acc4 = f32x4; };
template <> struct Cplx<double> { using type = double2; using acc4 = f64x4; };

template <typename C> __device__ __forceinline__ C cmk(decltype(C::x) x, decltype(C::x) y) { C r; r.x = x; r.y = y; return r; }
template <typename C> __device__ __forceinline__ C cmul(C a, C b) {
    return cmk<C>(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
template <typename C> __device__ __forceinline__ C cmulc(C a, C b) {   // a * conj(b)
    return cmk<C>(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}
template <typename C> __device__ __forceinline__ C cadd(C a, C b) { return cmk<C>(a.x + b.x, a.y + b.y); }
template <typename C> __device__ __forceinline__ C csub(C a, C b) { return cmk<C>(a.x - b.x, a.y - b.y); }
template <typename C> __device__ __forceinline__ C cconj(C a) { return cmk<C>(a.x, -a.y); }
// multiply by -i (forward) or +i (inverse)
template <bool INV, typename C> __device__ __forceinline__ C mul_mi(C a) {
    return INV ? cmk<C>(-a.y, a.x) : cmk<C>(a.y, -a.x);
}

// ---------------------------------------------------------------- twiddle constants

constexpr double kPiD = 3.14159265358979323846264338327950288;
constexpr double csin_series(double x) {
    double t = x, s = x;
    for (int k = 1; k < 30; ++k) { t *= -x * x / ((2.0 * k) * (2.0 * k + 1)); s += t; }
    return s;
}
constexpr double ccos_series(double x) {
    double t = 1, s = 1;
    for (int k = 1; k < 30; ++k) { t *= -x * x / ((2.0 * k - 1) * (2.0 * k)); s += t; }
    return s;
}
// exp(-2 pi i e / N) for e < N, evaluated at compile time.
template <int N> struct TwTab {
    double re[N > 0 ? N : 1], im[N > 0 ? N : 1];
    constexpr TwTab() : re(), im() {
        for (int e = 0; e < N; ++e) {
            double a = 2.0 * kPiD * e / N;
            if (a > kPiD) a -= 2.0 * kPiD;
            re[e] = ccos_series(a);
            im[e] = -csin_series(a);
        }
    }
};
template <int N> inline constexpr TwTab<N> kTw{};

template <int N, bool INV, typename C> __device__ __forceinline__ C twiddle_c(C v, int e) {
    using T = decltype(C::x);
    const T wr = (T)kTw<N>.re[e];
    const T wi = INV ? (T)-kTw<N>.im[e] : (T)kTw<N>.im[e];
    if (e == 0) return v;
    return cmk<C>(v.x * wr - v.y * wi, v.x * wi + v.y * wr);
}

// ---------------------------------------------------------------- small DFTs in registers
// Natural-order DFT of x[0..N-1]; forward uses exp(-2 pi i / N).

template <int N, bool INV, typename C> struct Dft;

template <bool INV, typename C> struct Dft<1, INV, C> { __device__ static void run(C*) {} };

template <bool INV, typename C> struct Dft<2, INV, C> {
    __device__ __forceinline__ static void run(C* x) {
        const C a = x[0], b = x[1];
        x[0] = cadd(a, b);
        x[1] = csub(a, b);
    }
};

template <bool INV, typename C> struct Dft<3, INV, C> {
    __device__ __forceinline__ static void run(C* x) {
        using T = decltype(C::x);
        const T h = (T)0.86602540378443864676372317075294;   // sqrt(3)/2
        const C a = x[0], t1 = cadd(x[1], x[2]), t2 = csub(x[1], x[2]);
        const C m = cmk<C>(a.x - (T)0.5 * t1.x, a.y - (T)0.5 * t1.y);
        const C r = mul_mi<INV>(cmk<C>(h * t2.x, h * t2.y));
        x[0] = cadd(a, t1);
        x[1] = cadd(m, r);
        x[2] = csub(m, r);
    }
};

template <bool INV, typename C> struct Dft<4, INV, C> {
    __device__ __forceinline__ static void run(C* x) {
        const C s0 = cadd(x[0], x[2]), s1 = csub(x[0], x[2]);
        const C s2 = cadd(x[1], x[3]), s3 = mul_mi<INV>(csub(x[1], x[3]));
        x[0] = cadd(s0, s2);
        x[2] = csub(s0, s2);
        x[1] = cadd(s1, s3);
        x[3] = csub(s1, s3);
    }
};

// Cooley-Tukey in registers: N1 inner transforms of length N2 over stride-N1
// elements, twiddles exp(-+2 pi i n1 k2 / N), then N2 transforms of length N1.
template <int N1, int N2, bool INV, typename C> __device__ __forceinline__ void dft_ct(C* x) {
    constexpr int N = N1 * N2;
    C y[N];
#pragma unroll
    for (int n1 = 0; n1 < N1; ++n1) {
        C v[N2];
#pragma unroll
        for (int n2 = 0; n2 < N2; ++n2) v[n2] = x[n1 + N1 * n2];
        Dft<N2, INV, C>::run(v);
#pragma unroll
        for (int k2 = 0; k2 < N2; ++k2) y[n1 * N2 + k2] = twiddle_c<N, INV>(v[k2], n1 * k2);
    }
#pragma unroll
    for (int k2 = 0; k2 < N2; ++k2) {
        C v[N1];
#pragma unroll
        for (int n1 = 0; n1 < N1; ++n1) v[n1] = y[n1 * N2 + k2];
        Dft<N1, INV, C>::run(v);
#pragma unroll
        for (int k1 = 0; k1 < N1; ++k1) x[k2 + N2 * k1] = v[k1];
    }
}

template <bool INV, typename C> struct Dft<6, INV, C> { __device__ static void run(C* x) { dft_ct<2, 3, INV>(x); } };
template <bool INV, typename C> struct Dft<8, INV, C> { __device__ static void run(C* x) { dft_ct<2, 4, INV>(x); } };
template <bool INV, typename C> struct Dft<9, INV, C> { __device__ static void run(C* x) { dft_ct<3, 3, INV>(x); } };
template <bool INV, typename C> struct Dft<12, INV, C> { __device__ static void run(C* x) { dft_ct<4, 3, INV>(x); } };
template <bool INV, typename C> struct Dft<16, INV, C> { __device__ static void run(C* x) { dft_ct<4, 4, INV>(x); } };

// ---------------------------------------------------------------- buffer loads

// Fourth dword of a raw buffer resource on gfx9-family GPUs (32-bit data format).
constexpr int kBufferFlags = 0x00020000;

template <typename T> __device__ __forceinline__ T buffer_load(__amdgpu_buffer_rsrc_t r, int voff, int soff);
template <> __device__ __forceinline__ float buffer_load<float>(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
template <> __device__ __forceinline__ double buffer_load<double>(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

// The first `cnt` (<= N) elements from byte offset voff of a buffer in
// 16-byte loads (elements past cnt up to the last load's end are loaded too;
// the rest of out is zero).  Offsets need element alignment only.  Each load
// is reinterpreted as a whole vector of elements before any element is taken
// out: taking 32-bit words out of the loaded vector and reinterpreting them
// one by one has been seen to compile into a single-word load whose value is
// copied to all four elements.
typedef double f64x2 __attribute__((ext_vector_type(2)));
template <int N>
__device__ __forceinline__ void load_run(__amdgpu_buffer_rsrc_t r, int voff, int cnt, float (&out)[N]) {
#pragma unroll
    for (int c = 0; c < (N + 3) / 4; ++c) {
        f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
        if (4 * c < cnt) v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff + 16 * c, 0, 0));
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (4 * c + e < N) out[4 * c + e] = v[e];
    }
}
template <int N>
__device__ __forceinline__ void load_run(__amdgpu_buffer_rsrc_t r, int voff, int cnt, double (&out)[N]) {
#pragma unroll
    for (int c = 0; c < (N + 1) / 2; ++c) {
        f64x2 v = {0.0, 0.0};
        if (2 * c < cnt) v = __builtin_bit_cast(f64x2, __builtin_amdgcn_raw_buffer_load_b128(r, voff + 16 * c, 0, 0));
        out[2 * c] = v[0];
        if (2 * c + 1 < N) out[2 * c + 1] = v[1];
    }
}

// ---------------------------------------------------------------- MFMA

__device__ __forceinline__ f32x4 mfma16(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f64x4 mfma16(double a, double b, f64x4 c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// Row of accumulator element q held by a lane in quarter rq = lane / 16 (the
// column is lane % 16).  The two 16x16x4 instructions lay their results out
// differently: f32 keeps four consecutive rows per lane, f64 strides by four.
template <typename T> __device__ __forceinline__ int acc_row(int rq, int q);
template <> __device__ __forceinline__ int acc_row<float>(int rq, int q) { return 4 * rq + q; }
template <> __device__ __forceinline__ int acc_row<double>(int rq, int q) { return rq + 4 * q; }

__device__ __forceinline__ int64_t rfl64(int64_t v) {
    const int lo = __builtin_amdgcn_readfirstlane((int)(v & 0xffffffff));
    const int hi = __builtin_amdgcn_readfirstlane((int)(v >> 32));
    return ((int64_t)hi << 32) | (uint32_t)lo;
}

// Orders a wave's own LDS accesses: every store issued before is complete and
// visible to the wave's later loads (no other wave is involved).
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Work-group barrier for LDS only.  The waves of this library's kernels never
// exchange data through global memory (they read inputs and tables and write
// disjoint outputs), so a barrier need not wait for outstanding global loads
// and stores: output stores drain and weight prefetches land across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

}  // namespace dev
}  // namespace cgtp

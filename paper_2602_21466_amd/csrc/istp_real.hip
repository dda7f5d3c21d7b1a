// Real spherical-harmonic basis for the signal products: conversion of
// real-basis rows to the real and imaginary parts of their complex-basis
// coefficients, and of the three products of those parts back to the real
// basis.  With the Condon-Shortley phase carried over from Y_l^m,
//   Y^R_{l,m} = sqrt(2) (-1)^m Re Y_l^m (m > 0), Y_l^0 (m = 0),
//               sqrt(2) (-1)^m Im Y_l^|m| (m < 0),
// a real function sum r_lm Y^R_lm has complex coefficients
//   c_{l,m} = (-1)^m (r_{l,m} - i r_{l,-m}) / sqrt 2,  c_{l,-m} = (r_{l,m} + i r_{l,-m}) / sqrt 2  (m > 0),
//   c_{l,0} = r_{l,0},
// and a real function's real-basis coefficients are read back as
//   r_{l,m} = sqrt 2 Re c_{l,-m},  r_{l,-m} = sqrt 2 Im c_{l,-m}  (m > 0),  r_{l,0} = Re c_{l,0}.
// The product of the complex coefficients is bilinear with real weights, so
// for c = a + i b, with three products (Karatsuba's form):
//   Re c3 = P(a1, a2) - P(b1, b2),  Im c3 = P(a1 + b1, a2 + b2) - P(a1, a2) - P(b1, b2).

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "../../include/istp.h"
#include "cgtp_internal.h"
#include "istp_internal.h"

namespace istp {
namespace {

constexpr int kConvThreads = 256;

__device__ __forceinline__ int degree_of(int c) {   // c = l^2 + l + m
    int l = (int)sqrtf((float)c);
    while ((l + 1) * (l + 1) <= c) ++l;
    while (l * l > c) --l;
    return l;
}

// One thread per (row, column): real and imaginary parts of c at that column, and their sum.
template <typename T>
__global__ __launch_bounds__(kConvThreads) void to_complex_kernel(const T* __restrict__ r, T* __restrict__ re,
                                                                  T* __restrict__ im, T* __restrict__ sum,
                                                                  int64_t total, int nin) {
    const int64_t e = (int64_t)blockIdx.x * kConvThreads + threadIdx.x;
    if (e >= total) return;
    const int64_t row = e / nin;
    const int c = (int)(e - row * nin), l = degree_of(c), m = c - l * l - l;
    const T* rr = r + row * nin + l * l + l;   // rr[m] = r_{l,m}
    const T s = (T)0.707106781186547524400844362104849039;
    T a, b;
    if (m == 0) {
        a = rr[0];
        b = (T)0;
    } else if (m > 0) {
        const T sg = (m & 1) ? -s : s;
        a = sg * rr[m];
        b = -sg * rr[-m];
    } else {
        a = s * rr[-m];
        b = s * rr[m];
    }
    re[e] = a;
    im[e] = b;
    sum[e] = a + b;
}

// One thread per (row, l, k >= 0) of the output: reads the three products at
// column (l, -k) and writes the real-basis values at (l, k) and (l, -k).  out
// holds P(a1, a2) on entry (read and written by the same thread only).
template <typename T>
__global__ __launch_bounds__(kConvThreads) void from_complex_kernel(T* __restrict__ out, const T* __restrict__ pbb,
                                                                    const T* __restrict__ pss, int64_t total,
                                                                    int Lo) {
    const int64_t e = (int64_t)blockIdx.x * kConvThreads + threadIdx.x;
    if (e >= total) return;
    const int per_row = (Lo + 1) * (Lo + 2) / 2, nout = (Lo + 1) * (Lo + 1);
    const int64_t row = e / per_row;
    const int t = (int)(e - row * per_row);   // t = l (l + 1) / 2 + k
    int l = (int)((sqrtf(8.0f * (float)t + 1.0f) - 1.0f) * 0.5f);
    while ((l + 1) * (l + 2) / 2 <= t) ++l;
    while (l * (l + 1) / 2 > t) --l;
    const int k = t - l * (l + 1) / 2;
    const int64_t base = row * nout + l * l + l;
    const T s = (T)1.41421356237309504880168872420969808;
    const T paa = out[base - k], pb = pbb[base - k];
    const T re = paa - pb;
    if (k == 0) {
        out[base] = re;
    } else {
        const T imv = pss[base - k] - paa - pb;
        out[base + k] = s * re;
        out[base - k] = s * imv;
    }
}

// ---- spin 1 and 2.  A real spin-s field sum c^(j,l)_m Y^{l,s}_{j,m} has
// c^(j,l)_{-m} = sigma (-1)^m conj(c^(j,l)_m), sigma = (-1)^(l+s-j): a label
// with sigma = +1 takes the scalar real basis above, one with sigma = -1 takes
// it for i c.  The spin-1 product of two real fields is i times a real field;
// it is read back after a factor i (spin 2 needs none).

// Column c of a spin-s row -> degree l, label j, order m (labels by l, then j
// from |l - s|; degree l starts at (2 s + 1) l^2, label j of it at j^2 - (l - s)^2).
__device__ __forceinline__ void spin_decode(int c, int s, int& l, int& j, int& m) {
    const int w = 2 * s + 1;
    l = (int)sqrtf((float)c / (float)w);
    while ((l + 1) * (l + 1) * w <= c) ++l;
    while (l * l * w > c) --l;
    const int e = c - w * l * l, ls = (l - s) * (l - s);
    j = (int)sqrtf((float)(e + ls));
    while ((j + 1) * (j + 1) - ls <= e) ++j;
    while (j * j - ls > e) --j;
    m = e - (j * j - ls) - j;
}

// One thread per (row, column): the label's real and imaginary parts at that
// column (with the label's phase), and their sum.
template <typename T>
__global__ __launch_bounds__(kConvThreads) void to_complex_spin_kernel(const T* __restrict__ r, T* __restrict__ re,
                                                                       T* __restrict__ im, T* __restrict__ sum,
                                                                       int64_t total, int nin, int s) {
    const int64_t e = (int64_t)blockIdx.x * kConvThreads + threadIdx.x;
    if (e >= total) return;
    const int64_t row = e / nin;
    const int c = (int)(e - row * nin);
    int l, j, m;
    spin_decode(c, s, l, j, m);
    const T* rr = r + row * nin + (c - m);   // rr[m] = r^(j,l)_m
    const T h = (T)0.707106781186547524400844362104849039;
    T a, b;
    if (m == 0) {
        a = rr[0];
        b = (T)0;
    } else if (m > 0) {
        const T sg = (m & 1) ? -h : h;
        a = sg * rr[m];
        b = -sg * rr[-m];
    } else {
        a = h * rr[-m];
        b = h * rr[m];
    }
    if ((l + s - j) & 1) {   // sigma = -1: c = -i (a + i b)
        const T t = a;
        a = b;
        b = -t;
    }
    re[e] = a;
    im[e] = b;
    sum[e] = a + b;
}

// One thread per (row, output column): the three products at the label's
// order -|m| give c_{-|m|} = (paa - pbb) + i (pss - paa - pbb); the label's
// phase (and the spin-1 factor i) applied, the column's real-basis value.
template <typename T>
__global__ __launch_bounds__(kConvThreads) void from_complex_spin_kernel(T* __restrict__ out,
                                                                         const T* __restrict__ paa,
                                                                         const T* __restrict__ pbb,
                                                                         const T* __restrict__ pss, int64_t total,
                                                                         int nout, int s) {
    const int64_t e = (int64_t)blockIdx.x * kConvThreads + threadIdx.x;
    if (e >= total) return;
    const int64_t row = e / nout;
    const int c = (int)(e - row * nout);
    int l, j, m;
    spin_decode(c, s, l, j, m);
    const int mu = m < 0 ? -m : m;
    const int64_t at = row * nout + (c - m) - mu;
    const T A = paa[at], Bv = pbb[at];
    T re = A - Bv, im = pss[at] - A - Bv;
    // quarter turns: sigma = -1 and the spin-1 factor each multiply by i
    const int turns = (((l + s - j) & 1) ? 1 : 0) + (s == 1 ? 1 : 0);
    for (int k = 0; k < turns; ++k) {
        const T t = re;
        re = -im;
        im = t;
    }
    const T r2 = (T)1.41421356237309504880168872420969808;
    out[e] = m == 0 ? re : (m > 0 ? r2 * re : r2 * im);
}

template <typename T>
int launch_to_complex_spin(const T* r, T* re, T* im, T* sum, int64_t rows, int nin, int s, void* stream) {
    const int64_t total = rows * nin;
    if (total <= 0) return 0;
    const int64_t grid = (total + kConvThreads - 1) / kConvThreads;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(to_complex_spin_kernel<T>, dim3((unsigned)grid), dim3(kConvThreads), 0, (hipStream_t)stream,
                       r, re, im, sum, total, nin, s);
    return (int)hipGetLastError();
}

template <typename T>
int launch_from_complex_spin(T* out, const T* paa, const T* pbb, const T* pss, int64_t rows, int nout, int s,
                             void* stream) {
    const int64_t total = rows * nout;
    if (total <= 0) return 0;
    const int64_t grid = (total + kConvThreads - 1) / kConvThreads;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(from_complex_spin_kernel<T>, dim3((unsigned)grid), dim3(kConvThreads), 0, (hipStream_t)stream,
                       out, paa, pbb, pss, total, nout, s);
    return (int)hipGetLastError();
}

template <typename T>
int launch_to_complex(const T* r, T* re, T* im, T* sum, int64_t rows, int nin, void* stream) {
    const int64_t total = rows * nin;
    if (total <= 0) return 0;
    const int64_t grid = (total + kConvThreads - 1) / kConvThreads;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(to_complex_kernel<T>, dim3((unsigned)grid), dim3(kConvThreads), 0, (hipStream_t)stream, r, re,
                       im, sum, total, nin);
    return (int)hipGetLastError();
}

template <typename T>
int launch_from_complex(T* out, const T* pbb, const T* pss, int64_t rows, int Lo, void* stream) {
    const int64_t total = rows * (int64_t)((Lo + 1) * (Lo + 2) / 2);
    if (total <= 0) return 0;
    const int64_t grid = (total + kConvThreads - 1) / kConvThreads;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(from_complex_kernel<T>, dim3((unsigned)grid), dim3(kConvThreads), 0, (hipStream_t)stream, out,
                       pbb, pss, total, Lo);
    return (int)hipGetLastError();
}

}  // namespace

int launch_real_to_complex_f32(const float* r, float* re, float* im, float* sum, int64_t rows, int nin,
                               void* stream) {
    return launch_to_complex<float>(r, re, im, sum, rows, nin, stream);
}
int launch_real_to_complex_f64(const double* r, double* re, double* im, double* sum, int64_t rows, int nin,
                               void* stream) {
    return launch_to_complex<double>(r, re, im, sum, rows, nin, stream);
}
int launch_real_from_complex_f32(float* out, const float* pbb, const float* pss, int64_t rows, int Lo,
                                 void* stream) {
    return launch_from_complex<float>(out, pbb, pss, rows, Lo, stream);
}
int launch_real_from_complex_f64(double* out, const double* pbb, const double* pss, int64_t rows, int Lo,
                                 void* stream) {
    return launch_from_complex<double>(out, pbb, pss, rows, Lo, stream);
}
int launch_real_to_complex_spin_f32(const float* r, float* re, float* im, float* sum, int64_t rows, int nin, int s,
                                    void* stream) {
    return launch_to_complex_spin<float>(r, re, im, sum, rows, nin, s, stream);
}
int launch_real_to_complex_spin_f64(const double* r, double* re, double* im, double* sum, int64_t rows, int nin,
                                    int s, void* stream) {
    return launch_to_complex_spin<double>(r, re, im, sum, rows, nin, s, stream);
}
int launch_real_from_complex_spin_f32(float* out, const float* paa, const float* pbb, const float* pss,
                                      int64_t rows, int nout, int s, void* stream) {
    return launch_from_complex_spin<float>(out, paa, pbb, pss, rows, nout, s, stream);
}
int launch_real_from_complex_spin_f64(double* out, const double* paa, const double* pbb, const double* pss,
                                      int64_t rows, int nout, int s, void* stream) {
    return launch_from_complex_spin<double>(out, paa, pbb, pss, rows, nout, s, stream);
}

}  // namespace istp

// ---------------------------------------------------------------- no-allocation entry point
//
// The workspace of istp_forward_real_static: one static array per device.  In
// host code the array's name is a host-side stand-in, not a device address;
// its device address is looked up once per device (with that device current)
// and only that address is ever passed to kernels.

namespace {

constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[ISTP_STATIC_SCRATCH_BYTES];
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array, or an error code.
int scratch_address(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        cgtp::set_last_hip_error((int)e);
        return CGTP_EHIP;
    }
    if (dev < 0 || dev >= kMaxDevices) return CGTP_EUNSUP;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            cgtp::set_last_hip_error((int)e);
            return CGTP_EHIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return CGTP_OK;
}

}  // namespace

extern "C" int istp_forward_real_static(istp_plan_t plan, const void* x1, const void* x2, void* out, int64_t N,
                                        void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (N == 0) return istp_forward_real(plan, x1, x2, out, 0, nullptr, 0, hip_stream);
    const int64_t need = istp_real_workspace_bytes(plan, N);
    if (need < 0) return istp_forward_real(plan, x1, x2, out, N, nullptr, 0, hip_stream);   // its own error
    if (need > ISTP_STATIC_SCRATCH_BYTES) return CGTP_ESCRATCH;
    void* ws = nullptr;
    const int rc = scratch_address(&ws);
    if (rc != CGTP_OK) return rc;
    return istp_forward_real(plan, x1, x2, out, N, ws, ISTP_STATIC_SCRATCH_BYTES, hip_stream);
}

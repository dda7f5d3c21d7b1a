// The full CGTP in the real spherical-harmonic basis: the basis changes around
// the complex-basis block kernel.
//
// A real function f = sum r_lm Y^R_lm, with the real harmonics
//   Y^R_{l,m} = sqrt(2) (-1)^m Re Y_l^m (m > 0), Y_l^0 (m = 0),
//               sqrt(2) (-1)^m Im Y_l^|m| (m < 0),
// has Hermitian complex coefficients c = a + i b:
//   c_0 = r_0,  c_m = (-1)^m (r_m - i r_-m) / sqrt(2),  c_-m = (r_m + i r_-m) / sqrt(2)   (m > 0).
// The CGTP is bilinear with real coefficients, so its value on c1, c2 is
// P(a1, a2) - P(b1, b2) + i (P(a1 + b1, a2 + b2) - P(a1, a2) - P(b1, b2)) with P
// the real-coefficient CGTP (three products, Karatsuba's form).  Path
// (l1, l2, l3) of two Hermitian inputs is Hermitian for even l1 + l2 + l3 and
// anti-Hermitian for odd; the odd ones are multiplied by i, and every path is
// read back in the real basis: r_0 = Re z_0, r_m = sqrt(2) Re z_-m,
// r_-m = sqrt(2) Im z_-m.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "cgtp_internal.h"

namespace cgtp {
namespace {

constexpr double kRsqrt2 = 0.70710678118654752440084436210485;
constexpr double kSqrt2 = 1.4142135623730950488016887242097;

// Real-basis rows -> (a, b, a + b) of their complex coefficients.  Thread per
// (input, pair, component).  xa[n] = a, xbc[n] = b, xbc[N + n] = a + b.
template <typename T>
__global__ __launch_bounds__(256) void real_in_kernel(const T* __restrict__ r1, const T* __restrict__ r2,
                                                      T* __restrict__ xa1, T* __restrict__ xbc1,
                                                      T* __restrict__ xa2, T* __restrict__ xbc2, int64_t N, int L) {
    const int nin = (L + 1) * (L + 1);
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= 2 * N * nin) return;
    const int which = (int)(e / (N * nin));
    const int64_t rest = e - (int64_t)which * N * nin;
    const int64_t n = rest / nin;
    const int i = (int)(rest - n * nin);
    int l = 0;
    while ((l + 1) * (l + 1) <= i) ++l;
    const int m = i - l * l - l, mu = m < 0 ? -m : m;
    const T* row = (which ? r2 : r1) + n * nin + l * l + l;
    T a, b;
    if (m == 0) {
        a = row[0];
        b = (T)0;
    } else {
        const T rp = row[mu] * (T)kRsqrt2, rm = row[-mu] * (T)kRsqrt2;
        if (m > 0) {
            const T s = (mu & 1) ? (T)-1 : (T)1;
            a = s * rp;
            b = -s * rm;
        } else {
            a = rp;
            b = rm;
        }
    }
    T* xa = which ? xa2 : xa1;
    T* xbc = which ? xbc2 : xbc1;
    xa[n * nin + i] = a;
    xbc[n * nin + i] = b;
    xbc[(N + n) * nin + i] = a + b;
}

// Products -> real basis, in place in out.  Thread per (pair, half-output
// entry); entry k of the table: index of m3 = 0 of its path in a pair's row
// (bits 0..20), |m3| (bits 21..27), odd path (bit 28).  out holds P(a1, a2),
// z[n] P(b1, b2), z[N + n] P(a1 + b1, a2 + b2).  The thread reads the three
// products at -|m3| and writes both +-|m3|.
template <typename T>
__global__ __launch_bounds__(256) void real_out_kernel(T* __restrict__ out, const T* __restrict__ z,
                                                       const int32_t* __restrict__ half, int64_t nhalf, int64_t N,
                                                       int64_t nout) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= N * nhalf) return;
    const int64_t n = e / nhalf;
    const int k = (int)(e - n * nhalf);
    const int code = half[k];
    const int base = code & 0x1fffff, mu = (code >> 21) & 0x7f;
    const bool odd = (code >> 28) & 1;
    T* orow = out + n * nout + base;
    const int64_t zo = n * nout + base - mu;
    const T A = orow[-mu], B = z[zo], Cc = z[N * nout + zo];
    T re = A - B, im = Cc - A - B;
    if (odd) {   // times i
        const T t = re;
        re = -im;
        im = t;
    }
    if (mu == 0) {
        orow[0] = re;
    } else {
        orow[mu] = (T)kSqrt2 * re;
        orow[-mu] = (T)kSqrt2 * im;
    }
}

template <typename T>
int launch_in(const T* r1, const T* r2, T* xa1, T* xbc1, T* xa2, T* xbc2, int64_t N, int L, void* stream) {
    const int64_t total = 2 * N * (int64_t)(L + 1) * (L + 1);
    const int64_t grid = (total + 255) / 256;
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(real_in_kernel<T>, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream, r1, r2, xa1, xbc1,
                       xa2, xbc2, N, L);
    return (int)hipGetLastError();
}

template <typename T>
int launch_out(T* out, const T* z, const int32_t* half, int64_t nhalf, int64_t N, int L, void* stream) {
    const int64_t nin = (int64_t)(L + 1) * (L + 1);
    const int64_t grid = (N * nhalf + 255) / 256;
    if (grid <= 0) return 0;
    if (grid > 0x7fffffffLL) return (int)hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(real_out_kernel<T>, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream, out, z, half,
                       nhalf, N, nin * nin);
    return (int)hipGetLastError();
}

}  // namespace

int launch_real_in_f32(const float* r1, const float* r2, float* xa1, float* xbc1, float* xa2, float* xbc2,
                       int64_t N, int L, void* stream) {
    return launch_in<float>(r1, r2, xa1, xbc1, xa2, xbc2, N, L, stream);
}
int launch_real_in_f64(const double* r1, const double* r2, double* xa1, double* xbc1, double* xa2, double* xbc2,
                       int64_t N, int L, void* stream) {
    return launch_in<double>(r1, r2, xa1, xbc1, xa2, xbc2, N, L, stream);
}
int launch_real_out_f32(float* out, const float* z, const int32_t* half, int64_t nhalf, int64_t N, int L,
                        void* stream) {
    return launch_out<float>(out, z, half, nhalf, N, L, stream);
}
int launch_real_out_f64(double* out, const double* z, const int32_t* half, int64_t nhalf, int64_t N, int L,
                        void* stream) {
    return launch_out<double>(out, z, half, nhalf, N, L, stream);
}

}  // namespace cgtp

// Sanitizer build of the plan sources: stand-ins for the HIP runtime calls the
// plans make and for the kernel launchers (no GPU, no device code).  The device
// is 0; every allocation fails, so a plan runs all of its host maths and table
// building and then returns CGTP_ENOMEM; every launch reports an error.
#include <hip/hip_runtime.h>

#include "../../paper_2602_21466_amd/csrc/cgtp_internal.h"
#include "../../paper_2602_21466_amd/csrc/istp_internal.h"

extern "C" {
hipError_t hipGetDevice(int* d) {
    *d = 0;
    return hipSuccess;
}
hipError_t hipMalloc(void** p, size_t) {
    *p = nullptr;
    return hipErrorOutOfMemory;
}
hipError_t hipFree(void*) { return hipSuccess; }
hipError_t hipMemcpy(void*, const void*, size_t, hipMemcpyKind) { return hipErrorInvalidValue; }
}

namespace cgtp {
int launch_blocks_f32(const Tables<float>&, const int32_t*, const LaunchMap&, int, const float*, const float*, float*,
                      int64_t, int, void*) { return 1; }
int launch_blocks_f64(const Tables<double>&, const int32_t*, const LaunchMap&, int, const double*, const double*,
                      double*, int64_t, int, void*) { return 1; }
int launch_blocks_channels_f32(const Tables<float>&, const int32_t*, const LaunchMap&, int, const float*,
                               const float*, float*, int64_t, int, const ChanArgs<float>&, void*) { return 1; }
int launch_blocks_channels_f64(const Tables<double>&, const int32_t*, const LaunchMap&, int, const double*,
                               const double*, double*, int64_t, int, const ChanArgs<double>&, void*) { return 1; }
int launch_blocks_real_f32(const Tables<float>&, const int32_t*, const LaunchMap&, int, const float*, const float*,
                           float*, int64_t, int, void*) { return 1; }
int launch_blocks_real_f64(const Tables<double>&, const int32_t*, const LaunchMap&, int, const double*,
                           const double*, double*, int64_t, int, void*) { return 1; }
int launch_backward_f32(const Tables<float>&, const BwdLaunch&, const float*, const float*, const float*, float*,
                        float*, float*, int64_t, int, void*) { return 1; }
int launch_backward_f64(const Tables<double>&, const BwdLaunch&, const double*, const double*, const double*,
                        double*, double*, double*, int64_t, int, void*) { return 1; }
}  // namespace cgtp

namespace istp {
int launch_istp_f32(const IstpTables<float>&, const IstpDesc&, const float*, const float*, float*, int64_t, void*) {
    return 1;
}
int launch_istp_f64(const IstpTables<double>&, const IstpDesc&, const double*, const double*, double*, int64_t,
                    void*) { return 1; }
int launch_real_to_complex_f32(const float*, float*, float*, float*, int64_t, int, void*) { return 1; }
int launch_real_to_complex_f64(const double*, double*, double*, double*, int64_t, int, void*) { return 1; }
int launch_real_from_complex_f32(float*, const float*, const float*, int64_t, int, void*) { return 1; }
int launch_real_from_complex_f64(double*, const double*, const double*, int64_t, int, void*) { return 1; }
int launch_real_to_complex_spin_f32(const float*, float*, float*, float*, int64_t, int, int, void*) { return 1; }
int launch_real_to_complex_spin_f64(const double*, double*, double*, double*, int64_t, int, int, void*) {
    return 1;
}
int launch_real_from_complex_spin_f32(float*, const float*, const float*, const float*, int64_t, int, int, void*) {
    return 1;
}
int launch_real_from_complex_spin_f64(double*, const double*, const double*, const double*, int64_t, int, int,
                                      void*) { return 1; }
int launch_istp_real_f32(const IstpTables<float>&, const IstpDesc&, const float*, const float*, float*, int64_t,
                         void*) { return 1; }
int launch_istp_real_f64(const IstpTables<double>&, const IstpDesc&, const double*, const double*, double*, int64_t,
                         void*) { return 1; }
int launch_istp_tensor_f32(const IstpTables<float>&, const IstpDesc&, const float*, const float*, float*, int64_t,
                           void*) { return 1; }
int launch_istp_tensor_f64(const IstpTables<double>&, const IstpDesc&, const double*, const double*, double*,
                           int64_t, void*) { return 1; }
int launch_istp_channels_tensor_f32(const IstpTables<float>&, const IstpDesc&, const float*, const float*, float*,
                                    int64_t, const IstpChan<float>&, void*) { return 1; }
int launch_istp_channels_tensor_f64(const IstpTables<double>&, const IstpDesc&, const double*, const double*,
                                    double*, int64_t, const IstpChan<double>&, void*) { return 1; }
int launch_istp_channels_f32(const IstpTables<float>&, const IstpDesc&, const float*, const float*, float*, int64_t,
                             const IstpChan<float>&, void*) { return 1; }
int launch_istp_channels_f64(const IstpTables<double>&, const IstpDesc&, const double*, const double*, double*,
                             int64_t, const IstpChan<double>&, void*) { return 1; }
}  // namespace istp

// The full CGTP in the real spherical-harmonic basis (block_kernel_real): the
// block body of cgtp_kernels.hip with real-basis rows in, the lifts and
// products of real signals, and real-basis outputs formed in the end phase.
#define CGTP_REAL_KERNELS 1
#include "cgtp_kernels.hip"

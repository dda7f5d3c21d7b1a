// The Gaunt product for rows in the real spherical-harmonic basis
// (istp_kernel_real) of istp_kernels.hip, in a translation unit of its own.
#define ISTP_REAL_KERNELS 1
#include "istp_kernels.hip"

// The channel-wise, label-weighted rank-2 tensor-harmonic signal-product
// kernel (spin 2) of istp_kernels.hip, in a translation unit of its own.
#define ISTP_CHANNEL_KERNELS 1
#define ISTP_TENSOR_KERNELS 1
#include "istp_kernels.hip"

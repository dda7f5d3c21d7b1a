// The channel-wise, path-weighted CGTP kernel (block_kernel_channels): the
// block body of cgtp_kernels.hip with multiplicity channels, a second input
// shared by the channels of a pair, and one weight per path, applied as the
// block is stored.
#define CGTP_CHANNEL_KERNELS 1
#include "cgtp_kernels.hip"

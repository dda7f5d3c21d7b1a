// The channel-wise, label-weighted signal-product kernels
// (istp_kernel_channels): the product of istp_kernels.hip with multiplicity
// channels, a second input shared by the channels of a pair, and one weight
// per (channel, irrep label) on each input and on the output, applied as the
// inputs are staged and as the outputs are stored.
#define ISTP_CHANNEL_KERNELS 1
#include "istp_kernels.hip"

// Host-only stand-in for <hip/hip_runtime.h> in the sanitizer build of the
// plan sources (g++, no device code): the runtime API declarations and empty
// function-space qualifiers.  Not used by the library build.
#pragma once
#include <hip/hip_runtime_api.h>
#define __host__
#define __device__
#define __global__
#define __forceinline__ inline

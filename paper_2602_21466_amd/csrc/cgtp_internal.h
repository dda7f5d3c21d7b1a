// Internal layout shared by the host plan (cgtp_plan.cpp) and the kernels
// (cgtp_kernels.hip).  Not part of the public ABI.
#pragma once

#include <cstdint>

namespace cgtp {

constexpr int kMaxRadix = 8;       // FFT stages per transform
constexpr int kThreads = 256;      // work-group size of the block kernel
constexpr int kLdsBudget = 64 * 1024;

// Product kinds per path (mirrors cgtp_path_norm's *kind).
enum PathKind : int32_t { kSS = 0, kCross = 1, kSV = 2, kDot = 3 };

// One (j1, j2) block: one irrep-signal tensor product on its own grid.
// Block kinds: which lifts/products the block needs.
enum BlockKind : int32_t {
    kBlockScalar = 0,   // only scalar-scalar paths (a degree-0 input)
    kBlockCross = 1,    // scalar-scalar (even paths) + cross (odd paths)
};

struct alignas(16) BlockDesc {
    int32_t j1, j2, J, d;      // d = |j1 - j2|
    int32_t R;                 // northern rings of the block's grid
    int32_t Phi;               // longitudes (FFT size)
    int32_t kind;              // BlockKind
    int32_t nrad;              // FFT stages
    int32_t rad[kMaxRadix];    // radices, first stage first
    int32_t tw_off;            // offset of the Phi-point twiddle table (complex entries)
    int32_t pbar_off;          // offset of the grid's Legendre table (elements)
    int32_t pbar_stride;       // Legendre entries per ring: (lmax+1)(lmax+2)/2
    int32_t wt_off;            // offset of the grid's ring weights
    int32_t kinv_off;          // offset of 1/K for j3 = d..J
    int32_t chunk;             // rings per pass through LDS
    int32_t pairs;             // pairs per work-group
    int32_t lds_bytes;         // dynamic LDS of one work-group
    int64_t out_off;           // offset of the block inside one pair's output
};

// Device tables, one allocation per plan; offsets in elements of T.
template <typename T>
struct Tables {
    const T* pbar;      // [grid][ring][l (l+1)/2 + m]
    const T* wt;        // [grid][ring]  2 * Gauss weight (north-south folding)
    const T* tw;        // complex pairs [Phi][2]: exp(-2 pi i k / Phi)
    const T* lcg;       // [j][q+1][m + j] = C^{j, m+q}_{j, m, 1, q}
    const T* rcg;       // [j3][q+1][m3 + j3] = C^{j3, m3}_{j3-1, m3-q, 1, q}
    const T* ccg;       // [q1+1][q2+1] = C^{1, q1+q2}_{1 q1 1 q2}
    const T* kinv;      // per block, j3 = d..J: 1 / K
    const BlockDesc* blocks;
};

// Blocks grouped by pairs-per-work-group.  One launch covers every class:
// work-groups [cum[c], cum[c+1]) belong to class c, ntiles[c] consecutive
// work-groups per block, heaviest classes first.
constexpr int kMaxClasses = 8;
struct LaunchMap {
    int32_t ncls;
    int32_t pairs[kMaxClasses];
    int32_t list_off[kMaxClasses];
    int64_t ntiles[kMaxClasses];
    int64_t cum[kMaxClasses + 1];
};

// Launches the block kernel over the whole map; returns a hipError_t value.
int launch_blocks_f32(const Tables<float>& tb, const int32_t* block_list, const LaunchMap& map,
                      int lds_bytes, const float* x1, const float* x2, float* out, int64_t N,
                      int L, void* stream);
int launch_blocks_f64(const Tables<double>& tb, const int32_t* block_list, const LaunchMap& map,
                      int lds_bytes, const double* x1, const double* x2, double* out, int64_t N,
                      int L, void* stream);

}  // namespace cgtp

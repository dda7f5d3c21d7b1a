// Host side of the CGTP library: the math the plan is built from, the plan
// itself (tables uploaded to device memory) and the C ABI entry points.
//
// Everything here runs once per plan and is not timed.  The device work is in
// cgtp_kernels.hip.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <map>
#include <new>
#include <vector>

#include "../../include/cgtp.h"
#include "cgtp_internal.h"

using cgtp::BlockDesc;

namespace {

thread_local int g_last_hip_error = 0;

// ------------------------------------------------------------------ factorials

constexpr int kFactMax = 700;

const long double* factorials() {
    static long double f[kFactMax + 1];
    static bool init = [] {
        f[0] = 1.0L;
        for (int i = 1; i <= kFactMax; ++i) f[i] = f[i - 1] * (long double)i;
        return true;
    }();
    (void)init;
    return f;
}

inline bool triangle(int a, int b, int c) {
    return a >= 0 && b >= 0 && c >= 0 && c >= std::abs(a - b) && c <= a + b;
}

// ------------------------------------------------------------------ Wigner symbols

// Triangle coefficient of a 6j symbol.
long double tri_delta(int a, int b, int c) {
    const long double* f = factorials();
    return sqrtl(f[a + b - c] * f[a - b + c] * f[-a + b + c] / f[a + b + c + 1]);
}

// Wigner 6j symbol {j1 j2 j3; j4 j5 j6} by Racah's single-sum formula.
long double sixj(int j1, int j2, int j3, int j4, int j5, int j6) {
    if (!triangle(j1, j2, j3) || !triangle(j1, j5, j6) || !triangle(j4, j2, j6) ||
        !triangle(j4, j5, j3))
        return 0.0L;
    const long double* f = factorials();
    const int a1 = j1 + j2 + j3, a2 = j1 + j5 + j6, a3 = j4 + j2 + j6, a4 = j4 + j5 + j3;
    const int b1 = j1 + j2 + j4 + j5, b2 = j2 + j3 + j5 + j6, b3 = j3 + j1 + j6 + j4;
    const int tmin = std::max(std::max(a1, a2), std::max(a3, a4));
    const int tmax = std::min(b1, std::min(b2, b3));
    long double s = 0.0L;
    for (int t = tmin; t <= tmax; ++t) {
        long double term = f[t + 1] / (f[t - a1] * f[t - a2] * f[t - a3] * f[t - a4] * f[b1 - t] *
                                       f[b2 - t] * f[b3 - t]);
        s += (t & 1) ? -term : term;
    }
    return s * tri_delta(j1, j2, j3) * tri_delta(j1, j5, j6) * tri_delta(j4, j2, j6) *
           tri_delta(j4, j5, j3);
}

// Wigner 9j symbol {a b c; d e f; g h i} as a sum over products of three 6j
// symbols (integer arguments only).
long double ninej(int a, int b, int c, int d, int e, int f, int g, int h, int i) {
    if (!triangle(a, b, c) || !triangle(d, e, f) || !triangle(g, h, i) || !triangle(a, d, g) ||
        !triangle(b, e, h) || !triangle(c, f, i))
        return 0.0L;
    int xmin = std::max(std::abs(a - i), std::max(std::abs(b - f), std::abs(d - h)));
    int xmax = std::min(a + i, std::min(b + f, d + h));
    long double s = 0.0L;
    for (int x = xmin; x <= xmax; ++x)
        s += (long double)(2 * x + 1) * sixj(a, b, c, f, i, x) * sixj(d, e, f, b, x, h) *
             sixj(g, h, i, x, a, d);
    return s;
}

// C^{j m}_{j1 m1 1 q}: closed forms of the coupling table with a vector.
long double cg_vec(int j1, int m1, int q, int j, int m) {
    if (j1 < 0 || j < 0 || q < -1 || q > 1) return 0.0L;
    if (m != m1 + q || std::abs(m1) > j1 || std::abs(m) > j) return 0.0L;
    if (!triangle(j1, 1, j)) return 0.0L;
    const long double J1 = j1, M = m;
    if (j == j1 + 1) {
        const long double den2 = (2 * J1 + 1) * (2 * J1 + 2);
        if (q == 1) return sqrtl((J1 + M) * (J1 + M + 1) / den2);
        if (q == 0) return sqrtl((J1 - M + 1) * (J1 + M + 1) / ((2 * J1 + 1) * (J1 + 1)));
        return sqrtl((J1 - M) * (J1 - M + 1) / den2);
    }
    if (j == j1) {
        const long double den = 2 * J1 * (J1 + 1);
        if (q == 1) return -sqrtl((J1 + M) * (J1 - M + 1) / den);
        if (q == 0) return M / sqrtl(J1 * (J1 + 1));
        return sqrtl((J1 - M) * (J1 + M + 1) / den);
    }
    // j == j1 - 1
    const long double den = 2 * J1 * (2 * J1 + 1);
    if (q == 1) return sqrtl((J1 - M) * (J1 - M + 1) / den);
    if (q == 0) return -sqrtl((J1 - M) * (J1 + M) / (J1 * (2 * J1 + 1)));
    return sqrtl((J1 + M + 1) * (J1 + M) / den);
}

// C^{l3 0}_{l1 0 l2 0} via the closed form of (l1 l2 l3; 0 0 0).
long double cg_zero(int l1, int l2, int l3) {
    if (!triangle(l1, l2, l3) || ((l1 + l2 + l3) & 1)) return 0.0L;
    const long double* f = factorials();
    const int g = (l1 + l2 + l3) / 2;
    long double w3 = sqrtl(f[2 * g - 2 * l1] * f[2 * g - 2 * l2] * f[2 * g - 2 * l3] / f[2 * g + 1]) *
                     f[g] / (f[g - l1] * f[g - l2] * f[g - l3]);
    if (g & 1) w3 = -w3;
    long double c = sqrtl((long double)(2 * l3 + 1)) * w3;
    return ((l1 - l2) & 1) ? -c : c;
}

const long double kPi = 3.141592653589793238462643383279502884L;

// Theorem 4.2's factor for lifts (j1, l1, s1), (j2, l2, s2) projected on
// (j3, l3, s3): raw = K * z.
long double gen_gaunt_K(int j1, int l1, int s1, int j2, int l2, int s2, int j3, int l3, int s3) {
    long double pre = sqrtl((long double)(2 * j1 + 1) * (2 * j2 + 1) * (2 * l1 + 1) * (2 * l2 + 1) *
                            (2 * s3 + 1) / (4.0L * kPi));
    return pre * ninej(j1, l1, s1, j2, l2, s2, j3, l3, s3) * cg_zero(l1, l2, l3);
}

// Accidental zeros of a cover's factor are replaced by a fallback product.
constexpr long double kMinAbsK = 1e-3L;

// Chooses the product for path (j1, j2, j3) and returns its K.
// Products the alternate cover uses in block (j1, j2), both inputs of degree
// >= 1: the dot product for even paths unless its factor vanishes by accident
// on one of the block's even paths, and scalar x1 times toroidal x2 for odd
// paths unless its factor vanishes on one of the odd paths.  A block that falls
// back uses the default product for all paths of that parity, so every block
// needs one product per parity.
void alt_block_products(int j1, int j2, bool* even_dot, bool* odd_sv) {
    *even_dot = true;
    *odd_sv = true;
    for (int j3 = std::abs(j1 - j2); j3 <= j1 + j2; ++j3) {
        if (((j1 + j2 + j3) & 1) == 0) {
            if (fabsl(gen_gaunt_K(j1, j1, 1, j2, j2, 1, j3, j3, 0)) < kMinAbsK) *even_dot = false;
        } else {
            if (fabsl(gen_gaunt_K(j1, j1, 0, j2, j2, 1, j3, j3 - 1, 1)) < kMinAbsK) *odd_sv = false;
        }
    }
}

int path_norm(int j1, int j2, int j3, int cover, long double* K, int* kind) {
    if (!triangle(j1, j2, j3)) return CGTP_EINVAL;
    const bool even = ((j1 + j2 + j3) & 1) == 0;
    const bool vec_ok = j1 > 0 && j2 > 0;  // a degree-0 input has no toroidal lift
    if (cover == CGTP_COVER_ALTERNATE && vec_ok) {
        bool even_dot, odd_sv;
        alt_block_products(j1, j2, &even_dot, &odd_sv);
        if (even && even_dot) {
            *K = gen_gaunt_K(j1, j1, 1, j2, j2, 1, j3, j3, 0);
            *kind = cgtp::kDot;
            return CGTP_OK;
        }
        if (!even && odd_sv) {
            *K = gen_gaunt_K(j1, j1, 0, j2, j2, 1, j3, j3 - 1, 1);
            *kind = cgtp::kSV;
            return CGTP_OK;
        }
    }
    if (even) {
        *K = gen_gaunt_K(j1, j1, 0, j2, j2, 0, j3, j3, 0);
        *kind = cgtp::kSS;
    } else {
        *K = gen_gaunt_K(j1, j1, 1, j2, j2, 1, j3, j3 - 1, 1);
        *kind = cgtp::kCross;
    }
    return CGTP_OK;
}

// ------------------------------------------------------------------ quadrature

void gauss_legendre(int n, std::vector<long double>& x, std::vector<long double>& w) {
    x.assign(n, 0.0L);
    w.assign(n, 0.0L);
    for (int i = 0; i < n; ++i) {
        long double z = cosl(kPi * (i + 0.75L) / (n + 0.5L));
        long double dp = 1.0L;
        for (int it = 0; it < 100; ++it) {
            long double p0 = 1.0L, p1 = z;
            for (int k = 2; k <= n; ++k) {
                long double p2 = ((2 * k - 1) * z * p1 - (k - 1) * p0) / k;
                p0 = p1;
                p1 = p2;
            }
            if (n == 1) { p1 = z; p0 = 1.0L; }
            dp = n * (z * p1 - p0) / (z * z - 1.0L);
            long double dz = p1 / dp;
            z -= dz;
            if (fabsl(dz) < 1e-19L) break;
        }
        // recompute the derivative at the converged node
        long double p0 = 1.0L, p1 = z;
        for (int k = 2; k <= n; ++k) {
            long double p2 = ((2 * k - 1) * z * p1 - (k - 1) * p0) / k;
            p0 = p1;
            p1 = p2;
        }
        dp = n * (z * p1 - p0) / (z * z - 1.0L);
        x[i] = z;
        w[i] = 2.0L / ((1.0L - z * z) * dp * dp);
    }
}

// Normalised P^m_l(x) with Condon-Shortley phase at out[l(l+1)/2 + m].
void legendre(int lmax, long double x, long double* out) {
    auto at = [&](int l, int m) -> long double& { return out[l * (l + 1) / 2 + m]; };
    const long double s = sqrtl(std::max(0.0L, 1.0L - x * x));
    at(0, 0) = 1.0L / sqrtl(4.0L * kPi);
    for (int m = 1; m <= lmax; ++m) at(m, m) = -sqrtl((2.0L * m + 1) / (2.0L * m)) * s * at(m - 1, m - 1);
    for (int m = 0; m < lmax; ++m) at(m + 1, m) = x * sqrtl(2.0L * m + 3) * at(m, m);
    for (int m = 0; m <= lmax; ++m)
        for (int l = m + 2; l <= lmax; ++l) {
            long double a = sqrtl((4.0L * l * l - 1) / ((long double)l * l - (long double)m * m));
            long double b = sqrtl(((long double)(l - 1) * (l - 1) - (long double)m * m) /
                                  (4.0L * (l - 1) * (l - 1) - 1));
            at(l, m) = a * (x * at(l - 1, m) - b * at(l - 2, m));
        }
}

// ------------------------------------------------------------------ grids

bool is_2a3b(int n) {
    if (n < 1) return false;
    while (n % 2 == 0) n /= 2;
    while (n % 3 == 0) n /= 3;
    return n == 1;
}

int smallest_2a3b(int n) {
    int m = std::max(n, 1);
    while (!is_2a3b(m)) ++m;
    return m;
}

constexpr int kMaxPhi = 144;

int check_grid(int L, const cgtp_grid* g) {
    if (g->dtype != CGTP_FP32 && g->dtype != CGTP_FP64) return CGTP_EDTYPE;
    if (g->cover != CGTP_COVER_DEFAULT && g->cover != CGTP_COVER_ALTERNATE) return CGTP_EINVAL;
    if (g->n_theta < 0 || g->n_phi < 0) return CGTP_EINVAL;
    if (g->n_theta > 0) {
        if (g->n_theta < 2 * L + 1) return CGTP_EGRID;
        if (g->n_theta & 1) return CGTP_EUNSUP;
        if (g->n_theta > 4 * CGTP_MAX_L + 64) return CGTP_EUNSUP;
    }
    if (g->n_phi > 0) {
        if (g->n_phi < 4 * L + 1) return CGTP_EGRID;
        int a, b;
        if (!cgtp::fft_factors(g->n_phi, &a, &b) || g->n_phi > kMaxPhi) return CGTP_EUNSUP;
    }
    return CGTP_OK;
}

void block_grid(const cgtp_grid& g, int j1, int j2, int* n_theta, int* n_phi) {
    const int J = j1 + j2;
    *n_theta = g.n_theta > 0 ? g.n_theta : 2 * (J / 2) + 2;
    *n_phi = g.n_phi > 0 ? g.n_phi : smallest_2a3b(2 * J + 1);
}

int64_t path_offset(int L, int l1, int l2, int l3) {
    if (L < 0 || l1 < 0 || l2 < 0 || l1 > L || l2 > L) return -1;
    if (l3 < std::abs(l1 - l2) || l3 > l1 + l2) return -1;
    return (int64_t)l1 * l1 * (L + 1) * (L + 1) + (int64_t)(2 * l1 + 1) * l2 * l2 + (int64_t)l3 * l3 -
           (int64_t)(l1 - l2) * (l1 - l2);
}

// Index of path (l1, l2, l3) when all paths of degree L are listed in (l1, l2,
// l3) order (block (a, b) holds the 2 min(a, b) + 1 paths l3 = |a - b|..a + b);
// -1 if it is not a path.  path_index(L, L + 1, 0, 1) is the number of paths.
int64_t path_index(int L, int l1, int l2, int l3) {
    const bool end = L >= 0 && l1 == L + 1 && l2 == 0 && l3 == 1;
    if (!end && path_offset(L, l1, l2, l3) < 0) return -1;
    int64_t k = 0;
    for (int a = 0; a < l1; ++a)
        for (int b = 0; b <= L; ++b) k += 2 * std::min(a, b) + 1;
    if (end) return k;
    for (int b = 0; b < l2; ++b) k += 2 * std::min(l1, b) + 1;
    return k + l3 - std::abs(l1 - l2);
}

// MFMA weight table geometry: rings padded to whole ring groups; entries per
// ring row (degrees l = par, par + 2, ..., <= lmax).
inline int wtab_rpad(int R) { return (R + cgtp::kRingGroup - 1) / cgtp::kRingGroup * cgtp::kRingGroup; }
inline int wtab_rowlen(int lmax, int par) { return lmax >= par ? (lmax - par) / 2 + 1 : 1; }

// Algorithmic flops of one block on its minimal exact grid (default cover),
// without the lifts: those are counted once per input, degree and grid by
// lift_flops, however many blocks of the grid use them.
double block_flops(int j1, int j2) {
    const int J = j1 + j2, d = std::abs(j1 - j2);
    const double R = J / 2 + 1, Phi = 2 * J + 1, H = J + 1;
    const double f = Phi > 1 ? 2.5 * Phi * std::log2(Phi) : 0.0;
    const bool vec = j1 > 0 && j2 > 0;
    const double nin = vec ? 4 : 1;
    double T = 0, rec = 0;
    for (int j3 = d; j3 <= J; ++j3) {
        if (((J + j3) & 1) == 0) { T += 2 * j3 + 1; rec += 2 * j3 + 1; }
        else { T += 3 * (2 * (j3 - 1) + 1); rec += 7 * (2 * j3 + 1); }
    }
    return R * H * (6 + (vec ? 60 : 0))          // pointwise products
         + nin * R * f                           // longitude analysis
         + 2 * R * T                             // Legendre projection
         + rec;                                  // recombination and 1/K
}

// Flops of a block's pointwise products (the products term of block_flops).
double block_product_flops(int j1, int j2) {
    const int J = j1 + j2;
    const double R = J / 2 + 1, H = J + 1;
    return R * H * (6 + ((j1 > 0 && j2 > 0) ? 60 : 0));
}

// Flops of lifting one input of degree j (nin series: 1 scalar, 4 scalar +
// vector) to a grid of R north rings that blocks up to degree Jmax share:
// latitude stage and longitude synthesis on the minimal exact longitudes
// 2 Jmax + 1.
double lift_flops(int j, int R, int Jmax, int nin) {
    const double Phi = 2 * Jmax + 1;
    const double f = Phi > 1 ? 2.5 * Phi * std::log2(Phi) : 0.0;
    return (double)R * (2 * j + 1) * nin + (double)nin * R * f;
}

}  // namespace

// ====================================================================== plan

struct cgtp_plan_s {
    int L = 0;
    cgtp_grid grid{};
    int device = 0;
    void* dmem = nullptr;      // all tables
    size_t dbytes = 0;
    cgtp::Tables<float> tf{};
    cgtp::Tables<double> td{};
    const int32_t* d_list = nullptr;   // block indices grouped by pairs-per-work-group
    struct Cls { int pairs; int off; int count; };
    std::vector<Cls> classes;
    int lds_bytes = 0;      // dynamic LDS of the plain kernel
    int lds_bytes_ch = 0;   // and of the channel kernel (with the shared second-input buffers)
    int bwd_lds_small = 0, bwd_lds_large = 0;   // dynamic LDS of the gradient kernel's two variants
    int bwd_nsmall = 0;     // blocks of the small variant: the first entries of the gradient block list
    int bwd_list_off = 0;   // the gradient block list's offset in the uploaded block lists
    const int32_t* d_bwd_list = nullptr;
    bool bwd_ok = true;     // every block fits one of the gradient kernel's variants
    int max_theta = 0, max_phi = 0;
    double min_abs_K = 0, flops_per_pair = 0, bytes_per_pair = 0;
    double bwd_flops_per_pair = 0;
    double cross_cg = 0, dot_cg = 0;
};

namespace {

template <typename T>
struct HostTables {
    std::vector<T> pbar, wtab, tw, lcg, coef, coefr;
    std::vector<int32_t> coefi, coefir;
    std::vector<cgtp::TileDesc> tdesc;
};

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int align16h(int v) { return (v + 15) & ~15; }

// Accumulator tiles of a block with the given pairs per work-group.
int block_tiles(const BlockDesc& b, int pairs) {
    const bool cross = b.kind == cgtp::kBlockCross;
    cgtp::TileGeom g{(b.J - b.d) / 2 + 1, cross ? 4 : 1, pairs};
    int n = 0;
    for (int mp = 0; mp <= b.J; ++mp) n += g.nrt(mp, b.d) * g.nct(mp);
    return n;
}

// Dynamic LDS of one work-group; mirrors the kernel's make_layout.
template <typename T>
int lds_for(const BlockDesc& b, int pairs, bool x2buf = false) {
    const int sz = (int)sizeof(T), csz = 2 * sz;
    const bool cross = b.kind == cgtp::kBlockCross;
    const int nslot = cross ? 4 : 2;
    const int n1 = 2 * b.j1 + 1, n2 = 2 * b.j2 + 1;
    const int FS = b.A * (b.B + 1);
    const int per_r = cgtp::ring_stride(pairs, cgtp::unit_stride(nslot, cgtp::slot_stride(b.A, b.B)));
    int o = 0;
    o = align16h(o + sz * 3 * (n1 + n2));
    o = align16h(o + sz * b.R * 2 * cgtp::pr_stride(b.Phi));
    o = align16h(o + csz * FS);
    o = align16h(o + 4 * block_tiles(b, pairs));
    o = align16h(o + csz * pairs * nslot * cgtp::cv_stride(b.Phi));
    if (x2buf) o = align16h(o + csz * cgtp::x2buf_entries(nslot, cgtp::slot_stride(b.A, b.B), cgtp::kRingGroup));
    const int fbuf = o;
    o += csz * cgtp::kRingGroup * per_r;
    const int end_phase = fbuf + sz * block_tiles(b, pairs) * cgtp::tile_stride<T>();
    return std::max(o, end_phase);
}

template <typename T>
int build(cgtp_plan_s* p, std::vector<BlockDesc>& blocks, HostTables<T>& h, std::vector<int32_t>& list) {
    const int L = p->L;
    const cgtp_grid& g = p->grid;
    // ---- grids: one Legendre table per distinct node count
    std::map<int, int> grid_lmax;          // n_theta -> largest degree needed
    std::map<int, int> grid_lmax_out;
    std::map<int, int> phi_set;            // Phi -> twiddle offset
    for (int j1 = 0; j1 <= L; ++j1)
        for (int j2 = 0; j2 <= L; ++j2) {
            int nt, np;
            block_grid(g, j1, j2, &nt, &np);
            grid_lmax[nt] = std::max(grid_lmax[nt], j1 + j2);
            phi_set[np] = 0;
        }
    std::map<int, int> grid_pbar_off, grid_wtab_off, grid_stride;
    std::map<int, std::array<int, 2>> grid_wtab_par;
    for (auto& kv : grid_lmax) {
        const int nt = kv.first, lmax = kv.second, R = nt / 2;
        std::vector<long double> x, w;
        gauss_legendre(nt, x, w);
        const int stride = (lmax + 1) * (lmax + 2) / 2;
        grid_pbar_off[nt] = (int)h.pbar.size();
        grid_wtab_off[nt] = (int)h.wtab.size();
        grid_stride[nt] = stride;
        std::vector<long double> rows((size_t)R * stride);
        for (int i = 0; i < R; ++i) {
            legendre(lmax, x[i], rows.data() + (size_t)i * stride);
            for (int e = 0; e < stride; ++e) h.pbar.push_back((T)rows[(size_t)i * stride + e]);
        }
        // MFMA weights, per parity of l: [m'][ring][t] = 2 w_r P^{m'}_l(x_r) for
        // l = par + 2t <= lmax (north and south folded; zero for l < m'), rings
        // padded with zeros to whole ring groups, so a tile's 16 rows are
        // contiguous; 16 zero entries close each parity.
        const int rpad = wtab_rpad(R);
        for (int par = 0; par < 2; ++par) {
            const int rl = wtab_rowlen(lmax, par);
            grid_wtab_par[nt][par] = (int)h.wtab.size() - grid_wtab_off[nt];
            for (int mp = 0; mp <= lmax; ++mp)
                for (int i = 0; i < rpad; ++i)
                    for (int t = 0; t < rl; ++t) {
                        const int l = par + 2 * t;
                        h.wtab.push_back((i < R && l >= mp && l <= lmax)
                                             ? (T)(2.0L * w[i] * rows[(size_t)i * stride + l * (l + 1) / 2 + mp])
                                             : (T)0);
                    }
            h.wtab.insert(h.wtab.end(), (size_t)16, (T)0);
        }
        p->max_theta = std::max(p->max_theta, nt);
    }
    for (auto& kv : phi_set) {
        const int n = kv.first;
        int A, B;
        if (!cgtp::fft_factors(n, &A, &B)) return CGTP_EUNSUP;
        kv.second = (int)(h.tw.size() / 2);
        // pass layout: [t < A][k2 < B + 1] = exp(-2 pi i t k2 / n), pad entry zero
        for (int t = 0; t < A; ++t)
            for (int k2 = 0; k2 <= B; ++k2) {
                const long double a = -2.0L * kPi * (long double)((t * k2) % n) / n;
                h.tw.push_back(k2 < B ? (T)cosl(a) : (T)0);
                h.tw.push_back(k2 < B ? (T)sinl(a) : (T)0);
            }
        p->max_phi = std::max(p->max_phi, n);
    }
    // ---- Clebsch-Gordan tables
    h.lcg.assign(3 * (size_t)(L + 1) * (L + 1), (T)0);
    for (int j = 0; j <= L; ++j)
        for (int q = -1; q <= 1; ++q)
            for (int m = -j; m <= j; ++m)
                h.lcg[3 * j * j + (q + 1) * (2 * j + 1) + m + j] = (T)cg_vec(j, m, q, j, m + q);
    // The kernel forms the cross product as c * (antisymmetric combination) with
    // c = C^{1,1}_{1,1,1,0}; check the coupling table has that structure.
    const long double c = cg_vec(1, 1, 0, 1, 1);
    for (int q1 = -1; q1 <= 1; ++q1)
        for (int q2 = -1; q2 <= 1; ++q2) {
            if (std::abs(q1 + q2) > 1) continue;
            const long double want = q1 == q2 ? 0.0L : (q1 > q2 ? c : -c);
            if (fabsl(cg_vec(1, q1, q2, 1, q1 + q2) - want) > 1e-15L) return CGTP_EINVAL;
        }
    p->cross_cg = (double)c;
    // the dot product as d * (a+ b- - a0 b0 + a- b+) with d = C^{0,0}_{1,1,1,-1}
    const long double dc = cg_vec(1, 1, -1, 0, 0);
    for (int q = -1; q <= 1; ++q)
        if (fabsl(cg_vec(1, q, -q, 0, 0) - (q == 0 ? -dc : dc)) > 1e-15L) return CGTP_EINVAL;
    p->dot_cg = (double)dc;
    // ---- blocks
    double min_abs_K = 1e300, flops = 0, bwd_extra = 0;
    // lifts: (input, degree, n_theta, Phi) -> (north rings, largest J of the grid, series)
    std::map<std::array<int, 4>, std::array<int, 3>> lifts;
    blocks.clear();
    for (int j1 = 0; j1 <= L; ++j1)
        for (int j2 = 0; j2 <= L; ++j2) {
            BlockDesc b{};
            b.j1 = j1; b.j2 = j2; b.J = j1 + j2; b.d = std::abs(j1 - j2);
            int nt, np;
            block_grid(g, j1, j2, &nt, &np);
            b.R = nt / 2;
            b.Phi = np;
            b.kind = (j1 > 0 && j2 > 0) ? cgtp::kBlockCross : cgtp::kBlockScalar;
            b.products = 0;
            if (b.kind == cgtp::kBlockCross && g.cover == CGTP_COVER_ALTERNATE) {
                bool even_dot, odd_sv;
                alt_block_products(j1, j2, &even_dot, &odd_sv);
                b.products = (even_dot ? cgtp::kEvenDot : 0) | (odd_sv ? cgtp::kOddSV : 0);
            }
            if (!cgtp::fft_factors(np, &b.A, &b.B)) return CGTP_EUNSUP;
            b.tw_off = phi_set[np];
            b.pbar_off = grid_pbar_off[nt];
            b.pbar_stride = grid_stride[nt];
            b.lmax = grid_lmax[nt];
            b.rpad = wtab_rpad(b.R);
            b.wrow = wtab_rowlen(b.lmax, b.J & 1);
            b.wtab_off = grid_wtab_off[nt] + grid_wtab_par[nt][b.J & 1];
            // 1/K of every path of the block (Theorem 4.2 for the cover's products)
            std::vector<long double> kinv(b.J + 1, 0.0L);
            for (int j3 = b.d; j3 <= b.J; ++j3) {
                long double K;
                int kind;
                if (path_norm(j1, j2, j3, g.cover, &K, &kind) != CGTP_OK) return CGTP_EINVAL;
                const bool odd = (b.J + j3) & 1;
                const int want = odd ? ((b.products & cgtp::kOddSV) ? cgtp::kSV : cgtp::kCross)
                                     : ((b.products & cgtp::kEvenDot) ? cgtp::kDot : cgtp::kSS);
                if (kind != want || fabsl(K) < kMinAbsK) return CGTP_EUNSUP;
                min_abs_K = std::min(min_abs_K, (double)fabsl(K));
                kinv[j3] = 1.0L / K;
            }
            b.out_off = path_offset(L, j1, j2, b.d);
            b.path_off = (int32_t)path_index(L, j1, j2, b.d);
            flops += block_flops(j1, j2);
            bwd_extra += block_product_flops(j1, j2);   // the products' adjoint yields both factors' gradients
            {
                const int nin = b.kind == cgtp::kBlockCross ? 4 : 1;
                for (int in = 0; in < 2; ++in) {
                    auto& e = lifts[std::array<int, 4>{in, in ? j2 : j1, nt, np}];
                    e[0] = b.R;
                    e[1] = std::max(e[1], b.J);
                    e[2] = std::max(e[2], nin);
                }
            }
            // pairs per work-group: as many as the accumulator registers and LDS allow
            const int max_tiles = cgtp::kWaves * cgtp::MaxTiles<T>::value;
            const int ncomp = b.kind == cgtp::kBlockCross ? 4 : 1;
            auto fits = [&](int P) {
                return block_tiles(b, P) <= max_tiles && lds_for<T>(b, P) <= cgtp::kLdsBudget;
            };
            int pairs = 0;
            for (int P = cgtp::kMaxPairs; P >= 1 && !pairs; P /= 2)
                if (fits(P)) pairs = P;
            if (pairs == 0) return CGTP_EUNSUP;
            b.pairs = pairs;
            b.lg_pairs = 0;
            while ((1 << b.lg_pairs) < pairs) ++b.lg_pairs;
            b.ntiles = block_tiles(b, pairs);
            b.lds_bytes = lds_for<T>(b, pairs);
            // the channel kernel's shared second-input buffer, where it fits
            const int lds_x2 = lds_for<T>(b, pairs, true);
            b.x2share = lds_x2 <= cgtp::kLdsBudget ? 1 : 0;
            p->lds_bytes_ch = std::max(p->lds_bytes_ch, b.x2share ? lds_x2 : b.lds_bytes);
            // gradient kernel: the largest ring group (kBwdMaxRings down to 1) whose LDS
            // fits, for small blocks within kBwdSmallLds where one does
            b.bwd_rings = 0;
            {
                const bool small = cgtp::bwd_small(b);
                const int bp = small ? cgtp::kBwdSmallPairs : cgtp::kBwdLargePairs;
                for (int pass = small ? 0 : 1; pass < 2 && !b.bwd_rings; ++pass)
                    for (int G = cgtp::kBwdMaxRings; G >= 1 && !b.bwd_rings; --G)
                        if (cgtp::bwd_layout(b, (int)sizeof(T), G, bp).end <=
                            (pass ? cgtp::kLdsBudget : cgtp::kBwdSmallLds))
                            b.bwd_rings = G;
                // the register-held entry gradients (B operands of the transposed projection)
                if (!cgtp::bwd_fits<T>(b)) b.bwd_rings = 0;
                if (b.bwd_rings) {
                    int& lds = small ? p->bwd_lds_small : p->bwd_lds_large;
                    lds = std::max(lds, cgtp::bwd_layout(b, (int)sizeof(T), b.bwd_rings, bp).end);
                }
            }
            if (b.bwd_rings == 0) p->bwd_ok = false;
            // MFMA tiles in the order the waves take them: by |m|, row tile, column tile
            b.tdesc_off = (int)h.tdesc.size();
            {
                cgtp::TileGeom geo{(b.J - b.d) / 2 + 1, ncomp, pairs};
                for (int mp = 0; mp <= b.J; ++mp)
                    for (int rt = 0; rt < geo.nrt(mp, b.d); ++rt)
                        for (int ct = 0; ct < geo.nct(mp); ++ct) {
                            const int row0 = geo.tmin(mp, b.d) + 16 * rt;
                            const int l30 = b.d + 2 * row0;
                            const int nv = std::min(16, geo.nrows - row0);
                            const int par = b.J & 1;
                            cgtp::TileDesc t;
                            t.a_off = mp * b.rpad * b.wrow + (l30 - par) / 2;
                            t.rs_nv = nv << 16;
                            // pass-layout positions k + k / B of longitudes +|m| and -|m|
                            const int kn = (b.Phi - mp) % b.Phi;
                            t.b_off = 2 * (mp + mp / b.B) | (2 * (kn + kn / b.B)) << 16;
                            t.code = (mp << 16) | (rt << 8) | ct;
                            h.tdesc.push_back(t);
                        }
            }
            // Output coefficients.  The end phase dumps MFMA tile u of the block
            // verbatim at u * kTileStride; entry (row r, column c) of a tile sits at
            // lane * 4 + q with the accumulator layout of the MFMA, and the columns of
            // the pairs of one (sign, component) are consecutive, so pair p adds 4 p.
            // Per output: up to three (weight, entry of pair 0) terms; the weights
            // carry 1/K, the recombination coefficient, the longitude quadrature and
            // unpacking scale, the product's coupling constant and (-1)^m for m < 0.
            b.coef_off = (int)(h.coef.size() / 4);
            {
                cgtp::TileGeom geo{(b.J - b.d) / 2 + 1, ncomp, pairs};
                const bool cross = b.kind == cgtp::kBlockCross;
                const long double sc_s = 2.0L * kPi / b.Phi * (cross ? 0.25L : 1.0L);
                // coupling constants C^{1,1}_{1,1,1,0} (cross) and C^{0,0}_{1,1,1,-1} (dot)
                const long double sc_v = sc_s * ((b.products & cgtp::kOddSV) ? 1.0L : cg_vec(1, 1, 0, 1, 1));
                const long double sc_e = sc_s * ((b.products & cgtp::kEvenDot) ? cg_vec(1, 1, -1, 0, 0) : 1.0L);
                // tile index of (|m|, row tile, column tile), in enumeration order
                std::vector<int> first_of_m(b.J + 2, 0);
                for (int mp = 0; mp <= b.J; ++mp)
                    first_of_m[mp + 1] = first_of_m[mp] + geo.nrt(mp, b.d) * geo.nct(mp);
                auto entry = [&](int comp, int m, int tr, long double* f) {
                    const int mp = std::abs(m), sg = m < 0 ? 1 : 0;
                    const int row = tr - geo.tmin(mp, b.d), rt = row / 16, r = row % 16;
                    const int col = sg * ncomp * pairs + comp * pairs, ct = col / 16, ci = col % 16;
                    const int u = first_of_m[mp] + rt * geo.nct(mp) + ct;
                    const int lin = sizeof(T) == 4 ? (ci + 16 * (r >> 2)) * 4 + (r & 3)
                                                   : (ci + 16 * (r & 3)) * 4 + (r >> 2);
                    *f = (comp == 0 ? sc_e : sc_v) * ((sg && (mp & 1)) ? -1.0L : 1.0L);
                    return u * cgtp::tile_stride<T>() + lin;
                };
                for (int j3 = b.d; j3 <= b.J; ++j3) {
                    const bool odd = (b.J + j3) & 1;
                    for (int m3 = -j3; m3 <= j3; ++m3) {
                        long double f;
                        if (!odd) {
                            const int e = entry(0, m3, (j3 - b.d) / 2, &f);
                            h.coef.push_back((T)(kinv[j3] * f));
                            h.coef.push_back((T)0);
                            h.coef.push_back((T)0);
                            h.coef.push_back((T)0);
                            h.coefi.insert(h.coefi.end(), {e, e, e, 1 | (j3 - b.d) << 1});
                        } else {
                            // q = -1, 0, +1 from components 2, 1, 3 at (j3 - 1, m3 - q)
                            const int l3 = j3 - 1, tr = (l3 - b.d) / 2;
                            const int comp_of_q[3] = {2, 1, 3};
                            long double w[3];
                            int e[3], valid = -1;
                            for (int k = 0; k < 3; ++k) {
                                const int q = k - 1, m = m3 - q;
                                w[k] = 0.0L;
                                e[k] = -1;
                                if (std::abs(m) <= l3) {
                                    e[k] = entry(comp_of_q[k], m, tr, &f);
                                    w[k] = kinv[j3] * cg_vec(l3, m, q, j3, m3) * f;
                                    valid = e[k];
                                }
                            }
                            for (int k = 0; k < 3; ++k) {
                                if (e[k] < 0) e[k] = valid;   // zero weight; any entry of the block
                                h.coef.push_back((T)w[k]);
                            }
                            h.coef.push_back((T)0);
                            h.coefi.insert(h.coefi.end(), {e[0], e[1], e[2], (j3 - b.d) << 1});
                        }
                    }
                }
                // The same outputs in the real basis (four terms each).  Blocks with
                // a degree-0 input scale the other input, the same in either basis:
                // their terms are the complex basis' ones.  Cross blocks: the
                // accumulators hold, per component c and order m, A_c[m] = the
                // projection of Re z1, Im z1, Re z2, Im z2 with P^|m|; with the true
                // P^m (sign (-1)^m for m < 0) they give Pi1[m] = A_0 + i A_1 and
                // Pi2[m] = A_2 + i A_3 per row.  z1 = gs + g0 and z2 = g+ with gs
                // real, g0 imaginary and g- = conj(g+) on the sphere, so per row
                //   Pi[gs][m] = (Pi1[m] + (-1)^m conj Pi1[-m]) / 2,
                //   Pi[g0][m] = (Pi1[m] - (-1)^m conj Pi1[-m]) / 2,
                //   Pi[g+][m] = Pi2[m],  Pi[g-][m] = (-1)^m conj Pi2[-m].
                // A path's complex output z (even: 1/K Pi[gs] at l3 = j3; odd: 1/K
                // sum over q of C^{j3 m3}_{j3-1, m3-q, 1, q} Pi[g_q] at j3 - 1) is
                // multiplied by i on odd paths and read in the real basis: r_0 =
                // Re z_0, r_mu = sqrt 2 Re z_-mu, r_-mu = sqrt 2 Im z_-mu.
                const size_t nr0 = h.coefr.size();
                if (!cross) {
                    for (size_t k = b.coef_off * (size_t)4; k < h.coef.size(); k += 4) {
                        h.coefr.insert(h.coefr.end(), {h.coef[k], (T)0, (T)0, (T)0});
                        const int32_t e0 = h.coefi[k];
                        h.coefir.insert(h.coefir.end(), {e0, e0, e0, e0});
                    }
                } else {
                    const long double sc_r = 2.0L * kPi / b.Phi;   // exact unpacking: no factor 1/4
                    const long double sr_e = sc_r * ((b.products & cgtp::kEvenDot) ? cg_vec(1, 1, -1, 0, 0) : 1.0L);
                    const long double sr_v = sc_r * ((b.products & cgtp::kOddSV) ? 1.0L : cg_vec(1, 1, 0, 1, 1));
                    // linear forms over accumulator entries (entry of pair 0 -> weight)
                    using Form = std::map<int, long double>;
                    auto put = [&](Form& f, int comp, int m, int tr, int l, long double w) {
                        if (std::abs(m) > l || w == 0.0L) return;
                        long double sg;
                        const int e = entry(comp, m, tr, &sg);
                        sg = (m < 0 && (std::abs(m) & 1)) ? -1.0L : 1.0L;
                        f[e] += w * sg;
                    };
                    auto par = [](int m) { return (std::abs(m) & 1) ? -1.0L : 1.0L; };
                    const long double rt2 = std::sqrt(2.0L);
                    for (int j3 = b.d; j3 <= b.J; ++j3) {
                        const bool odd = (b.J + j3) & 1;
                        const int l3 = odd ? j3 - 1 : j3, tr = (l3 - b.d) / 2;
                        for (int m3 = -j3; m3 <= j3; ++m3) {
                            const int M = -std::abs(m3);
                            Form zr, zi;   // Re z_M, Im z_M
                            if (!odd) {
                                const long double k = kinv[j3] * sr_e, s = par(M);
                                put(zr, 0, M, tr, l3, k / 2);
                                put(zr, 0, -M, tr, l3, k * s / 2);
                                put(zi, 1, M, tr, l3, k / 2);
                                put(zi, 1, -M, tr, l3, -k * s / 2);
                            } else {
                                for (int q = -1; q <= 1; ++q) {
                                    const int mq = M - q;
                                    if (std::abs(mq) > l3) continue;
                                    const long double c = kinv[j3] * sr_v * cg_vec(l3, mq, q, j3, M), s = par(mq);
                                    if (q == 0) {
                                        put(zr, 0, mq, tr, l3, c / 2);
                                        put(zr, 0, -mq, tr, l3, -c * s / 2);
                                        put(zi, 1, mq, tr, l3, c / 2);
                                        put(zi, 1, -mq, tr, l3, c * s / 2);
                                    } else if (q == 1) {
                                        put(zr, 2, mq, tr, l3, c);
                                        put(zi, 3, mq, tr, l3, c);
                                    } else {
                                        put(zr, 2, -mq, tr, l3, c * s);
                                        put(zi, 3, -mq, tr, l3, -c * s);
                                    }
                                }
                            }
                            // w = z (even) or i z (odd); output Re w (m3 >= 0) or Im w (m3 < 0)
                            const Form* f;
                            long double sgn = 1.0L;
                            if (!odd)
                                f = m3 < 0 ? &zi : &zr;
                            else if (m3 < 0)
                                f = &zr;   // Im(i z) = Re z
                            else {
                                f = &zi;   // Re(i z) = -Im z
                                sgn = -1.0L;
                            }
                            if (m3 != 0) sgn *= rt2;
                            T w[4] = {(T)0, (T)0, (T)0, (T)0};
                            int32_t ei[4] = {-1, -1, -1, -1};
                            int nt = 0;
                            for (const auto& kv : *f) {
                                if (kv.second == 0.0L) continue;
                                if (nt == 4) return CGTP_EUNSUP;   // cannot happen: at most four entries
                                w[nt] = (T)(sgn * kv.second);
                                ei[nt++] = kv.first;
                            }
                            long double unused;
                            const int32_t any = nt ? ei[0] : entry(0, 0, 0, &unused);
                            for (int k = 0; k < 4; ++k)
                                if (ei[k] < 0) ei[k] = any;   // zero weight; any entry of the block
                            h.coefr.insert(h.coefr.end(), {w[0], w[1], w[2], w[3]});
                            h.coefir.insert(h.coefir.end(), {ei[0], ei[1], ei[2], ei[3]});
                        }
                    }
                }
                if (h.coefr.size() - nr0 != h.coef.size() - (size_t)b.coef_off * 4) return CGTP_EUNSUP;
            }
            p->lds_bytes = std::max(p->lds_bytes, b.lds_bytes);
            blocks.push_back(b);
        }
    p->min_abs_K = min_abs_K;
    double lflops = 0;
    for (const auto& kv : lifts) lflops += lift_flops(kv.first[1], kv.second[0], kv.second[1], kv.second[2]);
    flops += lflops;
    p->flops_per_pair = flops;
    // gradients: the forward's work plus the adjoint's extra product term and
    // the transposed synthesis, which costs what the lift does
    p->bwd_flops_per_pair = flops + bwd_extra + lflops;
    p->bytes_per_pair = (double)sizeof(T) * (2.0 * (L + 1) * (L + 1) + std::pow((double)(L + 1), 4));
    // ---- launch classes: fewest pairs (heaviest blocks) first; inside, by cost
    std::map<int, std::vector<int>> by_pairs;
    for (int i = 0; i < (int)blocks.size(); ++i) by_pairs[blocks[i].pairs].push_back(i);
    list.clear();
    p->classes.clear();
    if ((int)by_pairs.size() > cgtp::kMaxClasses) return CGTP_EUNSUP;
    for (auto& kv : by_pairs) {
        auto& v = kv.second;
        std::stable_sort(v.begin(), v.end(), [&](int a, int b) {
            const BlockDesc &x = blocks[a], &y = blocks[b];
            return (double)x.R * x.Phi * (x.J + 1) > (double)y.R * y.Phi * (y.J + 1);
        });
        p->classes.push_back({kv.first, (int)list.size(), (int)v.size()});
        list.insert(list.end(), v.begin(), v.end());
    }
    // gradient kernel's block list, after the forward's: the small variant's
    // blocks, then the large variant's, each heaviest first
    p->bwd_list_off = (int)list.size();
    std::vector<int> bs, bl;
    for (int i = 0; i < (int)blocks.size(); ++i) (cgtp::bwd_small(blocks[i]) ? bs : bl).push_back(i);
    auto heavier = [&](int a, int b) {
        const BlockDesc &x = blocks[a], &y = blocks[b];
        return (double)x.R * x.Phi * (x.J + 1) > (double)y.R * y.Phi * (y.J + 1);
    };
    std::stable_sort(bs.begin(), bs.end(), heavier);
    std::stable_sort(bl.begin(), bl.end(), heavier);
    p->bwd_nsmall = (int)bs.size();
    list.insert(list.end(), bs.begin(), bs.end());
    list.insert(list.end(), bl.begin(), bl.end());
    return CGTP_OK;
}

template <typename T>
int upload(cgtp_plan_s* p, const std::vector<BlockDesc>& blocks, const HostTables<T>& h,
           const std::vector<int32_t>& list, cgtp::Tables<T>* tb) {
    const std::vector<T>* parts[] = {&h.pbar, &h.wtab, &h.tw, &h.lcg, &h.coef, &h.coefr};
    constexpr int kParts = 6;
    size_t offs[kParts + 2];
    size_t total = 0;
    for (int i = 0; i < kParts; ++i) {
        offs[i] = total;
        total = align_up(total + parts[i]->size() * sizeof(T), 256);
    }
    offs[kParts] = total;
    total = align_up(total + blocks.size() * sizeof(BlockDesc), 256);
    offs[kParts + 1] = total;
    total = align_up(total + list.size() * sizeof(int32_t), 256);
    const size_t tdesc_off = total;
    total = align_up(total + h.tdesc.size() * sizeof(cgtp::TileDesc), 256);
    const size_t coefi_off = total;
    total = align_up(total + h.coefi.size() * sizeof(int32_t), 256);
    const size_t coefir_off = total;
    total = align_up(total + h.coefir.size() * sizeof(int32_t), 256);
    std::vector<char> host(total, 0);
    if (!h.tdesc.empty())
        std::memcpy(host.data() + tdesc_off, h.tdesc.data(), h.tdesc.size() * sizeof(cgtp::TileDesc));
    if (!h.coefi.empty()) std::memcpy(host.data() + coefi_off, h.coefi.data(), h.coefi.size() * sizeof(int32_t));
    if (!h.coefir.empty())
        std::memcpy(host.data() + coefir_off, h.coefir.data(), h.coefir.size() * sizeof(int32_t));
    for (int i = 0; i < kParts; ++i)
        if (!parts[i]->empty()) std::memcpy(host.data() + offs[i], parts[i]->data(), parts[i]->size() * sizeof(T));
    std::memcpy(host.data() + offs[kParts], blocks.data(), blocks.size() * sizeof(BlockDesc));
    std::memcpy(host.data() + offs[kParts + 1], list.data(), list.size() * sizeof(int32_t));
    hipError_t e = hipMalloc(&p->dmem, total);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        p->dmem = nullptr;
        return e == hipErrorOutOfMemory ? CGTP_ENOMEM : CGTP_EHIP;
    }
    e = hipMemcpy(p->dmem, host.data(), total, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        (void)hipFree(p->dmem);
        p->dmem = nullptr;
        return CGTP_EHIP;
    }
    p->dbytes = total;
    char* base = (char*)p->dmem;
    tb->pbar = (const T*)(base + offs[0]);
    tb->wtab = (const T*)(base + offs[1]);
    tb->tw = (const T*)(base + offs[2]);
    tb->lcg = (const T*)(base + offs[3]);
    tb->coef = (const T*)(base + offs[4]);
    tb->coefi = (const int32_t*)(base + coefi_off);
    tb->coefr = (const T*)(base + offs[5]);
    tb->coefir = (const int32_t*)(base + coefir_off);
    tb->wtab_len = (int32_t)h.wtab.size();
    tb->blocks = (const BlockDesc*)(base + offs[kParts]);
    tb->tdesc = (const cgtp::TileDesc*)(base + tdesc_off);
    p->d_list = (const int32_t*)(base + offs[kParts + 1]);
    p->d_bwd_list = p->d_list + p->bwd_list_off;
    return CGTP_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char *pa = (const char*)a, *pb = (const char*)b;
    return pa < pb + nb && pb < pa + na;
}

}  // namespace

namespace cgtp {
void set_last_hip_error(int code) { g_last_hip_error = code; }
}  // namespace cgtp

// ====================================================================== C ABI

extern "C" {

const char* cgtp_strerror(int code) {
    switch (code) {
        case CGTP_OK: return "success";
        case CGTP_EINVAL: return "invalid argument";
        case CGTP_EGRID: return "grid too small for exact quadrature";
        case CGTP_EDTYPE: return "unknown dtype";
        case CGTP_ENOMEM: return "out of memory";
        case CGTP_EHIP: return "HIP runtime error";
        case CGTP_EUNSUP: return "unsupported by this build";
        case CGTP_ESCRATCH: return "request exceeds the static scratch of a no-allocation entry point";
        default: return "unknown status";
    }
}

int cgtp_last_hip_error(void) { return g_last_hip_error; }

int64_t cgtp_num_outputs(int32_t L) {
    if (L < 0) return -1;
    const int64_t a = (int64_t)(L + 1) * (L + 1);
    return a * a;
}

int64_t cgtp_path_offset(int32_t L, int32_t l1, int32_t l2, int32_t l3) { return path_offset(L, l1, l2, l3); }

int cgtp_path_norm(int32_t j1, int32_t j2, int32_t j3, int32_t cover, double* K, int32_t* kind) {
    if (cover != CGTP_COVER_DEFAULT && cover != CGTP_COVER_ALTERNATE) return CGTP_EINVAL;
    if (j1 > 4 * CGTP_MAX_L || j2 > 4 * CGTP_MAX_L) return CGTP_EUNSUP;
    long double k = 0;
    int kd = 0;
    int rc = path_norm(j1, j2, j3, cover, &k, &kd);
    if (rc != CGTP_OK) return rc;
    if (K) *K = (double)k;
    if (kind) *kind = kd;
    return CGTP_OK;
}

double cgtp_wigner_9j(int32_t a, int32_t b, int32_t c, int32_t d, int32_t e, int32_t f, int32_t g, int32_t h,
                      int32_t i) {
    if (a + b + c + d + e + f + g + h + i > kFactMax / 2) return NAN;
    return (double)ninej(a, b, c, d, e, f, g, h, i);
}

double cgtp_cg_vector(int32_t j1, int32_t m1, int32_t q, int32_t j, int32_t m) {
    return (double)cg_vec(j1, m1, q, j, m);
}

double cgtp_cg_zero(int32_t l1, int32_t l2, int32_t l3) {
    if (l1 + l2 + l3 > kFactMax / 2) return NAN;
    return (double)cg_zero(l1, l2, l3);
}

int cgtp_gauss_legendre(int32_t n, double* x, double* w) {
    if (n < 1 || n > 4096 || !x || !w) return CGTP_EINVAL;
    std::vector<long double> xs, ws;
    gauss_legendre(n, xs, ws);
    for (int i = 0; i < n; ++i) { x[i] = (double)xs[i]; w[i] = (double)ws[i]; }
    return CGTP_OK;
}

int cgtp_legendre(int32_t lmax, double x, double* out) {
    if (lmax < 0 || lmax > 4096 || !out || !(x >= -1.0 && x <= 1.0)) return CGTP_EINVAL;
    std::vector<long double> v((size_t)(lmax + 1) * (lmax + 2) / 2);
    legendre(lmax, x, v.data());
    for (size_t i = 0; i < v.size(); ++i) out[i] = (double)v[i];
    return CGTP_OK;
}

int cgtp_block_grid(int32_t L, const cgtp_grid* grid, int32_t l1, int32_t l2, int32_t* n_theta, int32_t* n_phi) {
    if (L < 0 || l1 < 0 || l2 < 0 || l1 > L || l2 > L || !n_theta || !n_phi) return CGTP_EINVAL;
    if (L > CGTP_MAX_L) return CGTP_EUNSUP;
    cgtp_grid g = grid ? *grid : cgtp_grid{0, 0, CGTP_FP32, CGTP_COVER_DEFAULT};
    int rc = check_grid(L, &g);
    if (rc != CGTP_OK) return rc;
    int nt, np;
    block_grid(g, l1, l2, &nt, &np);
    *n_theta = nt;
    *n_phi = np;
    return CGTP_OK;
}

int cgtp_plan(int32_t L, const cgtp_grid* grid, cgtp_plan_t* plan_out) {
    if (!plan_out || L < 0) return CGTP_EINVAL;
    if (L > CGTP_MAX_L) return CGTP_EUNSUP;
    cgtp_grid g = grid ? *grid : cgtp_grid{0, 0, CGTP_FP32, CGTP_COVER_DEFAULT};
    int rc = check_grid(L, &g);
    if (rc != CGTP_OK) return rc;
    cgtp_plan_s* p = new (std::nothrow) cgtp_plan_s();
    if (!p) return CGTP_ENOMEM;
    p->L = L;
    p->grid = g;
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        delete p;
        return CGTP_EHIP;
    }
    std::vector<BlockDesc> blocks;
    std::vector<int32_t> list;
    if (g.dtype == CGTP_FP32) {
        HostTables<float> h;
        rc = build<float>(p, blocks, h, list);
        if (rc == CGTP_OK) rc = upload<float>(p, blocks, h, list, &p->tf);
    } else {
        HostTables<double> h;
        rc = build<double>(p, blocks, h, list);
        if (rc == CGTP_OK) rc = upload<double>(p, blocks, h, list, &p->td);
    }
    if (rc != CGTP_OK) {
        delete p;
        return rc;
    }
    *plan_out = p;
    return CGTP_OK;
}

int cgtp_destroy(cgtp_plan_t plan) {
    if (!plan) return CGTP_OK;
    int rc = CGTP_OK;
    if (plan->dmem) {
        hipError_t e = hipFree(plan->dmem);
        if (e != hipSuccess) { g_last_hip_error = (int)e; rc = CGTP_EHIP; }
    }
    delete plan;
    return rc;
}

int cgtp_plan_query(cgtp_plan_t plan, int32_t* n_theta, int32_t* n_phi, double* min_abs_K, double* flops_per_pair,
                    double* bytes_per_pair) {
    if (!plan) return CGTP_EINVAL;
    if (n_theta) *n_theta = plan->max_theta;
    if (n_phi) *n_phi = plan->max_phi;
    if (min_abs_K) *min_abs_K = plan->min_abs_K;
    if (flops_per_pair) *flops_per_pair = plan->flops_per_pair;
    if (bytes_per_pair) *bytes_per_pair = plan->bytes_per_pair;
    return CGTP_OK;
}

}  // extern "C"

namespace {

// Shared by both forward entry points: N rows (pair, channel), x2 with one row
// per row or per pair, optional path weights.
int forward_rows(cgtp_plan_t plan, const void* x1, const void* x2, const void* w, void* out, int64_t N,
                 int32_t channels, int32_t flags, void* hip_stream, bool real_basis = false) {
    const int L = plan->L;
    const size_t esz = plan->grid.dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)(L + 1) * (L + 1), nout = (size_t)cgtp_num_outputs(L);
    const int64_t npaths = path_index(L, L + 1, 0, 1);
    if ((uint64_t)N > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const int64_t n2 = (flags & cgtp::kX2Shared) ? N / channels : N;
    const int64_t nw = (flags & cgtp::kWeightsPerRow) ? N : channels;
    if (w && (uint64_t)nw > (uint64_t)(INT64_MAX / (npaths * (int64_t)esz))) return CGTP_EINVAL;
    const size_t bin = (size_t)N * nin * esz, bin2 = (size_t)n2 * nin * esz, bout = (size_t)N * nout * esz;
    const size_t bw = w ? (size_t)nw * npaths * esz : 0;
    if (overlaps(out, bout, x1, bin) || overlaps(out, bout, x2, bin2) || (w && overlaps(out, bout, w, bw)))
        return CGTP_EINVAL;
    // the plan's tables live on the device current when it was built
    int dev = -1;
    const hipError_t de = hipGetDevice(&dev);
    if (de != hipSuccess) {
        g_last_hip_error = (int)de;
        return CGTP_EHIP;
    }
    if (dev != plan->device) return CGTP_EINVAL;
    cgtp::LaunchMap map{};
    map.ncls = (int32_t)plan->classes.size();
    map.cum[0] = 0;
    // pair tiles per work-group: enough work-groups to fill the device several
    // times over, the rest walked in a loop so block-level set-up is amortised
    int64_t total_tiles = 0;
    for (const auto& cl : plan->classes) total_tiles += (N + cl.pairs - 1) / cl.pairs * cl.count;
    const int64_t target_wgs = 16384;
    // (at most 16: same-process A/B against 8, 32 and 64 at L = 32 and 16)
    int tpw = (int)std::max<int64_t>(1, std::min<int64_t>(16, total_tiles / target_wgs));
    for (int c = 0; c < map.ncls; ++c) {
        const auto& cl = plan->classes[c];
        map.pairs[c] = cl.pairs;
        map.list_off[c] = cl.off;
        map.tpw[c] = tpw;
        map.ntiles[c] = (N + cl.pairs - 1) / cl.pairs;
        map.wpb[c] = (map.ntiles[c] + tpw - 1) / tpw;
        map.cum[c + 1] = map.cum[c] + map.wpb[c] * cl.count;
    }
    // one channel, no sharing, no weights: the plain kernel
    const bool plain = channels == 1 && flags == 0 && !w;
    int err;
    if (real_basis) {
        err = plan->grid.dtype == CGTP_FP32
                  ? cgtp::launch_blocks_real_f32(plan->tf, plan->d_list, map, plan->lds_bytes, (const float*)x1,
                                                 (const float*)x2, (float*)out, N, L, hip_stream)
                  : cgtp::launch_blocks_real_f64(plan->td, plan->d_list, map, plan->lds_bytes, (const double*)x1,
                                                 (const double*)x2, (double*)out, N, L, hip_stream);
    } else if (plan->grid.dtype == CGTP_FP32) {
        const cgtp::ChanArgs<float> ch{(const float*)w, channels, flags, (int32_t)npaths};
        err = plain ? cgtp::launch_blocks_f32(plan->tf, plan->d_list, map, plan->lds_bytes, (const float*)x1,
                                              (const float*)x2, (float*)out, N, L, hip_stream)
                    : cgtp::launch_blocks_channels_f32(plan->tf, plan->d_list, map, plan->lds_bytes_ch,
                                                       (const float*)x1, (const float*)x2, (float*)out, N, L, ch,
                                                       hip_stream);
    } else {
        const cgtp::ChanArgs<double> ch{(const double*)w, channels, flags, (int32_t)npaths};
        err = plain ? cgtp::launch_blocks_f64(plan->td, plan->d_list, map, plan->lds_bytes, (const double*)x1,
                                              (const double*)x2, (double*)out, N, L, hip_stream)
                    : cgtp::launch_blocks_channels_f64(plan->td, plan->d_list, map, plan->lds_bytes_ch,
                                                       (const double*)x1, (const double*)x2, (double*)out, N, L,
                                                       ch, hip_stream);
    }
    if (err != 0) {
        g_last_hip_error = err;
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

}  // namespace

extern "C" {

int cgtp_forward(cgtp_plan_t plan, const void* x1, const void* x2, void* out, int64_t N, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !out) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
    return forward_rows(plan, x1, x2, nullptr, out, N, 1, 0, hip_stream);
}

int cgtp_forward_weighted(cgtp_plan_t plan, const void* x1, const void* x2, const void* weights, void* out,
                          int64_t N, const cgtp_channels* ch, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    const int32_t C = ch ? ch->channels : 1;
    if (C < 1 || (ch && ((ch->x2_shared & ~1) || (ch->weights_per_pair & ~1) || ch->reserved))) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !out) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
    const size_t esz = plan->grid.dtype == CGTP_FP32 ? 4 : 8;
    if ((uintptr_t)weights & (esz - 1)) return CGTP_EINVAL;
    if (N > INT64_MAX / C) return CGTP_EINVAL;
    const int32_t flags = (ch && ch->x2_shared ? cgtp::kX2Shared : 0) |
                          (ch && ch->weights_per_pair ? cgtp::kWeightsPerRow : 0);
    return forward_rows(plan, x1, x2, weights, out, N * C, C, flags, hip_stream);
}

int64_t cgtp_num_paths(int32_t L) { return L < 0 ? -1 : path_index(L, L + 1, 0, 1); }

}  // extern "C"

extern "C" {

// The fused kernel needs no workspace; the call keeps its workspace arguments.
int64_t cgtp_real_workspace_bytes(cgtp_plan_t plan, int64_t N) { return (!plan || N < 0) ? -1 : 0; }

int cgtp_forward_real(cgtp_plan_t plan, const void* x1, const void* x2, void* out, int64_t N, void* workspace,
                      int64_t workspace_bytes, void* hip_stream) {
    (void)workspace;
    if (!plan || N < 0 || workspace_bytes < 0) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !out) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
    return forward_rows(plan, x1, x2, nullptr, out, N, 1, 0, hip_stream, true);
}

int cgtp_backward_query(cgtp_plan_t plan, double* flops_per_pair, double* bytes_per_pair) {
    if (!plan) return CGTP_EINVAL;
    if (!plan->bwd_ok) return CGTP_EUNSUP;
    const double esz = plan->grid.dtype == CGTP_FP32 ? 4 : 8;
    const double nin = (double)(plan->L + 1) * (plan->L + 1);
    if (flops_per_pair) *flops_per_pair = plan->bwd_flops_per_pair;
    if (bytes_per_pair) *bytes_per_pair = esz * (4 * nin + nin * nin);
    return CGTP_OK;
}

int64_t cgtp_backward_workspace_bytes(cgtp_plan_t plan, int64_t N) {
    if (!plan || N < 0) return -1;
    const int64_t esz = plan->grid.dtype == CGTP_FP32 ? 4 : 8;
    const int64_t per = 2 * (int64_t)(plan->L + 1) * (plan->L + 1) * (plan->L + 1) * esz;
    if (N > INT64_MAX / per) return -1;
    return N * per;
}

int cgtp_backward(cgtp_plan_t plan, const void* x1, const void* x2, const void* grad_out, void* grad_x1,
                  void* grad_x2, int64_t N, void* workspace, int64_t workspace_bytes, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (!plan->bwd_ok) return CGTP_EUNSUP;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !grad_out || (!grad_x1 && !grad_x2) || !workspace) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)grad_out | (uintptr_t)grad_x1 | (uintptr_t)grad_x2) & 15)
        return CGTP_EINVAL;
    if ((uintptr_t)workspace & 255) return CGTP_EINVAL;
    const int L = plan->L;
    const size_t esz = plan->grid.dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)(L + 1) * (L + 1), nout = (size_t)cgtp_num_outputs(L);
    if ((uint64_t)N > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const int64_t need = cgtp_backward_workspace_bytes(plan, N);
    if (need < 0 || workspace_bytes < need) return CGTP_EINVAL;
    const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
    const void* ins[3] = {x1, x2, grad_out};
    const size_t insz[3] = {bin, bin, bout};
    void* outs[3] = {grad_x1, grad_x2, workspace};
    const size_t outsz[3] = {bin, bin, (size_t)need};
    for (int a = 0; a < 3; ++a) {
        if (!outs[a]) continue;
        for (int b = 0; b < 3; ++b)
            if (overlaps(outs[a], outsz[a], ins[b], insz[b])) return CGTP_EINVAL;
        for (int b = a + 1; b < 3; ++b)
            if (outs[b] && overlaps(outs[a], outsz[a], outs[b], outsz[b])) return CGTP_EINVAL;
    }
    int dev = -1;
    const hipError_t de = hipGetDevice(&dev);
    if (de != hipSuccess) {
        g_last_hip_error = (int)de;
        return CGTP_EHIP;
    }
    if (dev != plan->device) return CGTP_EINVAL;
    // one work-group per (block, pair)
    if ((int64_t)nin * N > 0x7fffffffLL) return CGTP_EUNSUP;
    const int nblocks = (L + 1) * (L + 1);
    const cgtp::BwdLaunch bl{plan->d_bwd_list, plan->bwd_nsmall, nblocks - plan->bwd_nsmall, plan->bwd_lds_small,
                             plan->bwd_lds_large};
    int err;
    if (plan->grid.dtype == CGTP_FP32)
        err = cgtp::launch_backward_f32(plan->tf, bl, (const float*)x1, (const float*)x2, (const float*)grad_out,
                                        (float*)grad_x1, (float*)grad_x2, (float*)workspace, N, L, hip_stream);
    else
        err = cgtp::launch_backward_f64(plan->td, bl, (const double*)x1, (const double*)x2, (const double*)grad_out,
                                        (double*)grad_x1, (double*)grad_x2, (double*)workspace, N, L, hip_stream);
    if (err != 0) {
        g_last_hip_error = err;
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

int64_t cgtp_path_index(int32_t L, int32_t l1, int32_t l2, int32_t l3) {
    if (L >= 0 && l1 == L + 1) return -1;
    return path_index(L, l1, l2, l3);
}

}  // extern "C"

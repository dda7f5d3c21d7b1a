// Drives the host-side code of the library and the oracle under ASan/UBSan:
// every plan's host maths and table building (cgtp_plan and istp_plan up to
// L = 32, both dtypes, both covers, forced grids), the exported host maths,
// istp_plan_describe, argument validation, and the oracle's products and
// gradients.  Prints one line per section; any sanitizer report aborts it.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../include/cgtp.h"
#include "../../include/istp.h"

extern "C" {
double oracle_cg(int j1, int m1, int j2, int m2, int j, int m);
int oracle_cg_block(int l1, int l2, int l3, double* out);
int oracle_cgtp(int L, int64_t N, const double* x1, const double* x2, double* out, int nthreads);
int oracle_cgtp_backward(int L, int64_t N, const double* x1, const double* x2, const double* g, double* gx1,
                         double* gx2, int nthreads);
}

static int fails = 0;
#define EXPECT(cond)                                                       \
    do {                                                                   \
        if (!(cond)) {                                                     \
            std::printf("FAILED %s at line %d\n", #cond, __LINE__);        \
            ++fails;                                                       \
        }                                                                  \
    } while (0)

int main() {
    // cgtp plans: host maths and tables, then the allocation stand-in fails
    for (int L : {0, 1, 2, 3, 5, 8, 16, 32})
        for (int cover = 0; cover < 2; ++cover) {
            cgtp_grid g{0, 0, CGTP_FP32, cover};
            cgtp_plan_t p = nullptr;
            EXPECT(cgtp_plan(L, &g, &p) == CGTP_ENOMEM && p == nullptr);
        }
    for (int L : {0, 4, 12, 19}) {
        cgtp_grid g{0, 0, CGTP_FP64, 0};
        cgtp_plan_t p = nullptr;
        EXPECT(cgtp_plan(L, &g, &p) == CGTP_ENOMEM);
    }
    {
        cgtp_grid g{12, 27, CGTP_FP32, 0};   // one global grid for L = 5
        cgtp_plan_t p = nullptr;
        EXPECT(cgtp_plan(5, &g, &p) == CGTP_ENOMEM);
        cgtp_grid bad{10, 0, CGTP_FP32, 0};
        EXPECT(cgtp_plan(5, &bad, &p) == CGTP_EGRID);
        EXPECT(cgtp_plan(33, nullptr, &p) == CGTP_EUNSUP);
        EXPECT(cgtp_plan(-1, nullptr, &p) == CGTP_EINVAL);
    }
    std::printf("cgtp plans done\n");
    // exported host maths
    for (int j1 = 0; j1 <= 12; ++j1)
        for (int j2 = 0; j2 <= 12; ++j2)
            for (int j3 = std::abs(j1 - j2); j3 <= j1 + j2; ++j3)
                for (int cover = 0; cover < 2; ++cover) {
                    double K = 0;
                    int32_t kind = -1;
                    EXPECT(cgtp_path_norm(j1, j2, j3, cover, &K, &kind) == CGTP_OK);
                    EXPECT(std::isfinite(K));
                }
    EXPECT(std::fabs(cgtp_wigner_9j(1, 1, 1, 1, 1, 1, 1, 1, 1)) < 1e-12);
    for (int j = 0; j <= 40; ++j)
        for (int m = -j; m <= j; ++m)
            for (int q = -1; q <= 1; ++q) EXPECT(std::isfinite(cgtp_cg_vector(j, m, q, j, m + q)));
    for (int l = 0; l <= 64; ++l) EXPECT(std::isfinite(cgtp_cg_zero(l, l, 2 * (l / 2))));
    for (int n : {1, 2, 17, 66, 130}) {
        std::vector<double> x(n), w(n);
        EXPECT(cgtp_gauss_legendre(n, x.data(), w.data()) == CGTP_OK);
        double s = 0;
        for (double v : w) s += v;
        EXPECT(std::fabs(s - 2.0) < 1e-12);
    }
    {
        std::vector<double> out(65 * 66 / 2);
        EXPECT(cgtp_legendre(64, 0.3, out.data()) == CGTP_OK);
        EXPECT(cgtp_legendre(64, 1.5, out.data()) == CGTP_EINVAL);
    }
    for (int L = 0; L <= 32; ++L) {
        EXPECT(cgtp_num_outputs(L) == (int64_t)(L + 1) * (L + 1) * (L + 1) * (L + 1));
        int64_t total = 0;
        for (int l1 = 0; l1 <= L; ++l1)
            for (int l2 = 0; l2 <= L; ++l2) {
                int32_t nt = 0, np = 0;
                EXPECT(cgtp_block_grid(L, nullptr, l1, l2, &nt, &np) == CGTP_OK);
                for (int l3 = std::abs(l1 - l2); l3 <= l1 + l2; ++l3) {
                    EXPECT(cgtp_path_offset(L, l1, l2, l3) >= 0);
                    EXPECT(cgtp_path_index(L, l1, l2, l3) == total);
                    ++total;
                }
            }
        EXPECT(cgtp_num_paths(L) == total);
    }
    std::printf("host maths done\n");
    // signal products: descriptors for every degree, spin and dtype; a few plans
    std::vector<int32_t> desc(48);
    for (int L = 0; L <= 32; ++L)
        for (int spin = 0; spin <= 2; ++spin)
            for (int dt = 0; dt < 2; ++dt) {
                const int rc = istp_plan_describe(L, spin, dt, desc.data());
                EXPECT(rc == CGTP_OK || rc == CGTP_EUNSUP);
            }
    for (int spin = 0; spin <= 2; ++spin)
        for (int L : {1, 4, 16}) {
            istp_plan_t p = nullptr;
            EXPECT(istp_plan(L, spin, 0, &p) == CGTP_ENOMEM);
        }
    std::printf("signal-product plans done\n");
    // oracle: products and gradients on seeded rows
    {
        const int L = 4, N = 3, nin = (L + 1) * (L + 1), nout = nin * nin;
        std::vector<double> x1(N * nin), x2(N * nin), g(N * nout), z(N * nout), g1(N * nin), g2(N * nin);
        unsigned s = 12345;
        auto rnd = [&]() { s = s * 1103515245u + 12345u; return ((s >> 8) & 0xffff) / 32768.0 - 1.0; };
        for (auto* v : {&x1, &x2, &g})
            for (auto& e : *v) e = rnd();
        EXPECT(oracle_cgtp(L, N, x1.data(), x2.data(), z.data(), 2) == 0);
        EXPECT(oracle_cgtp_backward(L, N, x1.data(), x2.data(), g.data(), g1.data(), g2.data(), 2) == 0);
        // Euler's identity for a bilinear map
        for (int n = 0; n < N; ++n) {
            double a = 0, b = 0;
            for (int i = 0; i < nout; ++i) a += g[n * nout + i] * z[n * nout + i];
            for (int i = 0; i < nin; ++i) b += g1[n * nin + i] * x1[n * nin + i];
            EXPECT(std::fabs(a - b) <= 1e-10 * (1 + std::fabs(a)));
        }
        std::vector<double> blk(7 * 5);
        EXPECT(oracle_cg_block(2, 3, 3, blk.data()) == 0);
        EXPECT(std::isfinite(oracle_cg(3, 1, 2, -1, 4, 0)));
    }
    std::printf("oracle done\n");
    if (fails) return 1;
    std::printf("sanitized host code OK\n");
    return 0;
}

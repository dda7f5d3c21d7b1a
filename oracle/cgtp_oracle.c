/*
 * Oracle for the full Clebsch-Gordan tensor product (CGTP).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow reference that the
 * GPU path is checked against.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header,
 * table or constant with the GPU library, and it must never be called from the
 * product path.
 *
 * What it computes (the plain definition of the CGTP, Section 1 and the
 * notation of Appendix F.1; the output layout is this project's choice):
 *
 *   for every pair n, degrees l1, l2 in [0, L], l3 in [|l1-l2|, l1+l2] and
 *   m3 in [-l3, l3]:
 *     z[n, off(l1,l2) + l3^2 - (l1-l2)^2 + l3 + m3]
 *        = sum_{m1=-l1..l1} sum_{m2=-l2..l2}
 *              C^{l3 m3}_{l1 m1 l2 m2} * x1[n, l1^2+l1+m1] * x2[n, l2^2+l2+m2]
 *   with off(l1,l2) = l1^2 (L+1)^2 + (2 l1 + 1) l2^2.
 *
 * The double sum runs over every (m1, m2); the coefficient is zero unless
 * m1 + m2 = m3, so the loop is the naive O(L^6) one.  Inputs are real numbers
 * in the complex spherical basis (quantum-mechanics convention, footnote of
 * Section 3.3), components ordered m = -l..l, degrees 0..L.
 *
 * Clebsch-Gordan coefficients come from Racah's closed formula with the
 * Condon-Shortley phase convention, evaluated in long double:
 *
 *   C^{j m}_{j1 m1 j2 m2} = delta(m, m1+m2)
 *     * sqrt[(2j+1) (j1+j2-j)! (j1-j2+j)! (-j1+j2+j)! / (j1+j2+j+1)!]
 *     * sqrt[(j1+m1)! (j1-m1)! (j2+m2)! (j2-m2)! (j+m)! (j-m)!]
 *     * sum_k (-1)^k / [k! (j1+j2-j-k)! (j1-m1-k)! (j2+m2-k)!
 *                       (j-j2+m1+k)! (j-j1-m2+k)!]
 *
 * The gradients of the CGTP (oracle_cgtp_backward) are the same double sum
 * differentiated term by term by x1 and by x2.
 *
 * Arithmetic: products are accumulated in double (fp64).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_MAX_L 40
#define FACT_MAX (6 * ORACLE_MAX_L + 8)

static long double g_fact[FACT_MAX + 1];
static pthread_once_t g_fact_once = PTHREAD_ONCE_INIT;

static void init_fact(void) {
    g_fact[0] = 1.0L;
    for (int i = 1; i <= FACT_MAX; ++i) g_fact[i] = g_fact[i - 1] * (long double)i;
}

static int iabs_(int a) { return a < 0 ? -a : a; }

/* Racah's formula.  Returns 0 for any selection-rule violation. */
double oracle_cg(int j1, int m1, int j2, int m2, int j, int m) {
    pthread_once(&g_fact_once, init_fact);
    if (j1 < 0 || j2 < 0 || j < 0) return 0.0;
    if (m1 + m2 != m) return 0.0;
    if (iabs_(m1) > j1 || iabs_(m2) > j2 || iabs_(m) > j) return 0.0;
    if (j < iabs_(j1 - j2) || j > j1 + j2) return 0.0;
    if (j1 + j2 + j + 1 > FACT_MAX) return NAN;
    long double pre = sqrtl((long double)(2 * j + 1) * g_fact[j1 + j2 - j] * g_fact[j1 - j2 + j] *
                            g_fact[-j1 + j2 + j] / g_fact[j1 + j2 + j + 1]);
    pre *= sqrtl(g_fact[j1 + m1] * g_fact[j1 - m1] * g_fact[j2 + m2] * g_fact[j2 - m2] *
                 g_fact[j + m] * g_fact[j - m]);
    long double s = 0.0L;
    for (int k = 0; k <= j1 + j2 - j; ++k) {
        int a = j1 + j2 - j - k, b = j1 - m1 - k, c = j2 + m2 - k;
        int d = j - j2 + m1 + k, e = j - j1 - m2 + k;
        if (a < 0 || b < 0 || c < 0 || d < 0 || e < 0) continue;
        long double t = 1.0L / (g_fact[k] * g_fact[a] * g_fact[b] * g_fact[c] * g_fact[d] * g_fact[e]);
        s += (k & 1) ? -t : t;
    }
    return (double)(pre * s);
}

/* ---- coefficient table: for each (l1, l2, l3) a dense [m3][m1] block ---- */

typedef struct {
    int L;
    int64_t *off;   /* [(L+1)^2 * (2L+1)] offset of block (l1,l2,l3), -1 if invalid */
    double *val;
    double build_seconds;
} cg_table;

static cg_table g_tab = {-1, NULL, NULL, 0.0};
static pthread_mutex_t g_tab_lock = PTHREAD_MUTEX_INITIALIZER;

static int64_t tab_index(int L, int l1, int l2, int l3) {
    return ((int64_t)l1 * (L + 1) + l2) * (2 * L + 1) + l3;
}

static double now_seconds(void) {
#ifdef _OPENMP
    return omp_get_wtime();
#else
    return 0.0;
#endif
}

/* Builds (or reuses) the table for degree L.  Returns 0 on success. */
static int ensure_table(int L, int nthreads) {
    pthread_mutex_lock(&g_tab_lock);
    if (g_tab.L == L) { pthread_mutex_unlock(&g_tab_lock); return 0; }
    free(g_tab.off); free(g_tab.val);
    g_tab.off = NULL; g_tab.val = NULL; g_tab.L = -1;
    int64_t nblk = (int64_t)(L + 1) * (L + 1) * (2 * L + 1);
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * nblk);
    if (!off) { pthread_mutex_unlock(&g_tab_lock); return -1; }
    int64_t total = 0;
    for (int l1 = 0; l1 <= L; ++l1)
        for (int l2 = 0; l2 <= L; ++l2)
            for (int l3 = 0; l3 <= 2 * L; ++l3) {
                int64_t id = tab_index(L, l1, l2, l3);
                if (l3 < iabs_(l1 - l2) || l3 > l1 + l2) { off[id] = -1; continue; }
                off[id] = total;
                total += (int64_t)(2 * l3 + 1) * (2 * l1 + 1);
            }
    double *val = (double *)malloc(sizeof(double) * (total > 0 ? total : 1));
    if (!val) { free(off); pthread_mutex_unlock(&g_tab_lock); return -1; }
    double t0 = now_seconds();
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int l1 = 0; l1 <= L; ++l1)
        for (int l2 = 0; l2 <= L; ++l2)
            for (int l3 = iabs_(l1 - l2); l3 <= l1 + l2; ++l3) {
                double *blk = val + off[tab_index(L, l1, l2, l3)];
                for (int m3 = -l3; m3 <= l3; ++m3)
                    for (int m1 = -l1; m1 <= l1; ++m1)
                        blk[(m3 + l3) * (2 * l1 + 1) + (m1 + l1)] =
                            oracle_cg(l1, m1, l2, m3 - m1, l3, m3);
            }
    g_tab.build_seconds = now_seconds() - t0;
    g_tab.off = off; g_tab.val = val; g_tab.L = L;
    pthread_mutex_unlock(&g_tab_lock);
    return 0;
}

/* Table lookup with the CG selection rules spelled out. */
static inline double cg_lookup(int L, int l1, int m1, int l2, int m2, int l3, int m3) {
    if (m1 + m2 != m3) return 0.0;
    if (iabs_(m2) > l2) return 0.0;
    const double *blk = g_tab.val + g_tab.off[tab_index(L, l1, l2, l3)];
    (void)L;
    return blk[(m3 + l3) * (2 * l1 + 1) + (m1 + l1)];
}

int64_t oracle_num_outputs(int L) {
    int64_t a = (int64_t)(L + 1) * (L + 1);
    return a * a;
}

int64_t oracle_path_offset(int L, int l1, int l2, int l3) {
    if (L < 0 || l1 < 0 || l2 < 0 || l1 > L || l2 > L) return -1;
    if (l3 < iabs_(l1 - l2) || l3 > l1 + l2) return -1;
    return (int64_t)l1 * l1 * (L + 1) * (L + 1) + (int64_t)(2 * l1 + 1) * l2 * l2 +
           (int64_t)l3 * l3 - (int64_t)(l1 - l2) * (l1 - l2);
}

/* Fills out[(2 l3 + 1) * (2 l1 + 1)] with C^{l3 m3}_{l1 m1 l2 (m3-m1)}, [m3][m1]. */
int oracle_cg_block(int l1, int l2, int l3, double *out) {
    if (l1 < 0 || l2 < 0 || l3 < iabs_(l1 - l2) || l3 > l1 + l2) return -1;
    for (int m3 = -l3; m3 <= l3; ++m3)
        for (int m1 = -l1; m1 <= l1; ++m1)
            out[(m3 + l3) * (2 * l1 + 1) + (m1 + l1)] = oracle_cg(l1, m1, l2, m3 - m1, l3, m3);
    return 0;
}

/*
 * Full CGTP of N pairs.  x1, x2: [N, (L+1)^2]; out: [N, (L+1)^4]; all fp64,
 * row-major.  nthreads <= 0 uses the OpenMP default.  Returns 0 on success,
 * -1 on bad arguments or allocation failure.
 */
int oracle_cgtp(int L, int64_t N, const double *x1, const double *x2, double *out, int nthreads) {
    if (L < 0 || L > ORACLE_MAX_L || N < 0) return -1;
    if (N == 0) return 0;
    if (!x1 || !x2 || !out) return -1;
    if (ensure_table(L, nthreads) != 0) return -1;
    const int64_t nin = (int64_t)(L + 1) * (L + 1);
    const int64_t nout = oracle_num_outputs(L);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t n = 0; n < N; ++n)
        for (int l1 = 0; l1 <= L; ++l1) {
            const double *a = x1 + n * nin;
            const double *b = x2 + n * nin;
            double *z = out + n * nout;
            for (int l2 = 0; l2 <= L; ++l2)
                for (int l3 = iabs_(l1 - l2); l3 <= l1 + l2; ++l3) {
                    int64_t base = oracle_path_offset(L, l1, l2, l3);
                    for (int m3 = -l3; m3 <= l3; ++m3) {
                        double s = 0.0;
                        for (int m1 = -l1; m1 <= l1; ++m1)
                            for (int m2 = -l2; m2 <= l2; ++m2) {
                                double c = cg_lookup(L, l1, m1, l2, m2, l3, m3);
                                s += c * a[l1 * l1 + l1 + m1] * b[l2 * l2 + l2 + m2];
                            }
                        z[base + l3 + m3] = s;
                    }
                }
        }
    return 0;
}

/*
 * Gradients of the full CGTP: for an upstream gradient g = dLoss/dz of the
 * same layout as z, the plain definition of the derivative of the bilinear
 * map written out (each term of the double sum above, differentiated by x1
 * and by x2):
 *
 *   gx1[n, l1^2+l1+m1] = sum over paths (l1, l2, l3), m2:
 *                          C^{l3, m1+m2}_{l1 m1 l2 m2} g[n, path, m1+m2] x2[n, l2^2+l2+m2]
 *   gx2[n, l2^2+l2+m2] = sum over paths (l1, l2, l3), m1:
 *                          C^{l3, m1+m2}_{l1 m1 l2 m2} g[n, path, m1+m2] x1[n, l1^2+l1+m1]
 *
 * x1, x2, gx1, gx2: [N, (L+1)^2]; g: [N, (L+1)^4]; fp64.  Either output may
 * be NULL.  Returns 0 on success, -1 on bad arguments or allocation failure.
 */
int oracle_cgtp_backward(int L, int64_t N, const double *x1, const double *x2, const double *g, double *gx1,
                         double *gx2, int nthreads) {
    if (L < 0 || L > ORACLE_MAX_L || N < 0) return -1;
    if (N == 0) return 0;
    if (!x1 || !x2 || !g) return -1;
    if (ensure_table(L, nthreads) != 0) return -1;
    const int64_t nin = (int64_t)(L + 1) * (L + 1);
    const int64_t nout = oracle_num_outputs(L);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
    #pragma omp parallel for schedule(dynamic)
    for (int64_t n = 0; n < N; ++n) {
        const double *a = x1 + n * nin;
        const double *b = x2 + n * nin;
        const double *gz = g + n * nout;
        double *ga = gx1 ? gx1 + n * nin : NULL;
        double *gb = gx2 ? gx2 + n * nin : NULL;
        if (ga) memset(ga, 0, sizeof(double) * nin);
        if (gb) memset(gb, 0, sizeof(double) * nin);
        for (int l1 = 0; l1 <= L; ++l1)
            for (int l2 = 0; l2 <= L; ++l2)
                for (int l3 = iabs_(l1 - l2); l3 <= l1 + l2; ++l3) {
                    const int64_t base = oracle_path_offset(L, l1, l2, l3);
                    for (int m1 = -l1; m1 <= l1; ++m1)
                        for (int m2 = -l2; m2 <= l2; ++m2) {
                            const int m3 = m1 + m2;
                            if (iabs_(m3) > l3) continue;
                            const double c = cg_lookup(L, l1, m1, l2, m2, l3, m3) * gz[base + l3 + m3];
                            if (ga) ga[l1 * l1 + l1 + m1] += c * b[l2 * l2 + l2 + m2];
                            if (gb) gb[l2 * l2 + l2 + m2] += c * a[l1 * l1 + l1 + m1];
                        }
                }
    }
    return 0;
}

/* Seconds spent building the coefficient table for the current degree. */
double oracle_table_build_seconds(void) { return g_tab.build_seconds; }

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

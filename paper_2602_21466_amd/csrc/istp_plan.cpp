// Host side of the multiple-input, multiple-output irrep-signal tensor
// products: the plan (grid, MFMA weight tables, tile lists, recombination
// weights, uploaded once) and the C ABI of include/istp.h.
//
// The host math (Gauss-Legendre nodes, normalised Legendre functions, vector
// coupling coefficients) comes from the library's own exported helpers in
// cgtp_plan.cpp.  The device work is in istp_kernels.hip.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <new>
#include <vector>

#include "../../include/istp.h"
#include "cgtp_internal.h"
#include "istp_internal.h"

// One product's descriptor and device tables.
struct istp_prod {
    istp::IstpDesc desc{};
    void* dmem = nullptr;
    istp::IstpTables<float> tf{};
    istp::IstpTables<double> td{};
    int n_theta = 0, n_phi = 0;
    double flops_per_pair = 0, bytes_per_pair = 0;
    bool ok = false;
};

// A plan holds the forward product (degrees L, L -> 2L) and, when it fits the
// kernel's limits, the product its gradients use (degrees 2L, L -> L, second
// input time-reversed).
struct istp_plan_s {
    int L = 0, spin = 0, dtype = 0, device = 0;
    istp_prod fwd, bwd;
    istp_prod rfwd, rbwd;   // spin 0: the same two products for rows in the real basis (when they fit)
};

namespace {

const double kPi = 3.14159265358979323846264338327950288;

int64_t label_offset(int spin, int j, int l) {
    if (l < 0 || j < 0) return -1;
    if (spin == ISTP_GAUNT) return j == l ? (int64_t)l * l : -1;
    if (spin == ISTP_TENSOR) {   // j = |l - 2| .. l + 2 at 5 l^2 + j^2 - (l - 2)^2
        if (j < std::abs(l - 2) || j > l + 2) return -1;
        return 5LL * l * l + (int64_t)j * j - (int64_t)(l - 2) * (l - 2);
    }
    if (spin != ISTP_VECTOR || std::abs(j - l) > 1 || j + l < 1) return -1;
    const int jj = j - l + 1;
    return 3LL * l * l + (jj == 0 ? 0 : (jj == 1 ? 2 * l - 1 : 4 * l));
}

// Position of label (j, l) in a row of label weights: l for spin 0; for spin 1
// the labels in row order (l, then j = l - 1, l, l + 1), i.e. 2 l - 1 + j.
int64_t label_index(int spin, int j, int l) {
    if (label_offset(spin, j, l) < 0) return -1;
    if (spin == ISTP_TENSOR) {   // 2 min(l', 2) + 1 labels at each degree l' < l
        int64_t k = 0;
        for (int lp = 0; lp < l; ++lp) k += 2 * std::min(lp, 2) + 1;
        return k + j - std::abs(l - 2);
    }
    return spin == ISTP_GAUNT ? l : 2LL * l - 1 + j;
}

// Labels of a row of degree bound L: L + 1 (spin 0), 3 L + 1 (spin 1),
// 5 L - 1 (spin 2, L >= 1; 1 at L = 0).
int64_t num_labels(int L, int spin) {
    if (L < 0 || spin < ISTP_GAUNT || spin > ISTP_TENSOR) return -1;
    if (spin == ISTP_TENSOR) return L == 0 ? 1 : 5LL * L - 1;
    return spin == ISTP_GAUNT ? L + 1 : 3LL * L + 1;
}

// Label index of every column of a row of degree bound L, appended to v.
void append_column_labels(int L, int spin, std::vector<int32_t>& v) {
    for (int l = 0; l <= L; ++l)
        for (int j = l - spin; j <= l + spin; ++j) {
            if (label_offset(spin, j, l) < 0) continue;
            for (int m = -j; m <= j; ++m) v.push_back((int32_t)label_index(spin, j, l));
        }
}

int64_t row_size(int L, int spin) {
    if (L < 0 || spin < ISTP_GAUNT || spin > ISTP_TENSOR) return -1;
    return (int64_t)(2 * spin + 1) * (L + 1) * (L + 1);
}

int smallest_2a3b(int n) {
    for (int m = std::max(n, 1);; ++m) {
        int v = m;
        while (v % 2 == 0) v /= 2;
        while (v % 3 == 0) v /= 3;
        if (v == 1) return m;
    }
}

// Rows l3 = am + par, am + par + 2, ..., <= Lo of one projection GEMM.
int proj_rows(int Lo, int am, int par) {
    const int top = Lo - am - par;
    return top >= 0 ? top / 2 + 1 : 0;
}

int lift_kp(int L, int am) { return (L - am + 1 + 3) / 4 * 4; }
// both signs (complex basis) or parts (real basis) at order am; the real-basis
// spin-1 lift has both parts at am = 0 too
int lift_ncol(int NC, int P, int am, bool both0 = false) { return ((am || both0) ? 2 : 1) * 2 * NC * P; }

int acoef_len(int L, int NC, int P, bool both0 = false) {
    int n = 0;
    for (int am = 0; am <= L; ++am) n += lift_kp(L, am) * istp::istp_cstride(lift_ncol(NC, P, am, both0));
    return n;
}

// C^{j m}_{j1 m1 j2 m2} (Condon-Shortley phase) by Racah's single-sum formula,
// in long double with log-factorials; 0 outside the selection rules.
long double cg_racah(int j1, int m1, int j2, int m2, int j, int m) {
    if (m1 + m2 != m || std::abs(m1) > j1 || std::abs(m2) > j2 || std::abs(m) > j) return 0.0L;
    if (j < std::abs(j1 - j2) || j > j1 + j2) return 0.0L;
    auto lf = [](int n) { return lgammal((long double)n + 1.0L); };
    const long double pre = 0.5L * (logl(2.0L * j + 1.0L) + lf(j1 + j2 - j) + lf(j1 - j2 + j) + lf(-j1 + j2 + j) -
                                    lf(j1 + j2 + j + 1) + lf(j1 + m1) + lf(j1 - m1) + lf(j2 + m2) + lf(j2 - m2) +
                                    lf(j + m) + lf(j - m));
    const int kmin = std::max({0, j2 - j - m1, j1 - j + m2});
    const int kmax = std::min({j1 + j2 - j, j1 - m1, j2 + m2});
    long double sum = 0.0L;
    for (int k = kmin; k <= kmax; ++k) {
        const long double t = expl(pre - lf(k) - lf(j1 + j2 - j - k) - lf(j1 - m1 - k) - lf(j2 + m2 - k) -
                                   lf(j - j2 + m1 + k) - lf(j - j1 - m2 + k));
        sum += (k & 1) ? -t : t;
    }
    return sum;
}

double fft_flops(int n) { return n > 1 ? 5.0 * n * std::log2((double)n) : 0.0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char *pa = (const char*)a, *pb = (const char*)b;
    return pa < pb + nb && pb < pa + na;
}

template <typename T>
struct Host {
    std::vector<T> lw, pw, tw, liftcg, coef;
    std::vector<int32_t> coefi;
    std::vector<istp::LiftTile> lift;
    std::vector<istp::ProjTile> proj;
    std::vector<int32_t> bcol;   // 2 per operand column
    std::vector<int32_t> lab;    // label index of every column: input 1, input 2, output
};

// Tables of the product of a degree-L1 and a degree-L2 input projected on
// degrees <= Lo.  The grid is exact for every integrand: Gauss-Legendre with
// n_theta >= (L1 + L2 + Lo + 1) / 2 nodes (even), Phi >= L1 + L2 + Lo + 1.
template <typename T>
int build(int L1, int L2, int Lo, int S, int flags, istp_prod* pr, Host<T>& h) {
    const int NC = 2 * S + 1, Lm = std::max(L1, L2);
    const int D = L1 + L2 + Lo;
    const int nmin = (D + 2) / 2;
    const int nt = nmin + (nmin & 1), R = nt / 2;
    const int Phi = smallest_2a3b(D + 1);
    int A = 0, B = 0;
    if (!cgtp::fft_factors(Phi, &A, &B)) return CGTP_EUNSUP;
    if (Lm + 1 > 255) return CGTP_EUNSUP;   // the column table packs am in 8 bits
    // lifts longer than 4 istp::kMaxLiftSteps degrees run in a kernel built for fp32, Phi >= 72
    if (Lm + 1 > 4 * istp::kMaxLiftSteps && (sizeof(T) != 4 || Phi < 72)) return CGTP_EUNSUP;
    // spin 2 is built for grids of at most 81 longitudes (L <= 20 forward) and short lifts
    if (S == ISTP_TENSOR && (Phi > 81 || Lm + 1 > 4 * istp::kMaxLiftSteps)) return CGTP_EUNSUP;

    int nproj = 0;
    for (int am = 0; am <= Lo; ++am)
        for (int par = 0; par < 2; ++par) nproj += (proj_rows(Lo, am, par) + 15) / 16;
    if (nproj > istp::max_tiles<T>(S) * istp::kWaves) return CGTP_EUNSUP;

    // Pairs per work-group and ring pairs per group: the most pairs that fit in
    // LDS with the projection's columns (sign, component, pair) on one MFMA tile
    // (each pair more fills more of the lift's and the projection's columns),
    // then the most ring pairs (more units fill more of the work-group's
    // threads in the transform phases and take fewer passes over the rings).
    const bool rl1 = (flags & istp::kRealBasis) && S == ISTP_VECTOR;   // real basis, spin 1
    // spectra per pair: [component][(Lo + 1)^2] (the real-basis spin-1 kernel adds
    // the order-0 imaginary parts, Lo + 1 per component)
    const int hc_len = NC * ((Lo + 1) * (Lo + 1) + (rl1 ? Lo + 1 : 0));
    const int nin = (int)row_size(L1, S), nin2 = (int)row_size(L2, S);
    int bestP = 0, bestG = 0, bestBytes = 0;
    for (int P : {8, 4, 2, 1}) {
        if (2 * NC * P > 16) continue;
        // inputs and couplings are staged with one batch of loads per thread
        const int stage = P * (nin + nin2) + (S ? NC * NC * (Lm + 1) * (Lm + 1) : 0);
        if (stage > istp::kStageLoads * istp::kThreads) continue;
        for (int G : {16, 12, 8, 4}) {
            const istp::IstpLayout ly = istp::istp_layout<T>(A, B, NC, G, P, acoef_len(Lm, NC, P, rl1), hc_len,
                                                             istp::istp_stage_len(P, nin, nin2, Lm, S), nproj);
            if (ly.bytes > istp::kLdsBudget) continue;
            if (P > bestP || (P == bestP && G > bestG)) {
                bestP = P;
                bestG = G;
                bestBytes = ly.bytes;
            }
        }
    }
    if (bestP == 0) return CGTP_EUNSUP;
    const int P = bestP, G = bestG;
    const int rpad = (R + G - 1) / G * G;
    const int wrow = 16 * ((Lo / 2 + 1 + 15) / 16);   // most rows: am = 0, even parity
    const int Lp = std::max(Lm, Lo);                   // Legendre table degree

    std::vector<double> xs(nt), ws(nt);
    if (cgtp_gauss_legendre(nt, xs.data(), ws.data()) != CGTP_OK) return CGTP_EINVAL;
    // rings 0..R-1 are the northern nodes (x > 0); the south ones are their mirrors
    std::vector<std::vector<double>> plm(R);
    for (int r = 0; r < R; ++r) {
        if (!(xs[r] > 0.0)) return CGTP_EINVAL;
        plm[r].assign((Lp + 1) * (Lp + 2) / 2, 0.0);
        cgtp_legendre(Lp, xs[r], plm[r].data());
    }
    auto pbar = [&](int r, int l, int m) { return plm[r][l * (l + 1) / 2 + m]; };

    // lift weights [am][ring][k]: P_{am+k}^{am}(x_ring)
    std::vector<int> lw_off(Lm + 1);
    for (int am = 0; am <= Lm; ++am) {
        lw_off[am] = (int)h.lw.size();
        const int kp = lift_kp(Lm, am);
        for (int r = 0; r < rpad; ++r)
            for (int k = 0; k < kp; ++k) {
                const int l = am + k;
                h.lw.push_back(r < R && l <= Lm ? (T)pbar(r, l, am) : (T)0);
            }
    }
    // projection weights [am][par][ring][row]: w_ring P_{am+par+2 row}^{am}(x_ring)
    for (int am = 0; am <= Lo; ++am)
        for (int par = 0; par < 2; ++par)
            for (int r = 0; r < rpad; ++r)
                for (int row = 0; row < wrow; ++row) {
                    const int l3 = am + par + 2 * row;
                    h.pw.push_back(r < R && l3 <= Lo ? (T)(ws[r] * pbar(r, l3, am)) : (T)0);
                }
    // twiddles exp(-2 pi i t k2 / Phi), pass layout
    const int FS = A * (B + 1);
    h.tw.assign(2 * FS, (T)0);
    for (int t = 0; t < A; ++t)
        for (int k2 = 0; k2 < B; ++k2) {
            const long double ang = -2.0L * (long double)kPi * t * k2 / Phi;
            h.tw[2 * (t * (B + 1) + k2)] = (T)cosl(ang);
            h.tw[2 * (t * (B + 1) + k2) + 1] = (T)sinl(ang);
        }
    // lift couplings C^{j, ml+q}_{l, ml, s, q}, j = l - s .. l + s
    h.liftcg.assign((size_t)NC * NC * (Lm + 1) * (Lm + 1), (T)0);
    if (S == ISTP_TENSOR)
        for (int l = 0; l <= Lm; ++l)
            for (int jj = 0; jj < 5; ++jj)
                for (int c = 0; c < 5; ++c)
                    for (int ml = -l; ml <= l; ++ml) {
                        const int j = l - 2 + jj, q = c - 2;
                        if (j < std::abs(l - 2) || std::abs(ml + q) > j) continue;
                        h.liftcg[(size_t)25 * l * l + (jj * 5 + c) * (2 * l + 1) + ml + l] =
                            (T)cg_racah(l, ml, 2, q, j, ml + q);
                    }

    if (S == ISTP_VECTOR)
        for (int l = 0; l <= Lm; ++l)
            for (int jj = 0; jj < 3; ++jj)
                for (int c = 0; c < 3; ++c)
                    for (int ml = -l; ml <= l; ++ml) {
                        const int j = l - 1 + jj, q = c - 1;
                        if (j < 0 || j + l < 1 || std::abs(ml + q) > j) continue;
                        h.liftcg[(size_t)9 * l * l + (jj * 3 + c) * (2 * l + 1) + ml + l] =
                            (T)cgtp_cg_vector(l, ml, q, j, ml + q);
                    }
    // coefficient operand geometry and lift tiles
    int aoff = 0;
    for (int am = 0; am <= Lm; ++am) {
        const int kp = lift_kp(Lm, am), ncol = lift_ncol(NC, P, am, rl1), cs = istp::istp_cstride(ncol);
        for (int col = 0; col < cs; ++col) h.bcol.insert(h.bcol.end(), {am | (col << 8), aoff + col});
        for (int rb = 0; rb < (G + 7) / 8; ++rb)
            for (int ct = 0; ct < (ncol + 15) / 16; ++ct)
                h.lift.push_back(istp::LiftTile{am, ct, aoff + 16 * ct, cs, lw_off[am], kp, ncol, kp / 4, rb});
        aoff += kp * cs;
    }
    // projection tiles
    for (int am = 0; am <= Lo; ++am)
        for (int par = 0; par < 2; ++par)
            for (int rt = 0; rt < (proj_rows(Lo, am, par) + 15) / 16; ++rt)
                h.proj.push_back(istp::ProjTile{am, par, rt, ((am * 2 + par) * rpad) * wrow + 16 * rt});

    // the kernel packs (weight offset, am, parity) of a projection tile in one word
    if ((int64_t)h.pw.size() >= (1 << 20) || Lo >= 128) return CGTP_EUNSUP;

    // recombination: the raw spectrum of (l3, m) is 4 Phi / (2 pi) times the
    // projection of the product's scalar-harmonic coefficient (doubled unpacked
    // factors, unnormalised longitude sums), and negative orders carry
    // (-1)^|m| from P^{-m} = (-1)^m P^m
    const int no = (Lo + 1) * (Lo + 1);
    const double scale = 2.0 * kPi / (4.0 * Phi);
    auto sgn = [](int m) { return (m < 0 && (-m) % 2) ? -1.0 : 1.0; };
    const int64_t nout = row_size(Lo, S);
    h.coef.assign(4 * nout, (T)0);
    h.coefi.assign(4 * nout, 0);
    if (S == ISTP_TENSOR) {
        // five terms per output (two words of four): q = -2..2 at (l3, m3 - q).
        // The kernel forms the 2 (x) 2 -> 2 products with C^{2 q}_{2 q1 2 q2}
        // in units of c2 = 1 / sqrt(14) (+-1, +-2, +-sqrt(6)); c2 is applied here.
        const long double c2 = 1.0L / sqrtl(14.0L), r6 = sqrtl(6.0L);
        for (int q1 = -2; q1 <= 2; ++q1)
            for (int q2 = -2; q2 <= 2; ++q2) {
                const int q = q1 + q2;
                if (std::abs(q) > 2) continue;
                // the kernel's weight of a_q1 b_q2 in g_q
                long double w;
                const int lo = std::min(std::abs(q1), std::abs(q2)), hi = std::max(std::abs(q1), std::abs(q2));
                if (q == 0) w = q1 == 0 ? -2.0L : (std::abs(q1) == 2 ? 2.0L : 1.0L);
                else if (std::abs(q) == 2) w = (q1 == q2) ? -r6 : 2.0L;
                else w = (lo == 1 && hi == 2) ? r6 : -1.0L;
                if (fabsl(cg_racah(2, q1, 2, q2, 2, q) - w * c2) > 1e-15L) return CGTP_EINVAL;
            }
        h.coef.assign(8 * nout, (T)0);
        h.coefi.assign(8 * nout, 0);
        for (int l3 = 0; l3 <= Lo; ++l3)
            for (int j3 = std::abs(l3 - 2); j3 <= l3 + 2; ++j3) {
                const int64_t off = label_offset(ISTP_TENSOR, j3, l3);
                for (int m3 = -j3; m3 <= j3; ++m3) {
                    const int64_t o = off + j3 + m3;
                    for (int q = -2; q <= 2; ++q) {
                        const int ml = m3 - q;
                        h.coefi[8 * o + q + 2] = (int32_t)(l3 * l3 + l3);   // any entry; zero weight
                        if (std::abs(ml) > l3) continue;
                        h.coef[8 * o + q + 2] = (T)(cg_racah(l3, ml, 2, q, j3, m3) * c2 * scale * sgn(ml));
                        h.coefi[8 * o + q + 2] = (q + 2) * no + l3 * l3 + l3 + ml;
                    }
                }
            }
    } else if (S == ISTP_GAUNT && (flags & istp::kRealBasis)) {
        // real basis: the kernel's spectrum slots (l3, +mu) and (l3, -mu) hold Re and
        // Im of 2 Phi / (2 pi) times the complex coefficient h at +mu (exact
        // unpacking: no doubled factors; the projection's operand is doubled); the
        // real-basis output reads r_0 = h_0, r_mu = sqrt 2 (-1)^mu Re h_mu,
        // r_-mu = -sqrt 2 (-1)^mu Im h_mu
        const double sr = 2.0 * kPi / (2.0 * Phi), rt2 = std::sqrt(2.0);
        for (int l3 = 0; l3 <= Lo; ++l3)
            for (int m3 = -l3; m3 <= l3; ++m3) {
                const int o = l3 * l3 + l3 + m3, mu = std::abs(m3);
                const double par = (mu & 1) ? -1.0 : 1.0;
                h.coef[4 * o] = (T)(m3 == 0 ? sr : (m3 > 0 ? sr * rt2 * par : -sr * rt2 * par));
                h.coefi[4 * o] = h.coefi[4 * o + 1] = h.coefi[4 * o + 2] = o;
                h.coefi[4 * o + 3] = 1;
            }
    } else if (S == ISTP_GAUNT) {
        for (int l3 = 0; l3 <= Lo; ++l3)
            for (int m3 = -l3; m3 <= l3; ++m3) {
                const int o = l3 * l3 + l3 + m3;
                h.coef[4 * o] = (T)(scale * sgn(m3));
                h.coefi[4 * o] = h.coefi[4 * o + 1] = h.coefi[4 * o + 2] = o;
                h.coefi[4 * o + 3] = 1;
            }
    } else if (rl1) {
        // real basis, spin 1.  Spectrum slots (c, part, l3, m' >= 0): part Re at
        // l3^2 + l3 + m', part Im at l3^2 + l3 - m' (m' > 0) or (Lo + 1)^2 + l3 (m' = 0),
        // per component c at c * nos.  They are Phi / (2 pi) times the true
        // projections of g_+1 (c = 2) and g_-1 (c = 0) at +m', and 2 Phi / (2 pi) times
        // that of Im g_0 (c = 1; g_0 = i Im g_0).  Orders m' < 0 follow from the
        // product being i times a real field h: g_q[-m] = -(-1)^(m+q) conj g_-q[m].  A
        // label's complex output z (sum over q of C^{j3 m3}_{l3,m3-q,1,q} times the
        // coupling C^{1 1}_{1 1 1 0} times g_q) is read back as the three-product path
        // does: w = i^t z at order -|m3|, t = 1 + [sigma3 = -1], r_0 = Re w_0,
        // r_mu = sqrt 2 Re w_-mu, r_-mu = sqrt 2 Im w_-mu.
        const double c1 = cgtp_cg_vector(1, 1, 0, 1, 1);
        const int nos = no + Lo + 1;
        const double k1 = 2.0 * kPi / Phi, k0 = kPi / Phi, rt2 = std::sqrt(2.0);
        auto at = [&](int c, int part, int l3, int mp) {
            return c * nos + (part == 0 ? l3 * l3 + l3 + mp : (mp ? l3 * l3 + l3 - mp : no + l3));
        };
        using Form = std::map<int, double>;
        // adds a * (Re, Im) of the true projection of g_q at (l3, m') to (fr, fi)
        auto addg = [&](Form& fr, Form& fi, int q, int l3, int mp, double a) {
            if (mp >= 0) {
                if (q == 0) {   // g_0 = i H, H from c = 1 (doubled)
                    fr[at(1, 1, l3, mp)] += -a * k0;
                    fi[at(1, 0, l3, mp)] += a * k0;
                } else {
                    const int c = q == 1 ? 2 : 0;
                    fr[at(c, 0, l3, mp)] += a * k1;
                    fi[at(c, 1, l3, mp)] += a * k1;
                }
                return;
            }
            // g_q[-m] = s conj g_-q[m], s = -(-1)^(m+q)
            const int m = -mp;
            const double sgn = ((m + q) & 1) ? 1.0 : -1.0;
            Form xr, xi;
            if (q == 0) {
                xr[at(1, 1, l3, m)] += -k0;
                xi[at(1, 0, l3, m)] += k0;
            } else {
                const int c = q == 1 ? 0 : 2;   // -q
                xr[at(c, 0, l3, m)] += k1;
                xi[at(c, 1, l3, m)] += k1;
            }
            for (const auto& kv : xr) fr[kv.first] += a * sgn * kv.second;
            for (const auto& kv : xi) fi[kv.first] += -a * sgn * kv.second;
        };
        for (int l3 = 0; l3 <= Lo; ++l3)
            for (int j3 = l3 - 1; j3 <= l3 + 1; ++j3) {
                const int64_t off = label_offset(ISTP_VECTOR, j3, l3);
                if (off < 0) continue;
                const int turns = 1 + (((l3 + 1 - j3) & 1) ? 1 : 0);
                for (int m3 = -j3; m3 <= j3; ++m3) {
                    const int64_t o = off + j3 + m3;
                    const int M = -std::abs(m3);
                    Form zr, zi;
                    for (int q = -1; q <= 1; ++q) {
                        const int ml = M - q;
                        if (std::abs(ml) > l3) continue;
                        addg(zr, zi, q, l3, ml, c1 * cgtp_cg_vector(l3, ml, q, j3, M));
                    }
                    // w = i^turns z: one turn Re w = -Im z, Im w = Re z; two turns w = -z
                    const bool want_re = m3 >= 0;
                    const Form* f;
                    double sg = m3 == 0 ? 1.0 : rt2;
                    if (turns == 1) {
                        f = want_re ? &zi : &zr;
                        if (want_re) sg = -sg;
                    } else {
                        f = want_re ? &zr : &zi;
                        sg = -sg;
                    }
                    int k = 0;
                    for (const auto& kv : *f) {
                        if (kv.second == 0.0) continue;
                        if (k == 3) return CGTP_EINVAL;   // at most one entry per q
                        h.coef[4 * o + k] = (T)(sg * kv.second);
                        h.coefi[4 * o + k] = kv.first;
                        ++k;
                    }
                    for (; k < 3; ++k) h.coefi[4 * o + k] = at(1, 0, l3, 0);   // zero weight
                }
            }
    } else {
        // the kernel forms the antisymmetric 1 (x) 1 -> 1 combinations; their
        // common factor is C^{1 1}_{1 1 1 0}
        const double c1 = cgtp_cg_vector(1, 1, 0, 1, 1);
        const int pattern[7][4] = {{1, 0, 1, 1}, {0, 1, 1, -1}, {1, -1, 0, 1}, {-1, 1, 0, -1},
                                   {0, -1, -1, 1}, {-1, 0, -1, -1}, {0, 0, 0, 0}};
        for (const auto& q : pattern) {
            const double want = q[3] * c1;
            if (std::fabs(cgtp_cg_vector(1, q[0], q[1], 1, q[2]) - want) > 1e-14) return CGTP_EINVAL;
        }
        for (int l3 = 0; l3 <= Lo; ++l3)
            for (int j3 = l3 - 1; j3 <= l3 + 1; ++j3) {
                const int64_t off = label_offset(ISTP_VECTOR, j3, l3);
                if (off < 0) continue;
                for (int m3 = -j3; m3 <= j3; ++m3) {
                    const int64_t o = off + j3 + m3;
                    for (int q = -1; q <= 1; ++q) {
                        const int ml = m3 - q;
                        if (std::abs(ml) > l3) continue;
                        h.coef[4 * o + q + 1] = (T)(cgtp_cg_vector(l3, ml, q, j3, m3) * c1 * scale * sgn(ml));
                        h.coefi[4 * o + q + 1] = (q + 1) * no + l3 * l3 + l3 + ml;
                    }
                }
            }
    }

    istp::IstpDesc& d = pr->desc;
    d.L = L1;
    d.L2 = L2;
    d.Lo = Lo;
    d.spin = S;
    d.C = NC;
    d.R = R;
    d.G = G;
    d.Phi = Phi;
    d.A = A;
    d.B = B;
    d.pairs = P;
    d.nin = nin;
    d.nin2 = nin2;
    d.nout = (int32_t)nout;
    d.n_lift = (int32_t)h.lift.size();
    d.n_proj = (int32_t)h.proj.size();
    d.acoef_len = aoff;
    d.hc_len = hc_len;
    d.lw_len = (int32_t)h.lw.size();
    d.pw_len = (int32_t)h.pw.size();
    d.wrow = wrow;
    d.lds_bytes = bestBytes;
    d.n_bcol = (int32_t)(h.bcol.size() / 2);
    d.flags = flags;
    append_column_labels(L1, S, h.lab);
    append_column_labels(L2, S, h.lab);
    append_column_labels(Lo, S, h.lab);
    pr->n_theta = nt;
    pr->n_phi = Phi;

    // model counts per pair (what include/istp.h documents)
    const double fl_lift = 2.0 * NC * R * ((double)(L1 + 1) * (L1 + 1) + (double)(L2 + 1) * (L2 + 1));
    const double fl_syn = 2.0 * NC * R * fft_flops(Phi);
    // products per point and hemisphere: one complex product (spin 0); six
    // products and three differences (spin 1); nineteen products, each scaled by
    // a real constant, summed into five components (spin 2)
    const double pp = S == ISTP_GAUNT ? 6.0 : (S == ISTP_VECTOR ? 6 * 6.0 + 3 * 2.0 : 19 * 8.0 + 14 * 2.0);
    const double fl_prod = (double)R * (Phi / 2 + 1) * 2 * pp;
    const double fl_ana = (double)NC * R * fft_flops(Phi);
    const double fl_proj = 2.0 * NC * R * (double)no;
    const double fl_rec = S == ISTP_GAUNT ? 0.0 : 2.0 * NC * (double)nout;
    pr->flops_per_pair = fl_lift + fl_syn + fl_prod + fl_ana + fl_proj + fl_rec;
    pr->bytes_per_pair = (double)(d.nin + d.nin2 + d.nout) * sizeof(T);
    return CGTP_OK;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

template <typename T>
int upload(istp_prod* p, const Host<T>& h, istp::IstpTables<T>* tb) {
    struct Part { const void* src; size_t bytes; size_t off; };
    Part parts[] = {
        {h.lw.data(), h.lw.size() * sizeof(T), 0},
        {h.pw.data(), h.pw.size() * sizeof(T), 0},
        {h.tw.data(), h.tw.size() * sizeof(T), 0},
        {h.liftcg.data(), h.liftcg.size() * sizeof(T), 0},
        {h.coef.data(), h.coef.size() * sizeof(T), 0},
        {h.coefi.data(), h.coefi.size() * sizeof(int32_t), 0},
        {h.lift.data(), h.lift.size() * sizeof(istp::LiftTile), 0},
        {h.proj.data(), h.proj.size() * sizeof(istp::ProjTile), 0},
        {&p->desc, sizeof(istp::IstpDesc), 0},
        {h.bcol.data(), h.bcol.size() * sizeof(int32_t), 0},
        {h.lab.data(), h.lab.size() * sizeof(int32_t), 0},
    };
    size_t total = 0;
    for (auto& pt : parts) {
        pt.off = total;
        total = align_up(total + pt.bytes, 256);
    }
    std::vector<char> host(total, 0);
    for (const auto& pt : parts)
        if (pt.bytes) std::memcpy(host.data() + pt.off, pt.src, pt.bytes);
    hipError_t e = hipMalloc(&p->dmem, total);
    if (e != hipSuccess) {
        cgtp::set_last_hip_error((int)e);
        p->dmem = nullptr;
        return e == hipErrorOutOfMemory ? CGTP_ENOMEM : CGTP_EHIP;
    }
    e = hipMemcpy(p->dmem, host.data(), total, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        cgtp::set_last_hip_error((int)e);
        (void)hipFree(p->dmem);
        p->dmem = nullptr;
        return CGTP_EHIP;
    }
    char* base = (char*)p->dmem;
    tb->lw = (const T*)(base + parts[0].off);
    tb->pw = (const T*)(base + parts[1].off);
    tb->tw = (const T*)(base + parts[2].off);
    tb->liftcg = (const T*)(base + parts[3].off);
    tb->coef = (const T*)(base + parts[4].off);
    tb->coefi = (const int32_t*)(base + parts[5].off);
    tb->lift = (const istp::LiftTile*)(base + parts[6].off);
    tb->proj = (const istp::ProjTile*)(base + parts[7].off);
    tb->desc = (const istp::IstpDesc*)(base + parts[8].off);
    tb->bcol = (const int2*)(base + parts[9].off);
    tb->lab = (const int32_t*)(base + parts[10].off);
    p->ok = true;
    return CGTP_OK;
}

template <typename T> istp::IstpTables<T>* tables_of(istp_prod* pr);
template <> istp::IstpTables<float>* tables_of<float>(istp_prod* pr) { return &pr->tf; }
template <> istp::IstpTables<double>* tables_of<double>(istp_prod* pr) { return &pr->td; }

// Builds and uploads one product; a product outside the kernel's limits is
// left unbuilt (CGTP_EUNSUP) without an allocation.
template <typename T>
int make_prod(int L1, int L2, int Lo, int S, int flags, istp_prod* pr, bool upload_tables) {
    Host<T> h;
    const int rc = build<T>(L1, L2, Lo, S, flags, pr, h);
    if (rc != CGTP_OK || !upload_tables) return rc;
    return upload<T>(pr, h, tables_of<T>(pr));
}

void free_prod(istp_prod* pr, int* rc) {
    if (pr->dmem) {
        const hipError_t e = hipFree(pr->dmem);
        if (e != hipSuccess) {
            cgtp::set_last_hip_error((int)e);
            *rc = CGTP_EHIP;
        }
        pr->dmem = nullptr;
    }
}

int launch_prod(const istp_plan_s* plan, const istp_prod& pr, int flags, const void* a, const void* b, void* out,
                int64_t N, void* stream) {
    istp::IstpDesc d = pr.desc;
    if (d.flags & istp::kRealBasis) {   // the real-basis products run their own kernel
        const int er = plan->dtype == CGTP_FP32
                           ? istp::launch_istp_real_f32(pr.tf, d, (const float*)a, (const float*)b, (float*)out, N,
                                                        stream)
                           : istp::launch_istp_real_f64(pr.td, d, (const double*)a, (const double*)b, (double*)out,
                                                        N, stream);
        if (er != 0) {
            cgtp::set_last_hip_error(er);
            return CGTP_EHIP;
        }
        return CGTP_OK;
    }
    d.flags = flags;
    const bool t2 = d.spin == ISTP_TENSOR;
    const int err =
        plan->dtype == CGTP_FP32
            ? (t2 ? istp::launch_istp_tensor_f32 : istp::launch_istp_f32)(pr.tf, d, (const float*)a, (const float*)b,
                                                                          (float*)out, N, stream)
            : (t2 ? istp::launch_istp_tensor_f64 : istp::launch_istp_f64)(pr.td, d, (const double*)a,
                                                                          (const double*)b, (double*)out, N, stream);
    if (err != 0) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

int current_device_is(int device) {
    int dev = -1;
    const hipError_t de = hipGetDevice(&dev);
    if (de != hipSuccess) {
        cgtp::set_last_hip_error((int)de);
        return CGTP_EHIP;
    }
    return dev == device ? CGTP_OK : CGTP_EINVAL;
}

}  // namespace

extern "C" {

int64_t istp_num_inputs(int32_t L, int32_t spin) { return row_size(L, spin); }

int64_t istp_num_outputs(int32_t L, int32_t spin) { return L < 0 ? -1 : row_size(2 * L, spin); }

int64_t istp_label_offset(int32_t spin, int32_t j, int32_t l) { return label_offset(spin, j, l); }

int64_t istp_label_index(int32_t spin, int32_t j, int32_t l) { return label_index(spin, j, l); }

int64_t istp_num_labels(int32_t L, int32_t spin) { return num_labels(L, spin); }

static int check_plan_args(int32_t L, int32_t spin, int32_t dtype) {
    if (L < 0 || spin < ISTP_GAUNT || spin > ISTP_TENSOR) return CGTP_EINVAL;
    if (dtype != CGTP_FP32 && dtype != CGTP_FP64) return CGTP_EDTYPE;
    if (spin == ISTP_TENSOR && L > (dtype == CGTP_FP32 ? ISTP_TENSOR_MAX_L_FP32 : ISTP_TENSOR_MAX_L_FP64))
        return CGTP_EUNSUP;
    if (L > (dtype == CGTP_FP32 ? ISTP_MAX_L_FP32 : ISTP_MAX_L_FP64)) return CGTP_EUNSUP;
    return CGTP_OK;
}

int istp_plan(int32_t L, int32_t spin, int32_t dtype, istp_plan_t* plan_out) {
    if (!plan_out) return CGTP_EINVAL;
    int rc = check_plan_args(L, spin, dtype);
    if (rc != CGTP_OK) return rc;
    istp_plan_s* p = new (std::nothrow) istp_plan_s();
    if (!p) return CGTP_ENOMEM;
    p->L = L;
    p->spin = spin;
    p->dtype = dtype;
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        cgtp::set_last_hip_error((int)e);
        delete p;
        return CGTP_EHIP;
    }
    rc = dtype == CGTP_FP32 ? make_prod<float>(L, L, 2 * L, spin, 0, &p->fwd, true)
                            : make_prod<double>(L, L, 2 * L, spin, 0, &p->fwd, true);
    if (rc == CGTP_OK) {
        // the gradients' product; outside the kernel's limits it stays unbuilt
        const int rb = dtype == CGTP_FP32
                           ? make_prod<float>(2 * L, L, L, spin, istp::kReverseSecond, &p->bwd, true)
                           : make_prod<double>(2 * L, L, L, spin, istp::kReverseSecond, &p->bwd, true);
        if (rb != CGTP_OK && rb != CGTP_EUNSUP) rc = rb;
    }
    if (rc == CGTP_OK && spin != ISTP_TENSOR) {
        // the real-basis products (forward; spin 0 also the gradients); outside the
        // kernel's limits they stay unbuilt and the real-basis calls take three products
        const int f = istp::kRealBasis;
        int rr = dtype == CGTP_FP32 ? make_prod<float>(L, L, 2 * L, spin, f, &p->rfwd, true)
                                    : make_prod<double>(L, L, 2 * L, spin, f, &p->rfwd, true);
        if (rr != CGTP_OK && rr != CGTP_EUNSUP) rc = rr;
        if (rc == CGTP_OK && spin == ISTP_GAUNT && p->bwd.ok) {
            rr = dtype == CGTP_FP32 ? make_prod<float>(2 * L, L, L, spin, f, &p->rbwd, true)
                                    : make_prod<double>(2 * L, L, L, spin, f, &p->rbwd, true);
            if (rr != CGTP_OK && rr != CGTP_EUNSUP) rc = rr;
        }
    }
    if (rc != CGTP_OK) {
        int ignored = CGTP_OK;
        free_prod(&p->fwd, &ignored);
        free_prod(&p->bwd, &ignored);
        free_prod(&p->rfwd, &ignored);
        free_prod(&p->rbwd, &ignored);
        delete p;
        return rc;
    }
    *plan_out = p;
    return CGTP_OK;
}

int istp_plan_describe(int32_t L, int32_t spin, int32_t dtype, int32_t* desc_out) {
    if (!desc_out) return CGTP_EINVAL;
    int rc = check_plan_args(L, spin, dtype);
    if (rc != CGTP_OK) return rc;
    istp_prod pr, pb;
    rc = dtype == CGTP_FP32 ? make_prod<float>(L, L, 2 * L, spin, 0, &pr, false)
                            : make_prod<double>(L, L, 2 * L, spin, 0, &pr, false);
    if (rc != CGTP_OK) return rc;
    static_assert(sizeof(istp::IstpDesc) == 24 * sizeof(int32_t), "descriptor layout");
    std::memcpy(desc_out, &pr.desc, sizeof(istp::IstpDesc));
    // the gradients' product follows when it is within the kernel's limits
    rc = dtype == CGTP_FP32 ? make_prod<float>(2 * L, L, L, spin, istp::kReverseSecond, &pb, false)
                            : make_prod<double>(2 * L, L, L, spin, istp::kReverseSecond, &pb, false);
    if (rc == CGTP_OK) std::memcpy(desc_out + 24, &pb.desc, sizeof(istp::IstpDesc));
    else std::memset(desc_out + 24, 0, sizeof(istp::IstpDesc));
    return CGTP_OK;
}

int istp_destroy(istp_plan_t plan) {
    if (!plan) return CGTP_OK;
    int rc = CGTP_OK;
    free_prod(&plan->fwd, &rc);
    free_prod(&plan->bwd, &rc);
    free_prod(&plan->rfwd, &rc);
    free_prod(&plan->rbwd, &rc);
    delete plan;
    return rc;
}

int istp_plan_query(istp_plan_t plan, int32_t* n_theta, int32_t* n_phi, int32_t* pairs_per_group,
                    double* flops_per_pair, double* bytes_per_pair) {
    if (!plan) return CGTP_EINVAL;
    if (n_theta) *n_theta = plan->fwd.n_theta;
    if (n_phi) *n_phi = plan->fwd.n_phi;
    if (pairs_per_group) *pairs_per_group = plan->fwd.desc.pairs;
    if (flops_per_pair) *flops_per_pair = plan->fwd.flops_per_pair;
    if (bytes_per_pair) *bytes_per_pair = plan->fwd.bytes_per_pair;
    return CGTP_OK;
}

int istp_backward_query(istp_plan_t plan, int32_t* pairs_per_group, double* flops_per_pair,
                        double* bytes_per_pair) {
    if (!plan) return CGTP_EINVAL;
    if (!plan->bwd.ok) return CGTP_EUNSUP;
    if (pairs_per_group) *pairs_per_group = plan->bwd.desc.pairs;
    // both gradients: two launches of the gradients' product
    if (flops_per_pair) *flops_per_pair = 2 * plan->bwd.flops_per_pair;
    if (bytes_per_pair) *bytes_per_pair = 2 * plan->bwd.bytes_per_pair;
    return CGTP_OK;
}

int istp_forward(istp_plan_t plan, const void* x1, const void* x2, void* out, int64_t N, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !out) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    if ((uint64_t)N > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
    if (overlaps(out, bout, x1, bin) || overlaps(out, bout, x2, bin)) return CGTP_EINVAL;
    const int rc = current_device_is(plan->device);
    if (rc != CGTP_OK) return rc;
    return launch_prod(plan, plan->fwd, 0, x1, x2, out, N, hip_stream);
}

int istp_forward_weighted(istp_plan_t plan, const void* x1, const void* x2, const void* w1, const void* w2,
                          const void* wo, void* out, int64_t N, const istp_channels* ch, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    const int32_t C = ch ? ch->channels : 1;
    if (C < 1 || (ch && ((ch->x2_shared & ~1) || (ch->weights_per_pair & ~1) || ch->reserved))) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !out) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    if (((uintptr_t)w1 | (uintptr_t)w2 | (uintptr_t)wo) & (esz - 1)) return CGTP_EINVAL;
    const bool shared = ch && ch->x2_shared, per_row = ch && ch->weights_per_pair;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    const int64_t nl = num_labels(plan->L, plan->spin), nlo = num_labels(2 * plan->L, plan->spin);
    if (N > INT64_MAX / C) return CGTP_EINVAL;
    const int64_t rows = N * C;
    if ((uint64_t)rows > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const int64_t wrows = per_row ? rows : C;
    const size_t bin = (size_t)rows * nin * esz, bin2 = (size_t)(shared ? N : rows) * nin * esz;
    const size_t bout = (size_t)rows * nout * esz;
    const size_t bw = (size_t)wrows * nl * esz, bwo = (size_t)wrows * nlo * esz;
    if (overlaps(out, bout, x1, bin) || overlaps(out, bout, x2, bin2) || (w1 && overlaps(out, bout, w1, bw)) ||
        (w2 && overlaps(out, bout, w2, bw)) || (wo && overlaps(out, bout, wo, bwo)))
        return CGTP_EINVAL;
    const int rc = current_device_is(plan->device);
    if (rc != CGTP_OK) return rc;
    istp::IstpDesc d = plan->fwd.desc;
    d.flags = 0;
    const int32_t flags = (shared ? istp::kChanX2Shared : 0) | (per_row ? istp::kChanPerRow : 0);
    int err;
    if (plan->dtype == CGTP_FP32) {
        const istp::IstpChan<float> c{(const float*)w1, (const float*)w2, (const float*)wo, C, flags,
                                      (int32_t)nl, (int32_t)nl, (int32_t)nlo};
        err = (plan->spin == ISTP_TENSOR ? istp::launch_istp_channels_tensor_f32 : istp::launch_istp_channels_f32)(
            plan->fwd.tf, d, (const float*)x1, (const float*)x2, (float*)out, rows, c, hip_stream);
    } else {
        const istp::IstpChan<double> c{(const double*)w1, (const double*)w2, (const double*)wo, C, flags,
                                       (int32_t)nl, (int32_t)nl, (int32_t)nlo};
        err = (plan->spin == ISTP_TENSOR ? istp::launch_istp_channels_tensor_f64 : istp::launch_istp_channels_f64)(
            plan->fwd.td, d, (const double*)x1, (const double*)x2, (double*)out, rows, c, hip_stream);
    }
    if (err != 0) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

// Real-basis Gaunt product: workspace of the converted inputs (real part,
// imaginary part and their sum, for each input) and two products (the third
// lands in out), each 256-byte aligned.
static size_t real_part_bytes(size_t n) { return (n + 255) / 256 * 256; }

int64_t istp_real_workspace_bytes(istp_plan_t plan, int64_t N) {
    if (!plan || N < 0) return -1;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    if ((uint64_t)N > (uint64_t)(INT64_MAX / 16 / (int64_t)(nout * esz))) return -1;
    // spin 0 runs the real-basis kernel (no workspace) where it is built, else
    // forms the first product in out and reads it back in place; spin 1 and 2
    // keep all three products in the workspace
    if (plan->rfwd.ok) return 0;
    const size_t nprod = plan->spin == ISTP_GAUNT ? 2 : 3;
    return (int64_t)(6 * real_part_bytes((size_t)N * nin * esz) + nprod * real_part_bytes((size_t)N * nout * esz));
}

int istp_forward_real(istp_plan_t plan, const void* x1, const void* x2, void* out, int64_t N, void* workspace,
                      int64_t workspace_bytes, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (plan->rfwd.ok) {
        // one launch of the real-basis kernel; the workspace is not used
        if (!x1 || !x2 || !out || workspace_bytes < 0) return CGTP_EINVAL;
        if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
        const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
        const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
        if ((uint64_t)N > (uint64_t)(INT64_MAX / 16 / (int64_t)(nout * esz))) return CGTP_EINVAL;
        const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
        if (overlaps(out, bout, x1, bin) || overlaps(out, bout, x2, bin)) return CGTP_EINVAL;
        const int rc0 = current_device_is(plan->device);
        if (rc0 != CGTP_OK) return rc0;
        return launch_prod(plan, plan->rfwd, 0, x1, x2, out, N, hip_stream);
    }
    if (!x1 || !x2 || !out || !workspace) return CGTP_EINVAL;
    if ((((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) || ((uintptr_t)workspace & 255)) return CGTP_EINVAL;
    const int64_t need = istp_real_workspace_bytes(plan, N);
    if (need < 0 || workspace_bytes < need) return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
    if (overlaps(out, bout, x1, bin) || overlaps(out, bout, x2, bin) || overlaps(out, bout, workspace, need) ||
        overlaps(workspace, need, x1, bin) || overlaps(workspace, need, x2, bin))
        return CGTP_EINVAL;
    int rc = current_device_is(plan->device);
    if (rc != CGTP_OK) return rc;
    char* w = (char*)workspace;
    const size_t pin = real_part_bytes(bin), pout = real_part_bytes(bout);
    void* re1 = w;
    void* im1 = w + pin;
    void* sm1 = w + 2 * pin;
    void* re2 = w + 3 * pin;
    void* im2 = w + 4 * pin;
    void* sm2 = w + 5 * pin;
    void* pbb = w + 6 * pin;
    void* pss = w + 6 * pin + pout;
    const int Lo = 2 * plan->L;
    int err;
    if (plan->spin != ISTP_GAUNT) {
        // spin 1 and 2: per-label phases; the three products in the workspace
        const int sp = plan->spin;
        void* paa = w + 6 * pin + 2 * pout;
        if (plan->dtype == CGTP_FP32) {
            err = istp::launch_real_to_complex_spin_f32((const float*)x1, (float*)re1, (float*)im1, (float*)sm1, N,
                                                        (int)nin, sp, hip_stream);
            if (!err)
                err = istp::launch_real_to_complex_spin_f32((const float*)x2, (float*)re2, (float*)im2, (float*)sm2,
                                                            N, (int)nin, sp, hip_stream);
        } else {
            err = istp::launch_real_to_complex_spin_f64((const double*)x1, (double*)re1, (double*)im1, (double*)sm1,
                                                        N, (int)nin, sp, hip_stream);
            if (!err)
                err = istp::launch_real_to_complex_spin_f64((const double*)x2, (double*)re2, (double*)im2,
                                                            (double*)sm2, N, (int)nin, sp, hip_stream);
        }
        if (err) {
            cgtp::set_last_hip_error(err);
            return CGTP_EHIP;
        }
        rc = launch_prod(plan, plan->fwd, 0, re1, re2, paa, N, hip_stream);
        if (rc == CGTP_OK) rc = launch_prod(plan, plan->fwd, 0, im1, im2, pbb, N, hip_stream);
        if (rc == CGTP_OK) rc = launch_prod(plan, plan->fwd, 0, sm1, sm2, pss, N, hip_stream);
        if (rc != CGTP_OK) return rc;
        err = plan->dtype == CGTP_FP32
                  ? istp::launch_real_from_complex_spin_f32((float*)out, (const float*)paa, (const float*)pbb,
                                                            (const float*)pss, N, (int)nout, sp, hip_stream)
                  : istp::launch_real_from_complex_spin_f64((double*)out, (const double*)paa, (const double*)pbb,
                                                            (const double*)pss, N, (int)nout, sp, hip_stream);
        if (err) {
            cgtp::set_last_hip_error(err);
            return CGTP_EHIP;
        }
        return CGTP_OK;
    }
    if (plan->dtype == CGTP_FP32) {
        err = istp::launch_real_to_complex_f32((const float*)x1, (float*)re1, (float*)im1, (float*)sm1, N, (int)nin,
                                               hip_stream);
        if (!err)
            err = istp::launch_real_to_complex_f32((const float*)x2, (float*)re2, (float*)im2, (float*)sm2, N,
                                                   (int)nin, hip_stream);
    } else {
        err = istp::launch_real_to_complex_f64((const double*)x1, (double*)re1, (double*)im1, (double*)sm1, N,
                                               (int)nin, hip_stream);
        if (!err)
            err = istp::launch_real_to_complex_f64((const double*)x2, (double*)re2, (double*)im2, (double*)sm2, N,
                                                   (int)nin, hip_stream);
    }
    if (err) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    // P(a1, a2) into out, then P(b1, b2) and P(a1 + b1, a2 + b2)
    rc = launch_prod(plan, plan->fwd, 0, re1, re2, out, N, hip_stream);
    if (rc == CGTP_OK) rc = launch_prod(plan, plan->fwd, 0, im1, im2, pbb, N, hip_stream);
    if (rc == CGTP_OK) rc = launch_prod(plan, plan->fwd, 0, sm1, sm2, pss, N, hip_stream);
    if (rc != CGTP_OK) return rc;
    err = plan->dtype == CGTP_FP32
              ? istp::launch_real_from_complex_f32((float*)out, (const float*)pbb, (const float*)pss, N, Lo,
                                                   hip_stream)
              : istp::launch_real_from_complex_f64((double*)out, (const double*)pbb, (const double*)pss, N, Lo,
                                                   hip_stream);
    if (err) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

// Gradients in the real basis: the real Gaunt coefficients (integrals of three
// real harmonics) are fully symmetric, so grad_x1 = Q(g, x2) and grad_x2 =
// Q(g, x1) with Q the real-basis product of a degree-2L and a degree-L row
// projected on degrees <= L (the gradient product's grid, no time reversal).
// Workspace per gradient: the converted upstream gradient (three rows of
// (2L+1)^2), the converted input (three rows of (L+1)^2), two products.
int64_t istp_real_backward_workspace_bytes(istp_plan_t plan, int64_t N) {
    if (!plan || N < 0 || plan->spin != ISTP_GAUNT || !plan->bwd.ok) return -1;
    if (plan->rbwd.ok) return 0;   // the real-basis kernel: no workspace
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t ng = (size_t)plan->fwd.desc.nout, nin = (size_t)plan->fwd.desc.nin;
    if ((uint64_t)N > (uint64_t)(INT64_MAX / 16 / (int64_t)(ng * esz))) return -1;
    return (int64_t)(3 * real_part_bytes((size_t)N * ng * esz) + 5 * real_part_bytes((size_t)N * nin * esz));
}

static int real_bwd_one(istp_plan_t plan, const void* g, const void* x, void* grad, int64_t N, char* w,
                        void* stream) {
    if (plan->rbwd.ok) return launch_prod(plan, plan->rbwd, 0, g, x, grad, N, stream);
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t ng = (size_t)plan->fwd.desc.nout, nin = (size_t)plan->fwd.desc.nin;
    const size_t pg = real_part_bytes((size_t)N * ng * esz), px = real_part_bytes((size_t)N * nin * esz);
    void* ga = w;
    void* gb = w + pg;
    void* gs = w + 2 * pg;
    void* xa = w + 3 * pg;
    void* xb = w + 3 * pg + px;
    void* xs = w + 3 * pg + 2 * px;
    void* pbb = w + 3 * pg + 3 * px;
    void* pss = w + 3 * pg + 4 * px;
    int err = plan->dtype == CGTP_FP32
                  ? istp::launch_real_to_complex_f32((const float*)g, (float*)ga, (float*)gb, (float*)gs, N, (int)ng,
                                                     stream)
                  : istp::launch_real_to_complex_f64((const double*)g, (double*)ga, (double*)gb, (double*)gs, N,
                                                     (int)ng, stream);
    if (!err)
        err = plan->dtype == CGTP_FP32
                  ? istp::launch_real_to_complex_f32((const float*)x, (float*)xa, (float*)xb, (float*)xs, N,
                                                     (int)nin, stream)
                  : istp::launch_real_to_complex_f64((const double*)x, (double*)xa, (double*)xb, (double*)xs, N,
                                                     (int)nin, stream);
    if (err) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    int rc = launch_prod(plan, plan->bwd, 0, ga, xa, grad, N, stream);
    if (rc == CGTP_OK) rc = launch_prod(plan, plan->bwd, 0, gb, xb, pbb, N, stream);
    if (rc == CGTP_OK) rc = launch_prod(plan, plan->bwd, 0, gs, xs, pss, N, stream);
    if (rc != CGTP_OK) return rc;
    err = plan->dtype == CGTP_FP32
              ? istp::launch_real_from_complex_f32((float*)grad, (const float*)pbb, (const float*)pss, N, plan->L,
                                                   stream)
              : istp::launch_real_from_complex_f64((double*)grad, (const double*)pbb, (const double*)pss, N, plan->L,
                                                   stream);
    if (err) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

int istp_backward_real(istp_plan_t plan, const void* x1, const void* x2, const void* grad_out, void* grad_x1,
                       void* grad_x2, int64_t N, void* workspace, int64_t workspace_bytes, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (plan->spin != ISTP_GAUNT || !plan->bwd.ok) return CGTP_EUNSUP;
    if (N == 0) return CGTP_OK;
    const int64_t need = istp_real_backward_workspace_bytes(plan, N);
    if (!x1 || !x2 || !grad_out || (!grad_x1 && !grad_x2) || (need > 0 && !workspace)) return CGTP_EINVAL;
    if ((((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)grad_out | (uintptr_t)grad_x1 | (uintptr_t)grad_x2) & 15) ||
        ((uintptr_t)workspace & 255))
        return CGTP_EINVAL;
    if (need < 0 || workspace_bytes < need) return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
    const void* reads[4] = {x1, x2, grad_out, workspace};
    const size_t rlen[4] = {bin, bin, bout, (size_t)need};
    void* writes[2] = {grad_x1, grad_x2};
    for (void* w : writes) {
        if (!w) continue;
        for (int i = 0; i < 4; ++i)
            if (overlaps(w, bin, reads[i], rlen[i])) return CGTP_EINVAL;
    }
    if (overlaps(workspace, need, x1, bin) || overlaps(workspace, need, x2, bin) ||
        overlaps(workspace, need, grad_out, bout))
        return CGTP_EINVAL;
    if (grad_x1 && grad_x2 && overlaps(grad_x1, bin, grad_x2, bin)) return CGTP_EINVAL;
    int rc = current_device_is(plan->device);
    if (rc != CGTP_OK) return rc;
    if (grad_x1) rc = real_bwd_one(plan, grad_out, x2, grad_x1, N, (char*)workspace, hip_stream);
    if (rc == CGTP_OK && grad_x2) rc = real_bwd_one(plan, grad_out, x1, grad_x2, N, (char*)workspace, hip_stream);
    return rc;
}

// Gradients of the channel-wise product out = wo . P(w1 . x1, w2 . x2) (x2 per
// channel): grad_x1 = w1 . P'(wo . g, w2 . x2~), grad_x2 = +-w2 . P'(wo . g, w1 . x1~),
// P' the gradient product; the channel kernel applies the three weights with
// their roles exchanged.
int istp_backward_weighted(istp_plan_t plan, const void* x1, const void* x2, const void* w1, const void* w2,
                           const void* wo, const void* grad_out, void* grad_x1, void* grad_x2, int64_t N,
                           const istp_channels* ch, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (!plan->bwd.ok || plan->bwd.desc.L + 1 > 4 * istp::kMaxLiftSteps) return CGTP_EUNSUP;
    const int32_t C = ch ? ch->channels : 1;
    if (C < 1 || (ch && ((ch->x2_shared & ~1) || (ch->weights_per_pair & ~1) || ch->reserved))) return CGTP_EINVAL;
    if (ch && ch->x2_shared) return CGTP_EUNSUP;   // its gradient sums over the channels
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !grad_out || (!grad_x1 && !grad_x2)) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)grad_out | (uintptr_t)grad_x1 | (uintptr_t)grad_x2) & 15)
        return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    if (((uintptr_t)w1 | (uintptr_t)w2 | (uintptr_t)wo) & (esz - 1)) return CGTP_EINVAL;
    if (N > INT64_MAX / C) return CGTP_EINVAL;
    const int64_t rows = N * C;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    if ((uint64_t)rows > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const bool per_row = ch && ch->weights_per_pair;
    const int64_t nl = num_labels(plan->L, plan->spin), nlo = num_labels(2 * plan->L, plan->spin);
    const int64_t wrows = per_row ? rows : C;
    const size_t bin = (size_t)rows * nin * esz, bout = (size_t)rows * nout * esz;
    const void* reads[6] = {x1, x2, grad_out, w1, w2, wo};
    const size_t rlen[6] = {bin, bin, bout, (size_t)(wrows * nl) * esz, (size_t)(wrows * nl) * esz,
                            (size_t)(wrows * nlo) * esz};
    void* writes[2] = {grad_x1, grad_x2};
    for (void* w : writes) {
        if (!w) continue;
        for (int i = 0; i < 6; ++i)
            if (reads[i] && overlaps(w, bin, reads[i], rlen[i])) return CGTP_EINVAL;
    }
    if (grad_x1 && grad_x2 && overlaps(grad_x1, bin, grad_x2, bin)) return CGTP_EINVAL;
    int rc = current_device_is(plan->device);
    if (rc != CGTP_OK) return rc;
    const int32_t flags = per_row ? istp::kChanPerRow : 0;
    auto one = [&](const void* xo, const void* w_other, const void* w_self, void* grad, int extra) -> int {
        istp::IstpDesc d = plan->bwd.desc;
        d.flags = istp::kReverseSecond | extra;
        int err;
        const bool t2 = plan->spin == ISTP_TENSOR;
        if (plan->dtype == CGTP_FP32) {
            const istp::IstpChan<float> c{(const float*)wo, (const float*)w_other, (const float*)w_self, C, flags,
                                          (int32_t)nlo, (int32_t)nl, (int32_t)nl};
            err = (t2 ? istp::launch_istp_channels_tensor_f32 : istp::launch_istp_channels_f32)(
                plan->bwd.tf, d, (const float*)grad_out, (const float*)xo, (float*)grad, rows, c, hip_stream);
        } else {
            const istp::IstpChan<double> c{(const double*)wo, (const double*)w_other, (const double*)w_self, C,
                                           flags, (int32_t)nlo, (int32_t)nl, (int32_t)nl};
            err = (t2 ? istp::launch_istp_channels_tensor_f64 : istp::launch_istp_channels_f64)(
                plan->bwd.td, d, (const double*)grad_out, (const double*)xo, (double*)grad, rows, c, hip_stream);
        }
        if (err != 0) {
            cgtp::set_last_hip_error(err);
            return CGTP_EHIP;
        }
        return CGTP_OK;
    };
    if (grad_x1) rc = one(x2, w2, w1, grad_x1, 0);
    if (rc == CGTP_OK && grad_x2) rc = one(x1, w1, w2, grad_x2, plan->spin == ISTP_VECTOR ? istp::kNegate : 0);
    return rc;
}

int istp_backward(istp_plan_t plan, const void* x1, const void* x2, const void* grad_out, void* grad_x1,
                  void* grad_x2, int64_t N, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (!plan->bwd.ok) return CGTP_EUNSUP;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !grad_out || (!grad_x1 && !grad_x2)) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)grad_out | (uintptr_t)grad_x1 | (uintptr_t)grad_x2) & 15)
        return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)plan->fwd.desc.nin, nout = (size_t)plan->fwd.desc.nout;
    if ((uint64_t)N > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
    const void* reads[3] = {x1, x2, grad_out};
    const size_t rlen[3] = {bin, bin, bout};
    void* writes[2] = {grad_x1, grad_x2};
    for (void* w : writes) {
        if (!w) continue;
        for (int i = 0; i < 3; ++i)
            if (overlaps(w, bin, reads[i], rlen[i])) return CGTP_EINVAL;
    }
    if (grad_x1 && grad_x2 && overlaps(grad_x1, bin, grad_x2, bin)) return CGTP_EINVAL;
    int rc = current_device_is(plan->device);
    if (rc != CGTP_OK) return rc;
    // d/dx1 <g, z(x1, x2)> = P(g, reversed x2); for x2 the roles swap, and the
    // vector product changes sign under the swap
    if (grad_x1) rc = launch_prod(plan, plan->bwd, istp::kReverseSecond, grad_out, x2, grad_x1, N, hip_stream);
    if (rc == CGTP_OK && grad_x2)
        rc = launch_prod(plan, plan->bwd, istp::kReverseSecond | (plan->spin == ISTP_VECTOR ? istp::kNegate : 0),
                         grad_out, x1, grad_x2, N, hip_stream);
    return rc;
}

}  // extern "C"

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
#include <new>
#include <vector>

#include "../../include/istp.h"
#include "cgtp_internal.h"
#include "istp_internal.h"

struct istp_plan_s {
    int L = 0, spin = 0, dtype = 0, device = 0;
    istp::IstpDesc desc{};
    void* dmem = nullptr;
    size_t dbytes = 0;
    istp::IstpTables<float> tf{};
    istp::IstpTables<double> td{};
    int n_theta = 0, n_phi = 0;
    double flops_per_pair = 0, bytes_per_pair = 0;
};

namespace {

const double kPi = 3.14159265358979323846264338327950288;

int64_t label_offset(int spin, int j, int l) {
    if (l < 0 || j < 0) return -1;
    if (spin == ISTP_GAUNT) return j == l ? (int64_t)l * l : -1;
    if (spin != ISTP_VECTOR || std::abs(j - l) > 1 || j + l < 1) return -1;
    const int jj = j - l + 1;
    return 3LL * l * l + (jj == 0 ? 0 : (jj == 1 ? 2 * l - 1 : 4 * l));
}

int64_t row_size(int L, int spin) {
    if (L < 0 || (spin != ISTP_GAUNT && spin != ISTP_VECTOR)) return -1;
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
int lift_ncol(int NC, int P, int am) { return (am ? 2 : 1) * 2 * NC * P; }

int acoef_len(int L, int NC, int P) {
    int n = 0;
    for (int am = 0; am <= L; ++am) n += lift_kp(L, am) * istp::istp_cstride(lift_ncol(NC, P, am));
    return n;
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
};

template <typename T>
int build(istp_plan_s* p, Host<T>& h) {
    const int L = p->L, S = p->spin, NC = 2 * S + 1, Lo = 2 * L;
    const int nt = 2 * L + 2, R = L + 1;
    const int Phi = smallest_2a3b(4 * L + 1);
    int A = 0, B = 0;
    if (!cgtp::fft_factors(Phi, &A, &B)) return CGTP_EUNSUP;

    int nproj = 0;
    for (int am = 0; am <= Lo; ++am)
        for (int par = 0; par < 2; ++par) nproj += (proj_rows(Lo, am, par) + 15) / 16;
    if (nproj > istp::MaxTiles<T>::value * istp::kWaves) return CGTP_EUNSUP;

    // Pairs per work-group and ring pairs per group: the most pairs that fit in
    // LDS with the projection's columns (sign, component, pair) on one MFMA tile
    // (each pair more fills more of the lift's and the projection's columns),
    // then the most ring pairs (more units fill more of the work-group's
    // threads in the transform phases and take fewer passes over the rings).
    const int hc_len = NC * (Lo + 1) * (Lo + 1);
    int bestP = 0, bestG = 0, bestBytes = 0;
    const int nin = (int)row_size(L, S);
    for (int P : {8, 4, 2, 1}) {
        if (2 * NC * P > 16) continue;
        // inputs and couplings are staged with one batch of loads per thread
        const int stage = 2 * P * nin + (S ? 9 * (L + 1) * (L + 1) : 0);
        if (stage > istp::kStageLoads * istp::kThreads) continue;
        for (int G : {16, 12, 8, 4}) {
            const istp::IstpLayout ly = istp::istp_layout<T>(A, B, NC, G, P, acoef_len(L, NC, P), hc_len,
                                                             istp::istp_stage_len(P, nin, L, S), nproj);
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
    const int wrow = 16 * ((L + 1 + 15) / 16);   // most rows: am = 0, even parity, L + 1 of them

    std::vector<double> xs(nt), ws(nt);
    if (cgtp_gauss_legendre(nt, xs.data(), ws.data()) != CGTP_OK) return CGTP_EINVAL;
    // rings 0..R-1 are the northern nodes (x > 0); the south ones are their mirrors
    std::vector<std::vector<double>> plm(R);
    for (int r = 0; r < R; ++r) {
        if (!(xs[r] > 0.0)) return CGTP_EINVAL;
        plm[r].assign((Lo + 1) * (Lo + 2) / 2, 0.0);
        cgtp_legendre(Lo, xs[r], plm[r].data());
    }
    auto pbar = [&](int r, int l, int m) { return plm[r][l * (l + 1) / 2 + m]; };

    // lift weights [am][ring][k]: P_{am+k}^{am}(x_ring)
    std::vector<int> lw_off(L + 1);
    for (int am = 0; am <= L; ++am) {
        lw_off[am] = (int)h.lw.size();
        const int kp = lift_kp(L, am);
        for (int r = 0; r < rpad; ++r)
            for (int k = 0; k < kp; ++k) {
                const int l = am + k;
                h.lw.push_back(r < R && l <= L ? (T)pbar(r, l, am) : (T)0);
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
    // lift couplings C^{j, ml+q}_{l, ml, 1, q}, j = l - 1, l, l + 1
    h.liftcg.assign((size_t)9 * (L + 1) * (L + 1), (T)0);
    if (S == ISTP_VECTOR)
        for (int l = 0; l <= L; ++l)
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
    for (int am = 0; am <= L; ++am) {
        const int kp = lift_kp(L, am), ncol = lift_ncol(NC, P, am), cs = istp::istp_cstride(ncol);
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
    if (S == ISTP_GAUNT) {
        for (int l3 = 0; l3 <= Lo; ++l3)
            for (int m3 = -l3; m3 <= l3; ++m3) {
                const int o = l3 * l3 + l3 + m3;
                h.coef[4 * o] = (T)(scale * sgn(m3));
                h.coefi[4 * o] = h.coefi[4 * o + 1] = h.coefi[4 * o + 2] = o;
                h.coefi[4 * o + 3] = 1;
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

    istp::IstpDesc& d = p->desc;
    d.L = L;
    d.Lo = Lo;
    d.spin = S;
    d.C = NC;
    d.R = R;
    d.G = G;
    d.Phi = Phi;
    d.A = A;
    d.B = B;
    d.pairs = P;
    d.nin = (int32_t)row_size(L, S);
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
    p->n_theta = nt;
    p->n_phi = Phi;

    // model counts per pair (what include/istp.h documents)
    const double fl_lift = 2.0 * 2 * NC * R * (double)(L + 1) * (L + 1);
    const double fl_syn = 2.0 * NC * R * fft_flops(Phi);
    const double fl_prod = (double)R * (Phi / 2 + 1) * 2 * (S == ISTP_GAUNT ? 6.0 : 6 * 6.0 + 3 * 2.0);
    const double fl_ana = (double)NC * R * fft_flops(Phi);
    const double fl_proj = 2.0 * NC * R * (double)no;
    const double fl_rec = S == ISTP_GAUNT ? 0.0 : 2.0 * 3 * (double)nout;
    p->flops_per_pair = fl_lift + fl_syn + fl_prod + fl_ana + fl_proj + fl_rec;
    p->bytes_per_pair = (double)(2 * d.nin + d.nout) * sizeof(T);
    return CGTP_OK;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

template <typename T>
int upload(istp_plan_s* p, const Host<T>& h, istp::IstpTables<T>* tb) {
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
    p->dbytes = total;
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
    return CGTP_OK;
}

}  // namespace

extern "C" {

int64_t istp_num_inputs(int32_t L, int32_t spin) { return row_size(L, spin); }

int64_t istp_num_outputs(int32_t L, int32_t spin) { return L < 0 ? -1 : row_size(2 * L, spin); }

int64_t istp_label_offset(int32_t spin, int32_t j, int32_t l) { return label_offset(spin, j, l); }

int istp_plan(int32_t L, int32_t spin, int32_t dtype, istp_plan_t* plan_out) {
    if (!plan_out || L < 0 || (spin != ISTP_GAUNT && spin != ISTP_VECTOR)) return CGTP_EINVAL;
    if (dtype != CGTP_FP32 && dtype != CGTP_FP64) return CGTP_EDTYPE;
    if (L > (dtype == CGTP_FP32 ? ISTP_MAX_L_FP32 : ISTP_MAX_L_FP64)) return CGTP_EUNSUP;
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
    int rc;
    if (dtype == CGTP_FP32) {
        Host<float> h;
        rc = build<float>(p, h);
        if (rc == CGTP_OK) rc = upload<float>(p, h, &p->tf);
    } else {
        Host<double> h;
        rc = build<double>(p, h);
        if (rc == CGTP_OK) rc = upload<double>(p, h, &p->td);
    }
    if (rc != CGTP_OK) {
        delete p;
        return rc;
    }
    *plan_out = p;
    return CGTP_OK;
}

int istp_plan_describe(int32_t L, int32_t spin, int32_t dtype, int32_t* desc_out) {
    if (!desc_out || L < 0 || (spin != ISTP_GAUNT && spin != ISTP_VECTOR)) return CGTP_EINVAL;
    if (dtype != CGTP_FP32 && dtype != CGTP_FP64) return CGTP_EDTYPE;
    if (L > (dtype == CGTP_FP32 ? ISTP_MAX_L_FP32 : ISTP_MAX_L_FP64)) return CGTP_EUNSUP;
    istp_plan_s p;
    p.L = L;
    p.spin = spin;
    p.dtype = dtype;
    int rc;
    if (dtype == CGTP_FP32) {
        Host<float> h;
        rc = build<float>(&p, h);
    } else {
        Host<double> h;
        rc = build<double>(&p, h);
    }
    if (rc != CGTP_OK) return rc;
    static_assert(sizeof(istp::IstpDesc) == 24 * sizeof(int32_t), "descriptor layout");
    std::memcpy(desc_out, &p.desc, sizeof(istp::IstpDesc));
    return CGTP_OK;
}

int istp_destroy(istp_plan_t plan) {
    if (!plan) return CGTP_OK;
    int rc = CGTP_OK;
    if (plan->dmem) {
        hipError_t e = hipFree(plan->dmem);
        if (e != hipSuccess) {
            cgtp::set_last_hip_error((int)e);
            rc = CGTP_EHIP;
        }
    }
    delete plan;
    return rc;
}

int istp_plan_query(istp_plan_t plan, int32_t* n_theta, int32_t* n_phi, int32_t* pairs_per_group,
                    double* flops_per_pair, double* bytes_per_pair) {
    if (!plan) return CGTP_EINVAL;
    if (n_theta) *n_theta = plan->n_theta;
    if (n_phi) *n_phi = plan->n_phi;
    if (pairs_per_group) *pairs_per_group = plan->desc.pairs;
    if (flops_per_pair) *flops_per_pair = plan->flops_per_pair;
    if (bytes_per_pair) *bytes_per_pair = plan->bytes_per_pair;
    return CGTP_OK;
}

int istp_forward(istp_plan_t plan, const void* x1, const void* x2, void* out, int64_t N, void* hip_stream) {
    if (!plan || N < 0) return CGTP_EINVAL;
    if (N == 0) return CGTP_OK;
    if (!x1 || !x2 || !out) return CGTP_EINVAL;
    if (((uintptr_t)x1 | (uintptr_t)x2 | (uintptr_t)out) & 15) return CGTP_EINVAL;
    const size_t esz = plan->dtype == CGTP_FP32 ? 4 : 8;
    const size_t nin = (size_t)plan->desc.nin, nout = (size_t)plan->desc.nout;
    if ((uint64_t)N > (uint64_t)(INT64_MAX / (int64_t)(nout * esz))) return CGTP_EINVAL;
    const size_t bin = (size_t)N * nin * esz, bout = (size_t)N * nout * esz;
    if (overlaps(out, bout, x1, bin) || overlaps(out, bout, x2, bin)) return CGTP_EINVAL;
    int dev = -1;
    const hipError_t de = hipGetDevice(&dev);
    if (de != hipSuccess) {
        cgtp::set_last_hip_error((int)de);
        return CGTP_EHIP;
    }
    if (dev != plan->device) return CGTP_EINVAL;
    const int err = plan->dtype == CGTP_FP32
                        ? istp::launch_istp_f32(plan->tf, plan->desc, (const float*)x1, (const float*)x2,
                                                (float*)out, N, hip_stream)
                        : istp::launch_istp_f64(plan->td, plan->desc, (const double*)x1, (const double*)x2,
                                                (double*)out, N, hip_stream);
    if (err != 0) {
        cgtp::set_last_hip_error(err);
        return CGTP_EHIP;
    }
    return CGTP_OK;
}

}  // extern "C"

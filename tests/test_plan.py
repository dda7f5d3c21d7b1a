"""Host math the plan is built from (no GPU): pinned to sympy, scipy, numpy
and the paper's closed forms, and the method model checked against the oracle.
"""
import math
import re

import numpy as np
import pytest

import oracle
import paper_2602_21466_amd as lib
from method_model import model_cgtp


def test_vector_coupling_closed_forms_match_sympy():
    from sympy.physics.wigner import clebsch_gordan
    for j1 in list(range(0, 6)) + [17, 32, 63]:
        for j in (j1 - 1, j1, j1 + 1):
            if j < 0:
                continue
            for m1 in range(-j1, j1 + 1):
                for q in (-1, 0, 1):
                    want = float(clebsch_gordan(j1, 1, j, m1, q, m1 + q))
                    assert lib.cgtp_cg_vector(j1, m1, q, j, m1 + q) == pytest.approx(want, abs=1e-15)


def test_cg_zero_matches_sympy():
    from sympy.physics.wigner import clebsch_gordan
    for l1, l2, l3 in [(0, 0, 0), (1, 1, 2), (2, 3, 5), (7, 9, 4), (32, 32, 64), (32, 31, 1), (20, 25, 11),
                       (3, 4, 5), (1, 1, 1)]:
        want = float(clebsch_gordan(l1, l2, l3, 0, 0, 0).evalf(30))
        assert lib.cgtp_cg_zero(l1, l2, l3) == pytest.approx(want, abs=1e-15)


def test_ninej_matches_sympy(rng):
    from sympy.physics.wigner import wigner_9j
    cases = [(1, 1, 1, 1, 1, 1, 1, 1, 1), (3, 3, 1, 5, 5, 1, 6, 6, 0), (4, 4, 1, 2, 2, 1, 5, 4, 1),
             (7, 7, 0, 6, 6, 1, 8, 7, 1), (2, 3, 1, 4, 4, 1, 3, 4, 1)]
    for _ in range(15):
        a, b = int(rng.integers(1, 12)), int(rng.integers(1, 12))
        c = int(rng.integers(abs(a - b) + 1, a + b + 1))
        cases.append((a, a, 1, b, b, 1, c, c - 1, 1))
    for args in cases:
        want = float(wigner_9j(*args, prec=30))
        assert lib.cgtp_wigner_9j(*args) == pytest.approx(want, abs=1e-14), args


def _paper_9j_table():
    """Closed forms of {a+lam a 1; b+mu b 1; c+nu c 1} printed in the selection-rule proof
    (Appendix F.2, tables for nu = 1 and nu = -1), transcribed as functions of (a, b, c)."""
    f = math.factorial

    def row_nu1_00(a, b, c):       # lambda = mu = 0, nu = 1
        s = a + b + c
        return 2 * (c + 1) * math.sqrt((s + 2) * (s - 2 * c) * (s - 2 * b + 1) * (s - 2 * a + 1) * f(2 * a - 1) *
                                       f(2 * b - 1) * f(2 * c) / (3 * f(2 * a + 2) * f(2 * b + 2) * f(2 * c + 3)))

    def row_nu1_11(a, b, c):       # lambda = mu = 1, nu = 1
        s = a + b + c
        return -math.sqrt(f(s + 4) * (s - 2 * c + 1) * (s - 2 * b + 1) * (s - 2 * a + 1) * f(2 * a) * f(2 * b) *
                          f(2 * c) / (3 * f(s + 1) * f(2 * a + 3) * f(2 * b + 3) * f(2 * c + 3)))

    def row_num1_00(a, b, c, with_three):   # lambda = mu = 0, nu = -1
        s = a + b + c
        den = (3 if with_three else 1) * f(2 * a + 2) * f(2 * b + 2) * f(2 * c + 1)
        return 2 * c * math.sqrt((s + 1) * (s - 2 * c + 1) * (s - 2 * b) * (s - 2 * a) * f(2 * a - 1) *
                                 f(2 * b - 1) * f(2 * c - 2) / den)
    return row_nu1_00, row_nu1_11, row_num1_00


def test_ninej_against_paper_closed_forms():
    """The 9j rows the VSTP selection-rule proof lists.

    Readings: the (0, 0, -1) row needs a factor 3 in its denominator to agree
    (a dropped 3, as in every other row); the (1, 1, 1) row agrees in magnitude
    but has the opposite overall sign from the standard 9j symbol (sympy agrees
    with the generic sum here).  The proof only uses where the rows vanish, so
    neither changes its argument.  The (0, 0, 1) row is the one the default
    cover's factor uses and it agrees exactly."""
    r00, r11, rm00 = _paper_9j_table()
    for a in range(1, 8):
        for b in range(1, 8):
            for c in range(abs(a - b), a + b + 1):
                if c + 1 <= a + b and abs(a - b) <= c + 1 and c >= 0:
                    assert lib.cgtp_wigner_9j(a, a, 1, b, b, 1, c + 1, c, 1) == pytest.approx(r00(a, b, c), abs=1e-13)
                if abs(a + 1 - b - 1) <= c + 1 <= a + b + 2 and abs(a - b) <= c <= a + b:
                    assert abs(lib.cgtp_wigner_9j(a + 1, a, 1, b + 1, b, 1, c + 1, c, 1)) == pytest.approx(
                        abs(r11(a, b, c)), abs=1e-13)
                if c >= 1 and abs(a - b) <= c - 1:
                    got = lib.cgtp_wigner_9j(a, a, 1, b, b, 1, c - 1, c, 1)
                    assert got == pytest.approx(rm00(a, b, c, True), abs=1e-13)
                    if abs(got) > 1e-6:
                        assert got != pytest.approx(rm00(a, b, c, False), abs=1e-6)


def test_gauss_legendre_matches_numpy():
    for n in (1, 2, 6, 33, 66, 130):
        x, w = lib.cgtp_gauss_legendre(n)
        xr, wr = np.polynomial.legendre.leggauss(n)
        np.testing.assert_allclose(x, xr[::-1], atol=1e-14)
        np.testing.assert_allclose(w, wr[::-1], atol=1e-14)


def test_legendre_matches_scipy_harmonics():
    import scipy.special as sp
    for x in (0.93, 0.2, -0.7, 1.0):
        lmax = 64
        v = lib.cgtp_legendre(lmax, x)
        th = math.acos(x)
        for l in (0, 1, 2, 5, 17, 40, 64):
            for m in sorted({0, 1, l // 2, l}):
                if m > l:
                    continue
                want = (sp.sph_harm_y(l, m, th, 0.0) if hasattr(sp, "sph_harm_y") else sp.sph_harm(m, l, 0.0, th)).real
                assert v[l * (l + 1) // 2 + m] == pytest.approx(want, abs=1e-12), (l, m, x)


def test_gaunt_factor_is_the_scalar_case():
    """K for the scalar-scalar product equals the Gaunt prefactor (Section 3.3)."""
    for j1, j2, j3 in [(0, 0, 0), (1, 1, 2), (3, 5, 4), (16, 16, 32), (32, 30, 2)]:
        K, kind = lib.cgtp_path_norm(j1, j2, j3)
        assert kind == 0
        want = math.sqrt((2 * j1 + 1) * (2 * j2 + 1) / (4 * math.pi * (2 * j3 + 1))) * oracle.cg(j1, 0, j2, 0, j3, 0)
        assert K == pytest.approx(want, rel=1e-12)


def _tsh(l, s, j, mj, T, P):
    """Tensor spherical harmonic of Definition 4.1 on a grid, components m_s = -s..s (scipy + sympy)."""
    import scipy.special as sp
    from sympy.physics.wigner import clebsch_gordan
    comps = []
    for ms in range(-s, s + 1):
        f = 0
        for ml in range(-l, l + 1):
            c = float(clebsch_gordan(l, s, j, ml, ms, mj))
            if c:
                f = f + c * (sp.sph_harm_y(l, ml, T, P) if hasattr(sp, "sph_harm_y") else sp.sph_harm(ml, l, P, T))
        comps.append(f * np.ones_like(T))
    return comps


@pytest.mark.parametrize("j1,j2,j3,cover", [(1, 1, 1, 0), (2, 1, 2, 0), (2, 3, 2, 0), (3, 3, 4, 1),
                                            (2, 2, 3, 1), (1, 2, 2, 1), (3, 2, 4, 0)])
def test_path_factor_against_quadrature(j1, j2, j3, cover):
    """Theorem 4.2 by direct quadrature of products of tensor harmonics (independent of the plan)."""
    from sympy.physics.wigner import clebsch_gordan
    K, kind = lib.cgtp_path_norm(j1, j2, j3, cover)
    s1, s2, s3, l3 = {0: (0, 0, 0, j3), 1: (1, 1, 1, j3 - 1), 2: (0, 1, 1, j3 - 1), 3: (1, 1, 0, j3)}[kind]
    xs, ws = np.polynomial.legendre.leggauss(24)
    T, P = np.meshgrid(np.arccos(xs), 2 * np.pi * np.arange(48) / 48, indexing="ij")
    W = ws[:, None] * (2 * np.pi / 48)
    m1 = min(j1, 1)
    m2 = j3 - m1 if abs(j3 - m1) <= j2 else -j2
    m3 = m1 + m2
    A = _tsh(j1, s1, j1, m1, T, P)
    B = _tsh(j2, s2, j2, m2, T, P)
    prod = []
    for ms3 in range(-s3, s3 + 1):
        acc = 0
        for ma in range(-s1, s1 + 1):
            mb = ms3 - ma
            if abs(mb) <= s2:
                acc = acc + float(clebsch_gordan(s1, s2, s3, ma, mb, ms3)) * A[ma + s1] * B[mb + s2]
        prod.append(acc)
    C = _tsh(l3, s3, j3, m3, T, P)
    raw = sum((W * prod[k] * np.conj(C[k])).sum() for k in range(2 * s3 + 1))
    cg = float(clebsch_gordan(j1, j2, j3, m1, m2, m3))
    assert abs(cg) > 1e-3
    assert raw.real == pytest.approx(K * cg, abs=1e-12)
    assert abs(raw.imag) < 1e-12


def test_vector_selection_rule_zero():
    """Rule 5 of Theorem 5.1: toroidal j = 1 with itself projected on (j3, l3) = (2, 2) vanishes."""
    assert abs(lib.cgtp_wigner_9j(1, 1, 1, 1, 1, 1, 2, 2, 1)) < 1e-15
    assert abs(lib.cgtp_wigner_9j(2, 2, 1, 3, 3, 1, 4, 4, 1)) < 1e-15


def test_default_cover_is_complete():
    """Every path at L = 32 gets a nonzero factor (Theorem 5.2 / Corollary 5.3)."""
    worst = 1e9
    for j1 in range(33):
        for j2 in range(33):
            for j3 in range(abs(j1 - j2), j1 + j2 + 1):
                K, kind = lib.cgtp_path_norm(j1, j2, j3)
                assert kind == (0 if (j1 + j2 + j3) % 2 == 0 else 1)
                worst = min(worst, abs(K))
    assert worst > 0.02


def test_alternate_cover_falls_back_on_accidental_zeros():
    """The dot-product factor vanishes when j1(j1+1) + j2(j2+1) = j3(j3+1), e.g. (3, 5, 6)."""
    K, kind = lib.cgtp_path_norm(3, 5, 6, 1)
    assert kind == 0
    K, kind = lib.cgtp_path_norm(3, 4, 5, 1)    # even sum: dot product
    assert kind == 3
    K, kind = lib.cgtp_path_norm(3, 4, 6, 1)    # odd sum: scalar-vector product
    assert kind == 2


def test_alternate_cover_fall_back_is_per_block():
    """Each block uses one product per parity: blocks holding an exact zero of the dot factor
    (j1(j1+1) + j2(j2+1) = j3(j3+1), even sum) fall back to scalar-scalar for all their even
    paths, the others use the dot product throughout; odd paths use scalar-vector."""
    for j3 in range(2, 9):
        K, kind = lib.cgtp_path_norm(3, 5, j3, 1)
        assert kind == (0 if j3 % 2 == 0 else 2)
    zeros = {(a, b, c) for a in range(1, 33) for b in range(1, 33) for c in range(abs(a - b), a + b + 1)
             if (a + b + c) % 2 == 0 and a * (a + 1) + b * (b + 1) == c * (c + 1)}
    assert (3, 5, 6) in zeros and (5, 3, 6) in zeros
    for a in range(1, 33):
        for b in range(1, 33):
            even_kinds, odd_kinds = set(), set()
            for c in range(abs(a - b), a + b + 1):
                K, kind = lib.cgtp_path_norm(a, b, c, 1)
                (even_kinds if (a + b + c) % 2 == 0 else odd_kinds).add(kind)
                assert abs(K) >= 1e-3
            assert len(even_kinds) == 1 and even_kinds <= {0, 3}
            if any((a, b, c) in zeros for c in range(abs(a - b), a + b + 1)):
                assert even_kinds == {0}
            assert odd_kinds <= {2}               # no scalar-vector zero up to L = 32


@pytest.mark.parametrize("L", [0, 1, 2, 4])
@pytest.mark.parametrize("cover", [0, 1])
def test_method_model_matches_oracle(L, cover, rng):
    x1 = rng.standard_normal((3, (L + 1) ** 2))
    x2 = rng.standard_normal((3, (L + 1) ** 2))
    np.testing.assert_allclose(model_cgtp(L, x1, x2, cover), oracle.cgtp(L, x1, x2), atol=1e-12)


def test_method_model_alternate_cover_with_fall_back_block(rng):
    """L = 5 holds block (3, 5), whose even paths fall back to scalar-scalar."""
    L = 5
    x1 = rng.standard_normal((2, (L + 1) ** 2))
    x2 = rng.standard_normal((2, (L + 1) ** 2))
    np.testing.assert_allclose(model_cgtp(L, x1, x2, 1), oracle.cgtp(L, x1, x2), atol=1e-12)


def test_method_model_on_a_global_grid(rng):
    L = 3
    x1 = rng.standard_normal((2, 16))
    x2 = rng.standard_normal((2, 16))
    np.testing.assert_allclose(model_cgtp(L, x1, x2, 0, n_theta=10, n_phi=16), oracle.cgtp(L, x1, x2), atol=1e-12)


def test_aliasing_grid_breaks_exactness(rng):
    """One ring too few makes the quadrature inexact: the exactness bound is sharp."""
    L = 3
    x1 = rng.standard_normal((2, 16))
    x2 = rng.standard_normal((2, 16))
    with pytest.raises(lib.CgtpError) as e:
        lib.cgtp_block_grid(L, 1, 1, lib._grid(n_theta=2 * L, n_phi=0))
    assert e.value.code == lib.CGTP_EGRID

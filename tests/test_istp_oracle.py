"""Pins for the MIMO irrep-signal product oracle (no GPU needed).

The oracle (``oracle.istp``) works on coefficients.  These tests tie it to
things computed another way:
* direct quadrature, on an exact sphere grid, of products of scipy's
  spherical harmonics and of tensor harmonics built from them with sympy's
  exact Clebsch-Gordan values (Definition 4.1);
* Theorem 4.2 with sympy's 9j symbol;
* a closed form for a constant first input;
* rotation equivariance with Wigner matrices fitted from scipy's harmonics;
* the vector selection rule of Theorem 5.1.
A wrong sign, index or operand order in any of the oracle's three steps
fails the quadrature tests.
"""
import math

import numpy as np
import pytest

import oracle.istp as oi
from test_oracle import _quadrature_grid, _sph_harm, _wigner_D
from test_plan import _tsh


def _sympy_cg(j1, m1, j2, m2, j, m):
    from sympy.physics.wigner import clebsch_gordan
    return float(clebsch_gordan(j1, j2, j, m1, m2, m))


def test_layout():
    for L in range(5):
        labels = oi.vector_labels(L)
        offs = [oi.vector_offset(j, l) for j, l in labels]
        sizes = [2 * j + 1 for j, l in labels]
        assert offs == list(np.cumsum([0] + sizes[:-1]))
        assert sum(sizes) == oi.vector_size(L) == 3 * (L + 1) ** 2
    with pytest.raises(ValueError):
        oi.vector_offset(0, 0)
    with pytest.raises(ValueError):
        oi.vector_offset(3, 1)


def test_gaunt_product_against_quadrature(rng):
    """z[l3, m3] = integral of f1 f2 conj(Y_l3^m3) for f_i = sum x_i Y (scipy harmonics, exact grid)."""
    L = 3
    x1 = rng.standard_normal(oi.gaunt_size(L))
    x2 = rng.standard_normal(oi.gaunt_size(L))
    z = oi.gaunt_tp(L, x1, x2)[0]
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)
    Y = {(l, m): _sph_harm(l, m, T, P) for l in range(2 * L + 1) for m in range(-l, l + 1)}
    f1 = sum(x1[l * l + l + m] * Y[l, m] for l in range(L + 1) for m in range(-l, l + 1))
    f2 = sum(x2[l * l + l + m] * Y[l, m] for l in range(L + 1) for m in range(-l, l + 1))
    want = np.array([(W * f1 * f2 * np.conj(Y[l, m])).sum() for l in range(2 * L + 1) for m in range(-l, l + 1)])
    assert np.abs(want.imag).max() < 1e-12
    np.testing.assert_allclose(z, want.real, atol=1e-12)


def _vector_signal(L, x, T, P):
    """Spherical components q = -1, 0, +1 of sum_{j,l,m} x^(j,l)_m Y^{l,1}_{j,m} on the grid."""
    f = [np.zeros(T.shape, complex) for _ in range(3)]
    for j, l in oi.vector_labels(L):
        o = oi.vector_offset(j, l)
        for m in range(-j, j + 1):
            comps = _tsh(l, 1, j, m, T, P)
            for k in range(3):
                f[k] = f[k] + x[o + j + m] * comps[k]
    return f


@pytest.mark.parametrize("L", [1, 2])
def test_vector_product_against_quadrature(L, rng):
    """Every output against the integral of conj(Y^{l3,1}_{j3,m3}) . (f1 (x) f2)^(1) (Definition 4.1, Section 4.3)."""
    x1 = rng.standard_normal(oi.vector_size(L))
    x2 = rng.standard_normal(oi.vector_size(L))
    z = oi.vector_tp(L, x1, x2)[0]
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)
    f1 = _vector_signal(L, x1, T, P)
    f2 = _vector_signal(L, x2, T, P)
    g = []
    for q in (-1, 0, 1):
        acc = np.zeros(T.shape, complex)
        for q1 in (-1, 0, 1):
            q2 = q - q1
            if abs(q2) <= 1:
                acc = acc + _sympy_cg(1, q1, 1, q2, 1, q) * f1[q1 + 1] * f2[q2 + 1]
        g.append(acc)
    want = np.zeros(oi.vector_size(2 * L), complex)
    for j3, l3 in oi.vector_labels(2 * L):
        o = oi.vector_offset(j3, l3)
        for m3 in range(-j3, j3 + 1):
            basis = _tsh(l3, 1, j3, m3, T, P)
            want[o + j3 + m3] = sum((W * g[k] * np.conj(basis[k])).sum() for k in range(3))
    assert np.abs(want.imag).max() < 1e-12
    np.testing.assert_allclose(z, want.real, atol=1e-12)


def test_vector_product_theorem_4_2(rng):
    """Output label (j3, l3) = sum over input labels of K (x1^(j1,l1) (x) x2^(j2,l2))^(j3), K from Theorem 4.2 (sympy 9j)."""
    from sympy.physics.wigner import wigner_9j
    L = 2
    x1 = rng.standard_normal(oi.vector_size(L))
    x2 = rng.standard_normal(oi.vector_size(L))
    z = oi.vector_tp(L, x1, x2)[0]
    want = np.zeros_like(z)
    for j1, l1 in oi.vector_labels(L):
        for j2, l2 in oi.vector_labels(L):
            for j3, l3 in oi.vector_labels(2 * L):
                if not (abs(j1 - j2) <= j3 <= j1 + j2 and abs(l1 - l2) <= l3 <= l1 + l2) or (l1 + l2 + l3) & 1:
                    continue
                c0 = _sympy_cg(l1, 0, l2, 0, l3, 0)
                nj = float(wigner_9j(j1, l1, 1, j2, l2, 1, j3, l3, 1, prec=30))
                K = math.sqrt((2 * j1 + 1) * (2 * j2 + 1) * (2 * l1 + 1) * (2 * l2 + 1) * 3 / (4 * math.pi)) * nj * c0
                if K == 0.0:
                    continue
                a = x1[oi.vector_offset(j1, l1):][: 2 * j1 + 1]
                b = x2[oi.vector_offset(j2, l2):][: 2 * j2 + 1]
                o = oi.vector_offset(j3, l3)
                for m3 in range(-j3, j3 + 1):
                    s = sum(_sympy_cg(j1, m1, j2, m3 - m1, j3, m3) * a[j1 + m1] * b[j2 + m3 - m1]
                            for m1 in range(-j1, j1 + 1) if abs(m3 - m1) <= j2)
                    want[o + j3 + m3] += K * s
    np.testing.assert_allclose(z, want, atol=1e-12)


def test_gaunt_product_constant_input(rng):
    """f1 = c Y_0^0 = c / sqrt(4 pi) constant: z = c x2 / sqrt(4 pi) up to degree L, zero above."""
    L = 4
    x1 = np.zeros(oi.gaunt_size(L))
    x1[0] = 1.7
    x2 = rng.standard_normal(oi.gaunt_size(L))
    z = oi.gaunt_tp(L, x1, x2)[0]
    np.testing.assert_allclose(z[: (L + 1) ** 2], 1.7 / math.sqrt(4 * math.pi) * x2, atol=1e-14)
    np.testing.assert_allclose(z[(L + 1) ** 2:], 0.0, atol=1e-14)


def _complex(fn, L, x1, x2):
    """A bilinear real product applied to complex inputs."""
    rr = fn(L, x1.real, x2.real)
    ii = fn(L, x1.imag, x2.imag)
    ri = fn(L, x1.real, x2.imag)
    ir = fn(L, x1.imag, x2.real)
    return (rr - ii) + 1j * (ri + ir)


def test_vector_product_rotation_equivariance(rng):
    """Rotating both inputs (label (j, l) by D^j) rotates each output label (j3, l3) by D^{j3}."""
    from scipy.spatial.transform import Rotation
    L = 2
    R = Rotation.random(random_state=int(rng.integers(1 << 30)))
    D = {j: _wigner_D(j, R, rng) for j in range(2 * L + 2)}

    def rot(x, Lx):
        y = np.array(x, dtype=complex)
        for j, l in oi.vector_labels(Lx):
            o = oi.vector_offset(j, l)
            y[..., o: o + 2 * j + 1] = x[..., o: o + 2 * j + 1] @ D[j].T
        return y

    x1 = rng.standard_normal((2, oi.vector_size(L))).astype(complex)
    x2 = rng.standard_normal((2, oi.vector_size(L))).astype(complex)
    z = _complex(oi.vector_tp, L, x1, x2)
    zr = _complex(oi.vector_tp, L, rot(x1, L), rot(x2, L))
    np.testing.assert_allclose(zr, rot(z, 2 * L), atol=1e-10)


def test_vector_selection_rule():
    """Theorem 5.1 for labels (1,1) x (1,1): (j3, l3) = (2, 2) vanishes by rule 5, (1, 1), (2, 1), (0, 1) by rule 4."""
    L = 1
    x = np.zeros(oi.vector_size(L))
    o = oi.vector_offset(1, 1)
    rng = np.random.default_rng(5)
    x[o: o + 3] = rng.standard_normal(3)
    y = np.zeros(oi.vector_size(L))
    y[o: o + 3] = rng.standard_normal(3)
    z = oi.vector_tp(L, x, y)[0]
    for j3, l3, zero in [(2, 2, True), (1, 1, True), (2, 1, True), (0, 1, True), (1, 2, False), (1, 0, False)]:
        blk = z[oi.vector_offset(j3, l3):][: 2 * j3 + 1]
        if zero:
            np.testing.assert_allclose(blk, 0.0, atol=1e-14)
        else:
            assert np.abs(blk).max() > 1e-3, (j3, l3)


def _reverse(spin, L, x):
    """x~[(j,l), m] = (-1)^(m + j - l + spin) x[(j,l), -m] (time reversal of the coefficients)."""
    y = np.zeros_like(x)
    labels = [(l, l) for l in range(L + 1)] if spin == 0 else oi.spin_labels(spin, L)
    off = (lambda j, l: l * l) if spin == 0 else (lambda j, l: oi.spin_offset(spin, j, l))
    for j, l in labels:
        o = off(j, l)
        for m in range(-j, j + 1):
            y[..., o + j + m] = (-1) ** ((m + j - l + spin) % 2) * x[..., o + j - m]
    return y


def _fn(spin):
    return {0: oi.gaunt_tp, 1: oi.vector_tp}.get(spin, lambda *a, **k: oi.spin_tp(spin, *a, **k))


@pytest.mark.parametrize("spin", [0, 1, 2])
def test_vjp_against_time_reversed_product(spin, rng):
    """The gradients equal +-P(g, reversed other input): a degree-2L by degree-L product projected on degrees <= L,
    the adjoint of the integral of three harmonics (the vector product changes sign under the swap of its inputs;
    the spin-0 and spin-2 couplings are symmetric)."""
    L = 2
    size = lambda Lx: oi.spin_size(spin, Lx)
    fn = _fn(spin)
    x1 = rng.standard_normal((2, size(L)))
    x2 = rng.standard_normal((2, size(L)))
    g = rng.standard_normal((2, size(2 * L)))
    g1, g2 = oi.product_vjp(spin, L, x1, x2, g)
    np.testing.assert_allclose(g1, fn(2 * L, g, _reverse(spin, L, x2), L2=L, Lo=L), atol=1e-12)
    sign = -1.0 if spin == 1 else 1.0
    np.testing.assert_allclose(g2, sign * fn(2 * L, g, _reverse(spin, L, x1), L2=L, Lo=L), atol=1e-12)


@pytest.mark.parametrize("spin", [0, 1, 2])
def test_vjp_euler_identity(spin, rng):
    """Bilinearity: <g, z(x1, x2)> = <grad_x1, x1> = <grad_x2, x2>."""
    L = 3 if spin < 2 else 2
    size = lambda Lx: oi.spin_size(spin, Lx)
    fn = _fn(spin)
    x1 = rng.standard_normal((3, size(L)))
    x2 = rng.standard_normal((3, size(L)))
    g = rng.standard_normal((3, size(2 * L)))
    g1, g2 = oi.product_vjp(spin, L, x1, x2, g)
    want = (g * fn(L, x1, x2)).sum(1)
    np.testing.assert_allclose((g1 * x1).sum(1), want, rtol=1e-12)
    np.testing.assert_allclose((g2 * x2).sum(1), want, rtol=1e-12)


def test_unequal_bounds_against_quadrature(rng):
    """The Gaunt product with degree bounds (3, 1) -> 2 against direct quadrature of scipy's harmonics."""
    L1, L2, Lo = 3, 1, 2
    x1 = rng.standard_normal(oi.gaunt_size(L1))
    x2 = rng.standard_normal(oi.gaunt_size(L2))
    z = oi.gaunt_tp(L1, x1, x2, L2=L2, Lo=Lo)[0]
    T, P, W = _quadrature_grid(8, 16)
    Y = {(l, m): _sph_harm(l, m, T, P) for l in range(L1 + 1) for m in range(-l, l + 1)}
    f1 = sum(x1[l * l + l + m] * Y[l, m] for l in range(L1 + 1) for m in range(-l, l + 1))
    f2 = sum(x2[l * l + l + m] * Y[l, m] for l in range(L2 + 1) for m in range(-l, l + 1))
    want = np.array([(W * f1 * f2 * np.conj(Y[l, m])).sum() for l in range(Lo + 1) for m in range(-l, l + 1)])
    np.testing.assert_allclose(z, want.real, atol=1e-12)


# ---------------------------------------------------------------- spin 2

def test_spin_layout_and_spin_one():
    """Spin-s rows: labels tile the row; at s = 1 the general product is the vector product."""
    for s in (1, 2, 3):
        for L in range(4):
            labs = oi.spin_labels(s, L)
            offs = [oi.spin_offset(s, j, l) for j, l in labs]
            sizes = [2 * j + 1 for j, l in labs]
            assert offs == list(np.cumsum([0] + sizes[:-1])) and sum(sizes) == oi.spin_size(s, L)
    assert oi.spin_labels(1, 3) == oi.vector_labels(3)
    rng = np.random.default_rng(4)
    x1, x2 = rng.standard_normal((2, 2, oi.vector_size(2)))
    np.testing.assert_allclose(oi.spin_tp(1, 2, x1, x2), oi.vector_tp(2, x1, x2), atol=1e-14)


def test_spin_two_product_against_quadrature(rng):
    """Every output against the integral of conj(Y^{l3,2}_{j3,m3}) . (f1 (x) f2)^(2) on an exact grid
    (tensor harmonics of Definition 4.1 from scipy's harmonics and sympy's CG)."""
    L, s = 1, 2
    x1 = rng.standard_normal(oi.spin_size(s, L))
    x2 = rng.standard_normal(oi.spin_size(s, L))
    z = oi.spin_tp(s, L, x1, x2)[0]
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)

    def signal(x):
        f = [np.zeros(T.shape, complex) for _ in range(2 * s + 1)]
        for j, l in oi.spin_labels(s, L):
            o = oi.spin_offset(s, j, l)
            for m in range(-j, j + 1):
                comps = _tsh(l, s, j, m, T, P)
                for k in range(2 * s + 1):
                    f[k] = f[k] + x[o + j + m] * comps[k]
        return f

    f1, f2 = signal(x1), signal(x2)
    g = []
    for q in range(-s, s + 1):
        acc = np.zeros(T.shape, complex)
        for q1 in range(-s, s + 1):
            q2 = q - q1
            if abs(q2) <= s:
                acc = acc + _sympy_cg(s, q1, s, q2, s, q) * f1[q1 + s] * f2[q2 + s]
        g.append(acc)
    want = np.zeros(oi.spin_size(s, 2 * L), complex)
    for j3, l3 in oi.spin_labels(s, 2 * L):
        o = oi.spin_offset(s, j3, l3)
        for m3 in range(-j3, j3 + 1):
            basis = _tsh(l3, s, j3, m3, T, P)
            want[o + j3 + m3] = sum((W * g[k] * np.conj(basis[k])).sum() for k in range(2 * s + 1))
    assert np.abs(want.imag).max() < 1e-12
    np.testing.assert_allclose(z, want.real, atol=1e-12)


def test_spin_two_rotation_equivariance(rng):
    """Rotating both inputs (label (j, l) by D^j) rotates each output label (j3, l3) by D^{j3}."""
    from scipy.spatial.transform import Rotation
    L, s = 2, 2
    R = Rotation.random(random_state=int(rng.integers(1 << 30)))
    D = {j: _wigner_D(j, R, rng) for j in range(2 * L + s + 1)}

    def rot(x, Lx):
        y = np.array(x, dtype=complex)
        for j, l in oi.spin_labels(s, Lx):
            o = oi.spin_offset(s, j, l)
            y[..., o: o + 2 * j + 1] = x[..., o: o + 2 * j + 1] @ D[j].T
        return y

    x1 = rng.standard_normal((2, oi.spin_size(s, L))).astype(complex)
    x2 = rng.standard_normal((2, oi.spin_size(s, L))).astype(complex)
    f = lambda L_, a, b: oi.spin_tp(s, L_, a, b)
    z = _complex(f, L, x1, x2)
    zr = _complex(f, L, rot(x1, L), rot(x2, L))
    np.testing.assert_allclose(zr, rot(z, 2 * L), atol=1e-10)


# ---------------------------------------------------------------- real basis

def _real_sph_harm(l, m, T, P):
    """Real harmonic with the Condon-Shortley phase, built from scipy's complex harmonic."""
    y = _sph_harm(l, abs(m), T, P)
    if m > 0:
        return math.sqrt(2.0) * (-1) ** m * y.real
    if m < 0:
        return math.sqrt(2.0) * (-1) ** m * y.imag
    return y.real


def test_real_basis_round_trip(rng):
    """to_real(to_complex(r)) = r, and the complex coefficients of a real function are Hermitian."""
    L = 4
    r = rng.standard_normal((3, oi.gaunt_size(L)))
    c = oi.to_complex(L, r)
    np.testing.assert_allclose(oi.to_real(L, c), r, atol=1e-14)
    for l in range(L + 1):
        for m in range(1, l + 1):
            np.testing.assert_allclose(c[:, l * l + l - m], (-1) ** m * np.conj(c[:, l * l + l + m]), atol=1e-14)


def test_real_gaunt_product_against_quadrature(rng):
    """z[l3, m3] = integral of f1 f2 Y^R_{l3 m3} for f_i = sum r_i Y^R (scipy harmonics, exact grid)."""
    L = 3
    r1 = rng.standard_normal(oi.gaunt_size(L))
    r2 = rng.standard_normal(oi.gaunt_size(L))
    z = oi.gaunt_tp_real(L, r1, r2)[0]
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)
    Y = {(l, m): _real_sph_harm(l, m, T, P) for l in range(2 * L + 1) for m in range(-l, l + 1)}
    f1 = sum(r1[l * l + l + m] * Y[l, m] for l in range(L + 1) for m in range(-l, l + 1))
    f2 = sum(r2[l * l + l + m] * Y[l, m] for l in range(L + 1) for m in range(-l, l + 1))
    want = np.array([(W * f1 * f2 * Y[l, m]).sum() for l in range(2 * L + 1) for m in range(-l, l + 1)])
    np.testing.assert_allclose(z, want, atol=1e-12)


def test_real_gaunt_gradients(rng):
    """Euler identity, and grad_x1[i] = integral of Y^R_i f2 f_g (f_g = sum g Y^R; scipy harmonics, exact grid)."""
    L = 2
    r1 = rng.standard_normal((2, oi.gaunt_size(L)))
    r2 = rng.standard_normal((2, oi.gaunt_size(L)))
    g = rng.standard_normal((2, oi.gaunt_size(2 * L)))
    g1, g2 = oi.gaunt_tp_real_vjp(L, r1, r2, g)
    want = (g * oi.gaunt_tp_real(L, r1, r2)).sum(1)
    np.testing.assert_allclose((g1 * r1).sum(1), want, rtol=1e-12)
    np.testing.assert_allclose((g2 * r2).sum(1), want, rtol=1e-12)
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)
    Y = {(l, m): _real_sph_harm(l, m, T, P) for l in range(2 * L + 1) for m in range(-l, l + 1)}
    for n in range(2):
        f2 = sum(r2[n, l * l + l + m] * Y[l, m] for l in range(L + 1) for m in range(-l, l + 1))
        fg = sum(g[n, l * l + l + m] * Y[l, m] for l in range(2 * L + 1) for m in range(-l, l + 1))
        q = np.array([(W * Y[l, m] * f2 * fg).sum() for l in range(L + 1) for m in range(-l, l + 1)])
        np.testing.assert_allclose(g1[n], q, atol=1e-12)


# ---------------------------------------------------------------- real basis, spin 1 and 2

def _spin_field(s, L, c, T, P):
    """Spherical components q = -s..s on the grid of sum c^(j,l)_m Y^{l,s}_{j,m}."""
    f = [np.zeros(T.shape, complex) for _ in range(2 * s + 1)]
    for j, l in oi.spin_labels(s, L):
        o = oi.spin_offset(s, j, l)
        for m in range(-j, j + 1):
            if c[o + j + m] == 0:
                continue
            comps = _tsh(l, s, j, m, T, P)
            for k in range(2 * s + 1):
                f[k] = f[k] + c[o + j + m] * comps[k]
    return f


def _real_field_violation(f, s):
    """max |F_{-q} - (-1)^q conj(F_q)|: zero exactly for a real field in the spherical basis."""
    return max(np.abs(f[s - q] - (-1) ** q * np.conj(f[s + q])).max() for q in range(0, s + 1))


@pytest.mark.parametrize("s", [1, 2])
def test_spin_real_basis_round_trip_and_real_fields(s, rng):
    """spin_to_real inverts spin_to_complex, and real-basis rows synthesise real fields (the per-label phase
    (-1)^(l+s-j) of the conjugation rule)."""
    L = 2
    r = rng.standard_normal((3, oi.spin_size(s, L)))
    np.testing.assert_allclose(oi.spin_to_real(s, L, oi.spin_to_complex(s, L, r)), r, atol=1e-14)
    T, P, _ = _quadrature_grid(L + 2, 2 * L + 3)
    f = _spin_field(s, L, oi.spin_to_complex(s, L, r[0])[0], T, P)
    assert _real_field_violation(f, s) < 1e-12


@pytest.mark.parametrize("s", [1, 2])
def test_spin_real_product_against_quadrature(s, rng):
    """spin_tp_real against direct quadrature: the coupled pointwise product of the two real fields, times the
    oracle's output phase, is a real field, and its projections on the tensor harmonics, read back in the real
    basis, are the oracle's outputs."""
    L = 1
    r1 = rng.standard_normal(oi.spin_size(s, L))
    r2 = rng.standard_normal(oi.spin_size(s, L))
    z = oi.spin_tp_real(s, L, r1, r2)[0]
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)
    f1 = _spin_field(s, L, oi.spin_to_complex(s, L, r1)[0], T, P)
    f2 = _spin_field(s, L, oi.spin_to_complex(s, L, r2)[0], T, P)
    kappa = {1: 1j, 2: 1.0}[s]   # the convention: spin 2 as coupled, spin 1 times i (sign: the cross-product test)
    g = []
    for q in range(-s, s + 1):
        acc = np.zeros(T.shape, complex)
        for q1 in range(-s, s + 1):
            q2 = q - q1
            if abs(q2) <= s:
                acc = acc + _sympy_cg(s, q1, s, q2, s, q) * f1[q1 + s] * f2[q2 + s]
        g.append(kappa * acc)
    assert _real_field_violation(g, s) < 1e-12
    c3 = np.zeros(oi.spin_size(s, 2 * L), complex)
    for j3, l3 in oi.spin_labels(s, 2 * L):
        o = oi.spin_offset(s, j3, l3)
        for m3 in range(-j3, j3 + 1):
            basis = _tsh(l3, s, j3, m3, T, P)
            c3[o + j3 + m3] = sum((W * g[k] * np.conj(basis[k])).sum() for k in range(2 * s + 1))
    np.testing.assert_allclose(z, oi.spin_to_real(s, 2 * L, c3)[0], atol=1e-12)


def test_spin_one_real_basis_constant_fields():
    """Label (1, 0) holds a constant field: its real basis is the Cartesian (y, z, x) components times Y_0^0,
    and the spin-1 product of two constant fields A, B is (A x B) / sqrt 2 times Y_0^0 there."""
    rng = np.random.default_rng(9)
    L = 1
    o = oi.spin_offset(1, 1, 0)
    a = np.zeros((1, oi.spin_size(1, L)))
    b = np.zeros_like(a)
    A, B = rng.standard_normal(3), rng.standard_normal(3)   # (y, z, x)
    a[0, o:o + 3], b[0, o:o + 3] = A, B
    y00 = 1.0 / math.sqrt(4 * math.pi)
    T, P, _ = _quadrature_grid(3, 5)
    f = _spin_field(1, L, oi.spin_to_complex(1, L, a)[0], T, P)
    # spherical components -> Cartesian: F = sum_q F_q e_q, e_{+-1} = -+(x +- i y) / sqrt 2, e_0 = z
    fx = (-f[2] + f[0]) / math.sqrt(2)
    fy = (-1j * f[2] - 1j * f[0]) / math.sqrt(2)
    np.testing.assert_allclose(np.stack([fy, f[1], fx]).real.reshape(3, -1).mean(1), A * y00, atol=1e-12)
    z = oi.spin_tp_real(1, L, a, b)[0]
    cart = lambda v: np.array([v[2], v[0], v[1]])
    cr = np.cross(cart(A), cart(B))
    np.testing.assert_allclose(z[o:o + 3], np.array([cr[1], cr[2], cr[0]]) / math.sqrt(2) * y00, atol=1e-13)


def test_spin_zero_real_product_is_the_real_gaunt_product(rng):
    r1 = rng.standard_normal((2, 16))
    r2 = rng.standard_normal((2, 16))
    np.testing.assert_allclose(oi.spin_tp_real(0, 3, r1, r2), oi.gaunt_tp_real(3, r1, r2), atol=1e-14)

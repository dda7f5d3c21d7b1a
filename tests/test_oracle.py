"""Pins for the CPU oracle (no GPU needed).

Each test ties the oracle to something other than itself: sympy's exact
Clebsch-Gordan implementation, textbook values, quadrature of scipy's
spherical harmonics, Cartesian vector algebra, rotation matrices built from
scipy's harmonics, or identities that hold for any correct CGTP.  A dropped
term, a wrong sign or index, or swapped operands in the oracle fails at least
one of them.
"""
import math
import os

import numpy as np
import pytest

import oracle
from cgtp_inputs import block_slice

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sph_harm(l, m, theta, phi):
    """Complex orthonormal Y_l^m with Condon-Shortley phase (scipy)."""
    import scipy.special as sp
    if hasattr(sp, "sph_harm_y"):
        return sp.sph_harm_y(l, m, theta, phi)
    return sp.sph_harm(m, l, phi, theta)


def _paths(L):
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                yield l1, l2, l3


def _path(z, L, l1, l2, l3):
    off = oracle.path_offset(L, l1, l2, l3)
    return z[..., off:off + 2 * l3 + 1]


# ---------------------------------------------------------------- CG values

def test_cg_hand_values():
    """Textbook values (fixture with the closed forms they come from)."""
    n = 0
    for line in open(os.path.join(GOLDEN, "cg_hand_values.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        p = line.split()
        j1, m1, j2, m2, j, m = map(int, p[:6])
        want = eval(p[6], {"sqrt": math.sqrt})
        assert oracle.cg(j1, m1, j2, m2, j, m) == pytest.approx(want, abs=1e-15), p
        n += 1
    assert n >= 20


def test_cg_matches_sympy_exact(rng):
    """sympy's exact (rational-arithmetic) CG is an independent implementation."""
    from sympy.physics.wigner import clebsch_gordan
    cases = [(32, 3, 32, -5, 57, -2), (32, 32, 32, -32, 0, 0), (20, -7, 25, 7, 40, 0),
             (17, 17, 16, -16, 33, 1), (31, 0, 30, 0, 61, 0), (32, 32, 32, 32, 64, 64)]
    for _ in range(40):
        j1, j2 = int(rng.integers(0, 33)), int(rng.integers(0, 33))
        j = int(rng.integers(abs(j1 - j2), j1 + j2 + 1))
        m1 = int(rng.integers(-j1, j1 + 1))
        m = int(rng.integers(max(-j, m1 - j2), min(j, m1 + j2) + 1))
        cases.append((j1, m1, j2, m - m1, j, m))
    for j1, m1, j2, m2, j, m in cases:
        want = float(clebsch_gordan(j1, j2, j, m1, m2, m).evalf(30))
        assert oracle.cg(j1, m1, j2, m2, j, m) == pytest.approx(want, abs=2e-14), (j1, m1, j2, m2, j, m)


def test_cg_selection_rules():
    assert oracle.cg(1, 1, 1, 1, 1, 1) == 0.0          # m1 + m2 != m
    assert oracle.cg(1, 0, 1, 0, 3, 0) == 0.0          # triangle violated
    assert oracle.cg(2, 3, 1, 0, 2, 3) == 0.0          # |m1| > j1


@pytest.mark.parametrize("j1,j2", [(0, 5), (3, 3), (7, 12), (16, 16), (32, 31), (32, 32)])
def test_cg_orthogonality(j1, j2):
    """Both orthogonality relations (Appendix D.1): the CG matrix is orthogonal."""
    blocks = {j: oracle.cg_block(j1, j2, j) for j in range(abs(j1 - j2), j1 + j2 + 1)}
    # sum_{m1 m2} C^{j m} C^{j' m} = delta_{j j'}
    for m in range(-(j1 + j2), j1 + j2 + 1):
        rows = []
        for j, b in blocks.items():
            if abs(m) <= j:
                row = b[m + j].copy()
                for m1 in range(-j1, j1 + 1):
                    if abs(m - m1) > j2:
                        assert row[m1 + j1] == 0.0
                rows.append(row)
        A = np.array(rows)
        np.testing.assert_allclose(A @ A.T, np.eye(len(rows)), atol=1e-12)
        # and the columns with a valid m2 are complete: sum_j C C' = delta_{m1 m1'}
        valid = [m1 + j1 for m1 in range(-j1, j1 + 1) if abs(m - m1) <= j2]
        np.testing.assert_allclose(A[:, valid].T @ A[:, valid], np.eye(len(valid)), atol=1e-12)


def test_cg_symmetry_relation(rng):
    """C^{j mj}_{l ml s ms} = (-1)^{l-ml} sqrt((2j+1)/(2s+1)) C^{s ms}_{j mj l -ml} (Lemma F.1)."""
    for _ in range(300):
        l, s = int(rng.integers(0, 12)), int(rng.integers(0, 12))
        j = int(rng.integers(abs(l - s), l + s + 1))
        ml = int(rng.integers(-l, l + 1))
        ms = int(rng.integers(-s, s + 1))
        mj = ml + ms
        lhs = oracle.cg(l, ml, s, ms, j, mj)
        rhs = (-1) ** (l - ml) * math.sqrt((2 * j + 1) / (2 * s + 1)) * oracle.cg(j, mj, l, -ml, s, ms)
        assert lhs == pytest.approx(rhs, abs=1e-14)


# ---------------------------------------------------------------- CGTP

def test_brute_force_sympy_L2(rng):
    """Whole CGTP at L = 2 written out from sympy's exact coefficients."""
    from sympy.physics.wigner import clebsch_gordan
    L = 2
    x1 = rng.standard_normal((3, 9))
    x2 = rng.standard_normal((3, 9))
    z = oracle.cgtp(L, x1, x2)
    for l1, l2, l3 in _paths(L):
        want = np.zeros((3, 2 * l3 + 1))
        for m3 in range(-l3, l3 + 1):
            for m1 in range(-l1, l1 + 1):
                m2 = m3 - m1
                if abs(m2) > l2:
                    continue
                c = float(clebsch_gordan(l1, l2, l3, m1, m2, m3))
                want[:, m3 + l3] += c * x1[:, l1 * l1 + l1 + m1] * x2[:, l2 * l2 + l2 + m2]
        np.testing.assert_allclose(_path(z, L, l1, l2, l3), want, atol=1e-14)


def test_output_layout_is_a_bijection():
    for L in (0, 1, 3, 6):
        seen = np.zeros(oracle.num_outputs(L), dtype=int)
        for l1, l2, l3 in _paths(L):
            off = oracle.path_offset(L, l1, l2, l3)
            seen[off:off + 2 * l3 + 1] += 1
        assert (seen == 1).all()
        assert oracle.path_offset(L, 1, 1, 3) == -1


def test_special_cases(rng):
    L = 5
    x1 = rng.standard_normal((2, 36))
    x2 = rng.standard_normal((2, 36))
    z = oracle.cgtp(L, x1, x2)
    for l in range(L + 1):
        # (0, l, l): scalar times irrep
        np.testing.assert_allclose(_path(z, L, 0, l, l), x1[:, :1] * x2[:, block_slice(l)], atol=1e-14)
        np.testing.assert_allclose(_path(z, L, l, 0, l), x1[:, block_slice(l)] * x2[:, :1], atol=1e-14)
        # (l, l, 0): the invariant sum_m (-1)^(l-m) x1_m x2_-m / sqrt(2l+1)
        a, b = x1[:, block_slice(l)], x2[:, block_slice(l)]
        sgn = np.array([(-1) ** (l - m) for m in range(-l, l + 1)])
        want = (a * sgn * b[:, ::-1]).sum(1) / math.sqrt(2 * l + 1)
        np.testing.assert_allclose(_path(z, L, l, l, 0)[:, 0], want, atol=1e-13)
    # stretched: m3 = l1 + l2 is the single product of the top components
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            top = _path(z, L, l1, l2, l1 + l2)[:, -1]
            np.testing.assert_allclose(top, x1[:, l1 * l1 + 2 * l1] * x2[:, l2 * l2 + 2 * l2], atol=1e-13)
    # L = 0: a single product
    z0 = oracle.cgtp(0, x1[:, :1], x2[:, :1])
    np.testing.assert_allclose(z0[:, 0], x1[:, 0] * x2[:, 0], atol=0)


def test_block_energy_identity(rng):
    """CG unitarity: sum_l3 |z^(l1,l2,l3)|^2 = |x1^(l1)|^2 |x2^(l2)|^2 (Appendix D.1)."""
    L = 6
    x1 = rng.standard_normal((4, 49))
    x2 = rng.standard_normal((4, 49))
    z = oracle.cgtp(L, x1, x2)
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            e = sum((_path(z, L, l1, l2, l3) ** 2).sum(1) for l3 in range(abs(l1 - l2), l1 + l2 + 1))
            want = (x1[:, block_slice(l1)] ** 2).sum(1) * (x2[:, block_slice(l2)] ** 2).sum(1)
            np.testing.assert_allclose(e, want, rtol=1e-12)


def test_exchange_symmetry(rng):
    """z^(l2,l1,l3)(x2,x1) = (-1)^(l1+l2-l3) z^(l1,l2,l3)(x1,x2); odd paths vanish for x1 = x2."""
    L = 5
    x1 = rng.standard_normal((3, 36))
    x2 = rng.standard_normal((3, 36))
    z12 = oracle.cgtp(L, x1, x2)
    z21 = oracle.cgtp(L, x2, x1)
    zsq = oracle.cgtp(L, x1, x1)
    for l1, l2, l3 in _paths(L):
        s = (-1) ** (l1 + l2 - l3)
        np.testing.assert_allclose(_path(z21, L, l2, l1, l3), s * _path(z12, L, l1, l2, l3), atol=1e-13)
        if l1 == l2 and (2 * l1 + l3) % 2 == 1:
            np.testing.assert_allclose(_path(zsq, L, l1, l1, l3), 0.0, atol=1e-13)


def _cart_to_sph(v):
    """Spherical components (q = -1, 0, +1) of a Cartesian vector, standard convention."""
    x, y, z = v[..., 0], v[..., 1], v[..., 2]
    return np.stack([(x - 1j * y) / math.sqrt(2), z + 0j, -(x + 1j * y) / math.sqrt(2)], axis=-1)


def test_cross_and_dot_products(rng):
    """l = 1 paths against Cartesian algebra: (a(x)b)^(1) = (i/sqrt 2)(a x b), (a(x)b)^(0) = -(a.b)/sqrt 3.

    The cross product is the antisymmetric interaction Section 5.1 is built on;
    with standard spherical components its constant is i/sqrt(2) (the paper
    writes -1/sqrt(2), which holds for a different component phase).
    """
    a = rng.standard_normal((5, 3))
    b = rng.standard_normal((5, 3))
    L = 1
    pad = lambda v: np.concatenate([np.zeros((5, 1), complex), _cart_to_sph(v)], axis=1)
    z = oracle.cgtp_complex(L, pad(a), pad(b))
    np.testing.assert_allclose(_path(z, L, 1, 1, 1), 1j / math.sqrt(2) * _cart_to_sph(np.cross(a, b)), atol=1e-14)
    np.testing.assert_allclose(_path(z, L, 1, 1, 0)[:, 0], -(a * b).sum(1) / math.sqrt(3), atol=1e-14)


def _quadrature_grid(n_theta, n_phi):
    xs, ws = np.polynomial.legendre.leggauss(n_theta)
    theta = np.arccos(xs)
    phi = 2 * np.pi * np.arange(n_phi) / n_phi
    T, P = np.meshgrid(theta, phi, indexing="ij")
    W = np.repeat(ws[:, None] * (2 * np.pi / n_phi), n_phi, axis=1)
    return T, P, W


def test_gaunt_quadrature(rng):
    """Symmetric (even-sum) paths against the Gaunt integral of Section 3.3.

    For f_i = sum_m x_i,m Y_li^m, the integral of f1 f2 conj(Y_l3^m3) over the
    sphere, done by quadrature of scipy's harmonics, equals
    sqrt((2l1+1)(2l2+1) / (4 pi (2l3+1))) C^{l3 0}_{l1 0 l2 0} z^(l1,l2,l3)_m3.
    """
    L = 4
    x1 = rng.standard_normal((1, 25))[0]
    x2 = rng.standard_normal((1, 25))[0]
    z = oracle.cgtp(L, x1[None], x2[None])[0]
    T, P, W = _quadrature_grid(3 * L + 2, 6 * L + 2)
    Y = {(l, m): _sph_harm(l, m, T, P) for l in range(2 * L + 1) for m in range(-l, l + 1)}
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            f1 = sum(x1[l1 * l1 + l1 + m] * Y[l1, m] for m in range(-l1, l1 + 1))
            f2 = sum(x2[l2 * l2 + l2 + m] * Y[l2, m] for m in range(-l2, l2 + 1))
            for l3 in range(abs(l1 - l2), l1 + l2 + 1, 2):
                c0 = oracle.cg(l1, 0, l2, 0, l3, 0)
                k = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) / (4 * math.pi * (2 * l3 + 1))) * c0
                got = k * _path(z, L, l1, l2, l3)
                want = np.array([(W * f1 * f2 * np.conj(Y[l3, m3])).sum() for m3 in range(-l3, l3 + 1)])
                np.testing.assert_allclose(got, want.real, atol=1e-12)
                assert np.abs(want.imag).max() < 1e-12


def _wigner_D(l, R, rng):
    """Matrix D with x' = D x for f(r) = sum x_m Y_l^m(r) -> f(R^-1 r), fitted from scipy's harmonics."""
    pts = rng.standard_normal((8 * (2 * l + 1) + 8, 3))
    pts /= np.linalg.norm(pts, axis=1, keepdims=True)
    back = R.inv().apply(pts)

    def Ymat(p):
        th = np.arccos(np.clip(p[:, 2], -1, 1))
        ph = np.arctan2(p[:, 1], p[:, 0])
        return np.stack([_sph_harm(l, m, th, ph) for m in range(-l, l + 1)], axis=1)

    A, B = Ymat(pts), Ymat(back)
    D, *_ = np.linalg.lstsq(A, B, rcond=None)
    return D


def test_rotation_equivariance(rng):
    """z(D x1, D x2) = D z(x1, x2) for random rotations (equivariance, Section 1)."""
    from scipy.spatial.transform import Rotation
    L = 3
    for trial in range(3):
        R = Rotation.random(random_state=int(rng.integers(1 << 30)))
        D = {l: _wigner_D(l, R, rng) for l in range(2 * L + 1)}
        np.testing.assert_allclose(D[2] @ D[2].conj().T, np.eye(5), atol=1e-10)
        x1 = rng.standard_normal((2, 16))
        x2 = rng.standard_normal((2, 16))
        rot = lambda x: np.concatenate([x[:, block_slice(l)] @ D[l].T for l in range(L + 1)], axis=1)
        z = oracle.cgtp_complex(L, x1.astype(complex), x2.astype(complex))
        zr = oracle.cgtp_complex(L, rot(x1), rot(x2))
        for l1, l2, l3 in _paths(L):
            np.testing.assert_allclose(_path(zr, L, l1, l2, l3), _path(z, L, l1, l2, l3) @ D[l3].T, atol=1e-10)


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.cgtp(2, np.zeros((1, 9)), np.zeros((1, 8)))
    with pytest.raises(RuntimeError):
        oracle.cgtp(-1, np.zeros((1, 0)), np.zeros((1, 0)))

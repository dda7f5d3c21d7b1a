"""Pins of the real-basis CGTP oracle (oracle.cgtp_real) to facts it does not
compute itself:

* even paths: the generalized Gaunt formula read in the real basis, i.e. the
  integral of three real harmonics (built from scipy's complex ones, exact
  Gauss-Legendre x equispaced quadrature) divided by K_ss = sqrt((2l1+1)(2l2+1)
  / (4 pi (2l3+1))) C^{l3 0}_{l1 0 l2 0} (sympy);
* degree 1: path (1, 1, 0) is -a.b/sqrt(3) and path (1, 1, 1) the cross product
  over sqrt(2), with the real basis' order (y, z, x) for m = -1, 0, 1;
* orthogonality of the real CG tensor: each block keeps the norm, sum over l3 of
  |z(l1, l2, l3)|^2 = |r1^(l1)|^2 |r2^(l2)|^2;
* rotation equivariance with real Wigner matrices fitted from real harmonics;
* real outputs for real inputs, and the degree-0 input as a plain scale.
"""
import math

import numpy as np
import pytest

import oracle

from test_oracle import _paths, _path, _sph_harm


def _real_harm(l, m, th, ph):
    """Y^R_{l,m}: sqrt(2) (-1)^m Re Y_l^m (m > 0), Y_l^0, sqrt(2) (-1)^m Im Y_l^|m| (m < 0)."""
    if m == 0:
        return _sph_harm(l, 0, th, ph).real
    y = _sph_harm(l, abs(m), th, ph)
    return math.sqrt(2.0) * (-1) ** abs(m) * (y.real if m > 0 else y.imag)


def _grid(n):
    x, w = np.polynomial.legendre.leggauss(n)
    nphi = 2 * n + 1
    ph = 2 * np.pi * np.arange(nphi) / nphi
    TH, PH = np.meshgrid(np.arccos(x), ph, indexing="ij")
    W = np.outer(w, np.full(nphi, 2 * np.pi / nphi))
    return TH, PH, W


def test_even_paths_are_the_real_gaunt_integral():
    from sympy.physics.quantum.cg import CG
    L = 3
    TH, PH, W = _grid(2 * L + 2)
    Y = {(l, m): _real_harm(l, m, TH, PH) for l in range(2 * L + 1) for m in range(-l, l + 1)}
    n = (L + 1) ** 2
    eye = np.eye(n)
    for l1, l2, l3 in _paths(L):
        if (l1 + l2 + l3) % 2:
            continue
        c0 = float(CG(l1, 0, l2, 0, l3, 0).doit())
        K = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) / (4 * math.pi * (2 * l3 + 1))) * c0
        for m1 in range(-l1, l1 + 1):
            for m2 in range(-l2, l2 + 1):
                z = oracle.cgtp_real(L, eye[l1 * l1 + l1 + m1], eye[l2 * l2 + l2 + m2])
                got = _path(z, L, l1, l2, l3)[0]
                want = np.array([(W * Y[l1, m1] * Y[l2, m2] * Y[l3, m3]).sum() for m3 in range(-l3, l3 + 1)]) / K
                np.testing.assert_allclose(got, want, atol=1e-12)


def test_degree_one_dot_and_cross():
    rng = np.random.default_rng(3)
    a, b = rng.standard_normal((2, 5, 4))
    z = oracle.cgtp_real(1, a, b)
    cart = lambda v: v[:, [3, 1, 2]]             # (x, y, z) from the real basis' (y, z, x)
    back = lambda v: v[:, [1, 2, 0]]
    np.testing.assert_allclose(_path(z, 1, 1, 1, 0)[:, 0], -(a[:, 1:] * b[:, 1:]).sum(1) / math.sqrt(3), atol=1e-13)
    np.testing.assert_allclose(_path(z, 1, 1, 1, 1), back(np.cross(cart(a), cart(b))) / math.sqrt(2), atol=1e-13)


@pytest.mark.parametrize("L", [2, 5])
def test_blocks_keep_the_norm(L):
    rng = np.random.default_rng(L)
    r1, r2 = rng.standard_normal((2, 3, (L + 1) ** 2))
    z = oracle.cgtp_real(L, r1, r2)
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            got = sum((_path(z, L, l1, l2, l3) ** 2).sum(1) for l3 in range(abs(l1 - l2), l1 + l2 + 1))
            want = (r1[:, l1 * l1:(l1 + 1) ** 2] ** 2).sum(1) * (r2[:, l2 * l2:(l2 + 1) ** 2] ** 2).sum(1)
            np.testing.assert_allclose(got, want, rtol=1e-12)


def _real_wigner(l, R, rng):
    """Real D with r' = D r for f(x) = sum r_m Y^R_lm(x) -> f(R^-1 x), fitted from real harmonics."""
    pts = rng.standard_normal((8 * (2 * l + 1) + 8, 3))
    pts /= np.linalg.norm(pts, axis=1, keepdims=True)
    back = R.inv().apply(pts)

    def Ymat(p):
        th = np.arccos(np.clip(p[:, 2], -1, 1))
        ph = np.arctan2(p[:, 1], p[:, 0])
        return np.stack([_real_harm(l, m, th, ph) for m in range(-l, l + 1)], axis=1)

    D, *_ = np.linalg.lstsq(Ymat(pts), Ymat(back), rcond=None)
    return D


def test_rotation_equivariance_real_basis():
    from scipy.spatial.transform import Rotation
    rng = np.random.default_rng(11)
    L = 3
    for _ in range(2):
        R = Rotation.random(random_state=int(rng.integers(1 << 30)))
        D = {l: _real_wigner(l, R, rng) for l in range(2 * L + 1)}
        np.testing.assert_allclose(D[3] @ D[3].T, np.eye(7), atol=1e-10)
        r1, r2 = rng.standard_normal((2, 2, (L + 1) ** 2))
        rot = lambda x: np.concatenate([x[:, l * l:(l + 1) ** 2] @ D[l].T for l in range(L + 1)], axis=1)
        z, zr = oracle.cgtp_real(L, r1, r2), oracle.cgtp_real(L, rot(r1), rot(r2))
        for l1, l2, l3 in _paths(L):
            np.testing.assert_allclose(_path(zr, L, l1, l2, l3), _path(z, L, l1, l2, l3) @ D[l3].T, atol=1e-10)


def test_degree_zero_input_scales():
    rng = np.random.default_rng(5)
    L = 4
    r1, r2 = rng.standard_normal((2, 3, (L + 1) ** 2))
    r1[:, 1:] = 0.0
    z = oracle.cgtp_real(L, r1, r2)
    for l2 in range(L + 1):
        np.testing.assert_allclose(_path(z, L, 0, l2, l2), r1[:, :1] * r2[:, l2 * l2:(l2 + 1) ** 2], atol=1e-13)

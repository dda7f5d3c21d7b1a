"""Pins of the oracle's CGTP gradients (oracle.cgtp_backward) to properties the
mathematics fixes, none of which re-types the oracle's sum:

* the derivative by its definition: the CGTP is bilinear, so the directional
  derivative along x1 (or x2) is the forward oracle evaluated on the direction
  itself; on unit rows this gives the gradient column by column;
* Euler's identity for a bilinear map: <gx1, x1> = <gx2, x2> = <g, z>;
* exchange symmetry: z(x2, x1) is z(x1, x2) with paths (l2, l1, l3) and sign
  (-1)^(l1+l2-l3), so swapping the inputs and permuting g swaps the gradients;
* a closed form: with x1 of degree 0 only, gx2 is x1_0 times g on the paths
  (0, l2, l2) (C^{l2 m}_{0 0 l2 m} = 1);
* rotation equivariance: gx1(conj(D) g, D x2) = conj(D) gx1(g, x2) for unitary
  Wigner matrices D fitted from scipy's harmonics.
"""
import math

import numpy as np
import pytest

import oracle

from test_oracle import _paths, _path, _wigner_D


@pytest.fixture
def rng():
    return np.random.default_rng(20260)


def _rows(L, N, rng):
    n = (L + 1) ** 2
    return rng.standard_normal((N, n)), rng.standard_normal((N, n)), rng.standard_normal((N, n * n))


@pytest.mark.parametrize("L", [0, 1, 2, 3])
def test_gradient_is_the_derivative_on_unit_rows(L, rng):
    x1, x2, g = _rows(L, 3, rng)
    gx1, gx2 = oracle.cgtp_backward(L, x1, x2, g)
    n = (L + 1) ** 2
    for k in range(n):
        e = np.zeros_like(x1)
        e[:, k] = 1.0
        d1 = (g * oracle.cgtp(L, e, x2)).sum(1)     # d/dt <g, z(x1 + t e_k, x2)>
        d2 = (g * oracle.cgtp(L, x1, e)).sum(1)
        np.testing.assert_allclose(gx1[:, k], d1, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(gx2[:, k], d2, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("L", [4, 7])
def test_directional_derivative(L, rng):
    x1, x2, g = _rows(L, 4, rng)
    d1, d2 = rng.standard_normal(x1.shape), rng.standard_normal(x2.shape)
    gx1, gx2 = oracle.cgtp_backward(L, x1, x2, g)
    np.testing.assert_allclose((gx1 * d1).sum(1), (g * oracle.cgtp(L, d1, x2)).sum(1), rtol=1e-11)
    np.testing.assert_allclose((gx2 * d2).sum(1), (g * oracle.cgtp(L, x1, d2)).sum(1), rtol=1e-11)


@pytest.mark.parametrize("L", [2, 5, 9])
def test_euler_identity(L, rng):
    x1, x2, g = _rows(L, 5, rng)
    gx1, gx2 = oracle.cgtp_backward(L, x1, x2, g)
    want = (g * oracle.cgtp(L, x1, x2)).sum(1)
    np.testing.assert_allclose((gx1 * x1).sum(1), want, rtol=1e-11)
    np.testing.assert_allclose((gx2 * x2).sum(1), want, rtol=1e-11)


def test_exchange_symmetry(rng):
    L = 4
    x1, x2, g = _rows(L, 3, rng)
    gs = np.empty_like(g)
    for l1, l2, l3 in _paths(L):
        a = oracle.path_offset(L, l1, l2, l3)
        b = oracle.path_offset(L, l2, l1, l3)
        gs[:, b:b + 2 * l3 + 1] = (-1) ** (l1 + l2 - l3) * g[:, a:a + 2 * l3 + 1]
    gx1, gx2 = oracle.cgtp_backward(L, x1, x2, g)
    hx1, hx2 = oracle.cgtp_backward(L, x2, x1, gs)
    np.testing.assert_allclose(hx1, gx2, atol=1e-12)
    np.testing.assert_allclose(hx2, gx1, atol=1e-12)


def test_degree_zero_closed_form(rng):
    L = 5
    x1, x2, g = _rows(L, 3, rng)
    x1[:, 1:] = 0.0
    _, gx2 = oracle.cgtp_backward(L, x1, x2, g)
    for l2 in range(L + 1):
        want = x1[:, :1] * _path(g, L, 0, l2, l2)
        np.testing.assert_allclose(gx2[:, l2 * l2:(l2 + 1) ** 2], want, atol=1e-13)


def _backward_complex(L, x1, x2, g):
    """Complex-bilinear extension of the gradients (four real oracle calls each)."""
    def part(a, b, c):
        return oracle.cgtp_backward(L, a, b, c)
    out1 = np.zeros(x1.shape, complex)
    out2 = np.zeros(x2.shape, complex)
    # gx1 is bilinear in (g, x2), gx2 in (g, x1)
    for (gp, gs), (xp, xs) in (((g.real, 1), (x2.real, 1)), ((g.imag, 1j), (x2.imag, 1j)),
                               ((g.real, 1), (x2.imag, 1j)), ((g.imag, 1j), (x2.real, 1))):
        out1 += gs * xs * part(np.zeros(x1.shape), xp, gp)[0]
    for (gp, gs), (xp, xs) in (((g.real, 1), (x1.real, 1)), ((g.imag, 1j), (x1.imag, 1j)),
                               ((g.real, 1), (x1.imag, 1j)), ((g.imag, 1j), (x1.real, 1))):
        out2 += gs * xs * part(xp, np.zeros(x2.shape), gp)[1]
    return out1, out2


def test_rotation_equivariance_of_the_gradients(rng):
    from scipy.spatial.transform import Rotation
    L = 3
    blk = lambda l: slice(l * l, (l + 1) ** 2)
    for trial in range(2):
        R = Rotation.random(random_state=int(rng.integers(1 << 30)))
        D = {l: _wigner_D(l, R, rng) for l in range(2 * L + 1)}
        x1, x2, g = _rows(L, 2, rng)
        rot = lambda x, conj=False: np.concatenate(
            [x[:, blk(l)] @ (D[l].conj() if conj else D[l]).T for l in range(L + 1)], axis=1)
        gr = np.zeros(g.shape, complex)
        for l1, l2, l3 in _paths(L):
            a = oracle.path_offset(L, l1, l2, l3)
            gr[:, a:a + 2 * l3 + 1] = g[:, a:a + 2 * l3 + 1] @ D[l3].conj().T
        gx1, gx2 = _backward_complex(L, x1.astype(complex), x2.astype(complex), g.astype(complex))
        hx1, hx2 = _backward_complex(L, rot(x1), rot(x2), gr)
        np.testing.assert_allclose(hx1, rot(gx1, conj=True), atol=1e-10)
        np.testing.assert_allclose(hx2, rot(gx2, conj=True), atol=1e-10)


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.cgtp_backward(2, np.zeros((1, 9)), np.zeros((1, 9)), np.zeros((1, 80)))

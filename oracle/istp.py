"""Oracle for the MIMO irrep-signal tensor products: TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The GPU library never imports or calls
it.

Two products of two feature rows, each the (0,0,0) or (1,1,1) case of the
irrep-signal tensor product of Section 4.3, in the multiple-input,
multiple-output setting of Appendix D (every input irrep lifted into one
signal, every output irrep read back from one product):

* ``gaunt_tp`` (s = 0, the Gaunt tensor product of Section 3.3): inputs hold
  one copy of each degree l = 0..L (index l^2 + l + m), outputs one copy of
  each degree l3 = 0..2L (index l3^2 + l3 + m3).  The result is the integral
  of f1 f2 conj(Y_l3^m3) over the sphere for f_i = sum x_i,lm Y_l^m, written
  with the integral of three spherical harmonics:

      z[l3, m3] = sum_{l1, l2} g(l1, l2, l3) (x1^(l1) (x) x2^(l2))^(l3)_{m3},
      g = sqrt((2 l1 + 1)(2 l2 + 1) / (4 pi (2 l3 + 1))) C^{l3 0}_{l1 0 l2 0}.

* ``vector_tp`` (s = 1, the vector signal tensor product of Section 5): the
  inputs are coefficients of tensor spherical harmonics Y^{l,1}_{j,m}
  (Definition 4.1) with labels (j, l), l = 0..L, |j - l| <= 1, j >= 0
  (3 (L+1)^2 numbers); the outputs are the coefficients of the (1)-coupled
  pointwise product in the same basis up to l3 = 2L (3 (2L+1)^2 numbers).
  The steps are those of the encoding / interaction / decoding of
  Appendix D.1, done on coefficients instead of a grid:

      1. a[q][l][ml] = sum_j C^{j, ml+q}_{l, ml, 1, q} x^(j,l)_{ml+q}
         (scalar-harmonic coefficients of spherical component q of the signal);
      2. b[q] = sum_{q1+q2=q} C^{1 q}_{1 q1 1 q2} gaunt_tp(a1[q1], a2[q2])
         (the (1) part of the pointwise tensor product, Section 4.3);
      3. z^(j3,l3)_{m3} = sum_q C^{j3 m3}_{l3, m3-q, 1, q} b[q][l3][m3-q]
         (coefficients in the orthonormal basis of Definition 4.1).

Row layout of the vector product: labels ordered by l, then j = l-1, l, l+1
(for l = 0 only j = 1), components m = -j..j; label (j, l) starts at
3 l^2 + {0, 2l - 1, 4l}[j - l + 1].

The coupling sums come from the CGTP oracle (``oracle.cgtp``, the plain
double sum of the CGTP definition) and its Racah-formula coefficients.
"""
from __future__ import annotations

import math

import numpy as np

from . import cg as _cg
from . import cgtp as _cgtp
from . import path_offset as _path_offset


def gaunt_size(L: int) -> int:
    return (L + 1) ** 2


def vector_size(L: int) -> int:
    return 3 * (L + 1) ** 2


def vector_labels(L: int):
    """(j, l) labels of a vector-product row, in row order."""
    out = []
    for l in range(L + 1):
        for j in (l - 1, l, l + 1):
            if j >= 0 and abs(j - l) <= 1 and j + l >= 1:
                out.append((j, l))
    return out


def vector_offset(j: int, l: int) -> int:
    """First column of label (j, l) in a vector-product row."""
    if l < 0 or j < 0 or abs(j - l) > 1 or j + l < 1:
        raise ValueError("(%d, %d) is not a vector-harmonic label" % (j, l))
    return 3 * l * l + (0, 2 * l - 1, 4 * l)[j - l + 1]


def _rows(x, n):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if a.ndim == 1:
        a = a[None]
    if a.shape[1] != n:
        raise ValueError("expected rows of %d values, got %s" % (n, a.shape))
    return a


def gaunt_tp(L: int, x1, x2, threads: int = 0) -> np.ndarray:
    """(0,0,0) product (Section 3.3).  x1, x2: [N, (L+1)^2] real; returns [N, (2L+1)^2]."""
    a = _rows(x1, gaunt_size(L))
    b = _rows(x2, gaunt_size(L))
    if a.shape != b.shape:
        raise ValueError("inputs must have the same shape")
    z = _cgtp(L, a, b, threads)
    out = np.zeros((a.shape[0], (2 * L + 1) ** 2))
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                if (l1 + l2 + l3) & 1:
                    continue   # C^{l3 0}_{l1 0 l2 0} vanishes
                g = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) / (4 * math.pi * (2 * l3 + 1))) * _cg(l1, 0, l2, 0, l3, 0)
                off = _path_offset(L, l1, l2, l3)
                out[:, l3 * l3: (l3 + 1) ** 2] += g * z[:, off: off + 2 * l3 + 1]
    return out


def vector_components(L: int, x) -> np.ndarray:
    """Step 1: [N, 3 (q = -1, 0, +1), (L+1)^2] scalar-harmonic coefficients of the vector signal."""
    x = _rows(x, vector_size(L))
    a = np.zeros((x.shape[0], 3, (L + 1) ** 2))
    for j, l in vector_labels(L):
        o = vector_offset(j, l)
        for q in (-1, 0, 1):
            for ml in range(-l, l + 1):
                mj = ml + q
                if abs(mj) <= j:
                    a[:, q + 1, l * l + l + ml] += _cg(l, ml, 1, q, j, mj) * x[:, o + j + mj]
    return a


def vector_tp(L: int, x1, x2, threads: int = 0) -> np.ndarray:
    """(1,1,1) product (Section 5).  x1, x2: [N, 3 (L+1)^2] real; returns [N, 3 (2L+1)^2]."""
    a1 = vector_components(L, x1)
    a2 = vector_components(L, x2)
    if a1.shape != a2.shape:
        raise ValueError("inputs must have the same shape")
    n = a1.shape[0]
    Lo = 2 * L
    b = np.zeros((n, 3, (Lo + 1) ** 2))
    for q1 in (-1, 0, 1):
        for q2 in (-1, 0, 1):
            q = q1 + q2
            if abs(q) > 1:
                continue
            c = _cg(1, q1, 1, q2, 1, q)
            if c == 0.0:
                continue
            b[:, q + 1] += c * gaunt_tp(L, a1[:, q1 + 1], a2[:, q2 + 1], threads)
    out = np.zeros((n, vector_size(Lo)))
    for j3, l3 in vector_labels(Lo):
        o = vector_offset(j3, l3)
        for m3 in range(-j3, j3 + 1):
            for q in (-1, 0, 1):
                ml = m3 - q
                if abs(ml) <= l3:
                    out[:, o + j3 + m3] += _cg(l3, ml, 1, q, j3, m3) * b[:, q + 1, l3 * l3 + l3 + ml]
    return out

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

``spin_tp`` is the same product for any spin s (s = 2: tensor spherical
harmonics of rank 2).  ``product_vjp`` gives the gradients of sum(g * z) w.r.t. both inputs by the
plain definition of a bilinear map's derivatives.  ``channel_product`` is the
layer around a product: C channels, the second input per channel or shared,
and one weight per (channel, irrep label) on each input and on the output.

Both products take separate degree bounds for the two inputs and the output
(L, L2, Lo; by default L2 = L and Lo = L + L2).

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


def gaunt_tp(L: int, x1, x2, threads: int = 0, L2: int | None = None, Lo: int | None = None) -> np.ndarray:
    """(0,0,0) product (Section 3.3).  x1: [N, (L+1)^2], x2: [N, (L2+1)^2] real (L2 = L by default);
    returns the degrees 0..Lo (default L + L2): [N, (Lo+1)^2]."""
    L1 = L
    L2 = L1 if L2 is None else L2
    Lo = L1 + L2 if Lo is None else Lo
    a = _rows(x1, gaunt_size(L1))
    b = _rows(x2, gaunt_size(L2))
    if a.shape[0] != b.shape[0]:
        raise ValueError("inputs must hold the same number of rows")
    Lm = max(L1, L2)
    pad = lambda v, l: np.concatenate([v, np.zeros((v.shape[0], gaunt_size(Lm) - gaunt_size(l)))], axis=1)
    z = _cgtp(Lm, pad(a, L1), pad(b, L2), threads)
    out = np.zeros((a.shape[0], (Lo + 1) ** 2))
    for l1 in range(L1 + 1):
        for l2 in range(L2 + 1):
            for l3 in range(abs(l1 - l2), min(l1 + l2, Lo) + 1):
                if (l1 + l2 + l3) & 1:
                    continue   # C^{l3 0}_{l1 0 l2 0} vanishes
                g = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) / (4 * math.pi * (2 * l3 + 1))) * _cg(l1, 0, l2, 0, l3, 0)
                off = _path_offset(Lm, l1, l2, l3)
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


def vector_tp(L: int, x1, x2, threads: int = 0, L2: int | None = None, Lo: int | None = None) -> np.ndarray:
    """(1,1,1) product (Section 5).  x1: [N, 3 (L+1)^2], x2: [N, 3 (L2+1)^2] real (L2 = L by default);
    returns the labels up to l = Lo (default L + L2): [N, 3 (Lo+1)^2]."""
    L1 = L
    L2 = L1 if L2 is None else L2
    Lo = L1 + L2 if Lo is None else Lo
    a1 = vector_components(L1, x1)
    a2 = vector_components(L2, x2)
    if a1.shape[0] != a2.shape[0]:
        raise ValueError("inputs must hold the same number of rows")
    n = a1.shape[0]
    b = np.zeros((n, 3, (Lo + 1) ** 2))
    for q1 in (-1, 0, 1):
        for q2 in (-1, 0, 1):
            q = q1 + q2
            if abs(q) > 1:
                continue
            c = _cg(1, q1, 1, q2, 1, q)
            if c == 0.0:
                continue
            b[:, q + 1] += c * gaunt_tp(L1, a1[:, q1 + 1], a2[:, q2 + 1], threads, L2=L2, Lo=Lo)
    out = np.zeros((n, vector_size(Lo)))
    for j3, l3 in vector_labels(Lo):
        o = vector_offset(j3, l3)
        for m3 in range(-j3, j3 + 1):
            for q in (-1, 0, 1):
                ml = m3 - q
                if abs(ml) <= l3:
                    out[:, o + j3 + m3] += _cg(l3, ml, 1, q, j3, m3) * b[:, q + 1, l3 * l3 + l3 + ml]
    return out


# ---------------------------------------------------------------- any spin s
#
# The (s, s, s) product for any s (the general irrep-signal tensor product of
# Section 4.3 with tensor spherical harmonics of spin s, Definition 4.1): labels
# (j, l), l = 0..L, |l - s| <= j <= l + s, (2 s + 1)(L + 1)^2 numbers per row
# (label (j, l) at (2 s + 1) l^2 + j^2 - (l - s)^2); the same three steps as
# ``vector_tp`` with spin s in place of 1:
#
#     a[q][l][ml] = sum_j C^{j, ml+q}_{l, ml, s, q} x^(j,l)_{ml+q},   q = -s..s
#     b[q] = sum_{q1+q2=q} C^{s q}_{s q1 s q2} gaunt_tp(a1[q1], a2[q2])
#     z^(j3,l3)_{m3} = sum_q C^{j3 m3}_{l3, m3-q, s, q} b[q][l3][m3-q]

def spin_labels(s: int, L: int):
    """(j, l) labels of a spin-s row, in row order (l, then j ascending)."""
    return [(j, l) for l in range(L + 1) for j in range(abs(l - s), l + s + 1)]


def spin_offset(s: int, j: int, l: int) -> int:
    if l < 0 or not (abs(l - s) <= j <= l + s):
        raise ValueError("(%d, %d) is not a spin-%d label" % (j, l, s))
    return (2 * s + 1) * l * l + j * j - (l - s) ** 2


def spin_size(s: int, L: int) -> int:
    return (2 * s + 1) * (L + 1) ** 2


def spin_components(s: int, L: int, x) -> np.ndarray:
    """[N, 2 s + 1 (q = -s..s), (L+1)^2] scalar-harmonic coefficients of the spin-s signal."""
    x = _rows(x, spin_size(s, L))
    a = np.zeros((x.shape[0], 2 * s + 1, (L + 1) ** 2))
    for j, l in spin_labels(s, L):
        o = spin_offset(s, j, l)
        for q in range(-s, s + 1):
            for ml in range(-l, l + 1):
                mj = ml + q
                if abs(mj) <= j:
                    a[:, q + s, l * l + l + ml] += _cg(l, ml, s, q, j, mj) * x[:, o + j + mj]
    return a


def spin_tp(s: int, L: int, x1, x2, threads: int = 0, L2: int | None = None, Lo: int | None = None) -> np.ndarray:
    """(s, s, s) product: x1 [N, (2s+1)(L+1)^2], x2 [N, (2s+1)(L2+1)^2]; returns labels up to l = Lo (default L + L2)."""
    L1 = L
    L2 = L1 if L2 is None else L2
    Lo = L1 + L2 if Lo is None else Lo
    a1 = spin_components(s, L1, x1)
    a2 = spin_components(s, L2, x2)
    if a1.shape[0] != a2.shape[0]:
        raise ValueError("inputs must hold the same number of rows")
    n = a1.shape[0]
    b = np.zeros((n, 2 * s + 1, (Lo + 1) ** 2))
    for q1 in range(-s, s + 1):
        for q2 in range(-s, s + 1):
            q = q1 + q2
            if abs(q) > s:
                continue
            c = _cg(s, q1, s, q2, s, q)
            if c == 0.0:
                continue
            b[:, q + s] += c * gaunt_tp(L1, a1[:, q1 + s], a2[:, q2 + s], threads, L2=L2, Lo=Lo)
    out = np.zeros((n, spin_size(s, Lo)))
    for j3, l3 in spin_labels(s, Lo):
        o = spin_offset(s, j3, l3)
        for m3 in range(-j3, j3 + 1):
            for q in range(-s, s + 1):
                ml = m3 - q
                if abs(ml) <= l3:
                    out[:, o + j3 + m3] += _cg(l3, ml, s, q, j3, m3) * b[:, q + s, l3 * l3 + l3 + ml]
    return out


def product_vjp(spin: int, L: int, x1, x2, g, threads: int = 0):
    """Gradients of sum(g * z(x1, x2)) w.r.t. x1 and x2 for the spin-0, 1 or 2 product above, by the
    plain definition: z is bilinear, so d/dx1[b] = sum_a g_a z_a(e_b, x2) and d/dx2[b] = sum_a g_a z_a(x1, e_b),
    with z evaluated by ``gaunt_tp`` / ``vector_tp`` on unit rows (one pair at a time).
    x1, x2: [N, n_in]; g: [N, n_out]; returns (grad_x1, grad_x2), each [N, n_in]."""
    fn = gaunt_tp if spin == 0 else (vector_tp if spin == 1 else (lambda *a_, **k_: spin_tp(spin, *a_, **k_)))
    size = lambda Lx: spin_size(spin, Lx)
    a = _rows(x1, size(L))
    b = _rows(x2, size(L))
    gg = _rows(g, size(2 * L))
    eye = np.eye(size(L))
    g1 = np.zeros_like(a)
    g2 = np.zeros_like(b)
    for n in range(a.shape[0]):
        j1 = fn(L, eye, np.repeat(b[n:n + 1], size(L), 0), threads)   # row k: z(e_k, x2)
        j2 = fn(L, np.repeat(a[n:n + 1], size(L), 0), eye, threads)   # row k: z(x1, e_k)
        g1[n] = j1 @ gg[n]
        g2[n] = j2 @ gg[n]
    return g1, g2


# ---------------------------------------------------------------- channels and label weights
#
# A layer holds C channels of the input feature.  Equivariant linear maps
# before and after the product can only scale each irrep label (Schur's
# lemma; the degrees-of-freedom count of Appendix E), so per pair n and
# channel c:
#
#     out[n, c] = wo[c] . P(w1[c] . x1[n, c], w2[c] . y)
#
# with y = x2[n, c], or x2[n] when the second input is shared by the
# channels, P the product above and "w . x" scaling every column of label k
# by w[k].  Weight rows list the labels in row order: degree l for spin 0,
# (j, l) as ``vector_labels`` gives them for spin 1.

def labels(spin: int, L: int):
    """(j, l) of every label of a row of degree bound L, in row order."""
    return [(l, l) for l in range(L + 1)] if spin == 0 else (vector_labels(L) if spin == 1 else spin_labels(spin, L))


def column_labels(spin: int, L: int) -> np.ndarray:
    """Label index (position in ``labels``) of every column of a row."""
    if spin == 0:
        return np.concatenate([np.full(2 * l + 1, l) for l in range(L + 1)])
    out = np.empty(spin_size(spin, L), dtype=np.int64)
    for k, (j, l) in enumerate(labels(spin, L)):
        o = spin_offset(spin, j, l)
        out[o: o + 2 * j + 1] = k
    return out


def channel_product(spin: int, L: int, x1, x2, w1=None, w2=None, wo=None, threads: int = 0) -> np.ndarray:
    """x1: [N, C, n_in]; x2: [N, C, n_in] or [N, n_in]; w1, w2: None, [C, n_lab(L)] or [N, C, n_lab(L)];
    wo: None, [C, n_lab(2L)] or [N, C, n_lab(2L)].  Returns [N, C, n_out] in fp64."""
    fn = gaunt_tp if spin == 0 else (vector_tp if spin == 1 else (lambda *a_, **k_: spin_tp(spin, *a_, **k_)))
    nin = spin_size(spin, L)
    a = np.asarray(x1, dtype=np.float64)
    if a.ndim != 3 or a.shape[2] != nin:
        raise ValueError("x1 must be [N, C, %d]" % nin)
    n, c = a.shape[:2]
    b = np.asarray(x2, dtype=np.float64)
    if b.shape == (n, nin):
        b = np.repeat(b[:, None, :], c, axis=1)
    elif b.shape != (n, c, nin):
        raise ValueError("x2 must be [N, C, %d] or [N, %d]" % (nin, nin))

    def scale(x, w, Lx):
        if w is None:
            return x
        nl = len(labels(spin, Lx))
        wt = np.asarray(w, dtype=np.float64)
        if wt.shape == (c, nl):
            wt = np.broadcast_to(wt, (n, c, nl))
        elif wt.shape != (n, c, nl):
            raise ValueError("weights must be [C, %d] or [N, C, %d]" % (nl, nl))
        return x * wt[:, :, column_labels(spin, Lx)]

    z = fn(L, scale(a, w1, L).reshape(n * c, nin), scale(b, w2, L).reshape(n * c, nin), threads)
    return scale(z.reshape(n, c, -1), wo, 2 * L)


# ---------------------------------------------------------------- real spherical harmonics
#
# Real harmonics with the Condon-Shortley phase carried over from Y_l^m:
#     Y^R_{l,m} = sqrt(2) (-1)^m Re Y_l^m      (m > 0)
#     Y^R_{l,0} = Y_l^0
#     Y^R_{l,m} = sqrt(2) (-1)^m Im Y_l^{|m|}  (m < 0)
# (index l^2 + l + m, as for the complex basis).  A real function
# f = sum r_lm Y^R_lm has complex coefficients c = to_complex(r), and the
# real-basis Gaunt product is the complex-basis one on c, read back in the real
# basis; the complex-basis product is bilinear with real coefficients, so it
# applies to complex inputs part by part.

def to_complex(L: int, r) -> np.ndarray:
    """Complex-basis coefficients [N, (L+1)^2] of the real-basis rows r."""
    r = _rows(r, gaunt_size(L))
    c = np.zeros(r.shape, dtype=complex)
    s = 1.0 / math.sqrt(2.0)
    for l in range(L + 1):
        o = l * l + l
        c[:, o] = r[:, o]
        for m in range(1, l + 1):
            c[:, o + m] = (-1) ** m * s * (r[:, o + m] - 1j * r[:, o - m])
            c[:, o - m] = s * (r[:, o + m] + 1j * r[:, o - m])
    return c


def to_real(L: int, c) -> np.ndarray:
    """Real-basis coefficients of a real function from its complex-basis coefficients [N, (L+1)^2]."""
    c = np.atleast_2d(np.asarray(c, dtype=complex))
    r = np.zeros(c.shape)
    s = math.sqrt(2.0)
    for l in range(L + 1):
        o = l * l + l
        r[:, o] = c[:, o].real
        for m in range(1, l + 1):
            r[:, o + m] = s * c[:, o - m].real
            r[:, o - m] = s * c[:, o - m].imag
    return r


def gaunt_tp_real(L: int, r1, r2, threads: int = 0) -> np.ndarray:
    """Gaunt product of real-basis rows: degrees 0..L in, 0..2L out, all in the real basis."""
    c1, c2 = to_complex(L, r1), to_complex(L, r2)
    f = lambda a, b: gaunt_tp(L, a, b, threads)
    z = (f(c1.real, c2.real) - f(c1.imag, c2.imag)) + 1j * (f(c1.real, c2.imag) + f(c1.imag, c2.real))
    return to_real(2 * L, z)


# Real basis for spin-s signals.  A real spin-s field sum c^(j,l)_m Y^{l,s}_{j,m}
# has c^(j,l)_{-m} = sigma (-1)^m conj(c^(j,l)_m) with sigma = (-1)^(l+s-j)
# (conj Y^{l,s}_{j,m} = (-1)^(m+l+s-j) Y^{l,s}_{j,-m} with Condon-Shortley
# phases for Y_l^m and the spherical basis vectors).  A label with sigma = +1
# takes the scalar real basis above; one with sigma = -1 takes it for i c
# (which is then Hermitian).  The spin-1 product of two real fields is i times
# a real field (the 1 (x) 1 -> 1 coupling is i / sqrt 2 times the cross
# product, up to the sign of the basis), so its output is read back after a
# factor i, which makes the product of two constant fields their cross product
# over sqrt 2 (times Y_0^0); spin 0 and 2 need none.

def _label_sigma(s: int, j: int, l: int) -> int:
    return -1 if (l + s - j) % 2 else 1


def spin_to_complex(s: int, L: int, r) -> np.ndarray:
    """Complex-basis coefficients [N, spin_size] of real-basis spin-s rows r."""
    r = _rows(r, spin_size(s, L))
    c = np.zeros(r.shape, dtype=complex)
    h = 1.0 / math.sqrt(2.0)
    for j, l in spin_labels(s, L):
        o = spin_offset(s, j, l) + j
        blk = np.zeros((r.shape[0], 2 * j + 1), dtype=complex)
        blk[:, j] = r[:, o]
        for m in range(1, j + 1):
            blk[:, j + m] = (-1) ** m * h * (r[:, o + m] - 1j * r[:, o - m])
            blk[:, j - m] = h * (r[:, o + m] + 1j * r[:, o - m])
        if _label_sigma(s, j, l) < 0:
            blk = -1j * blk
        c[:, o - j:o + j + 1] = blk
    return c


def spin_to_real(s: int, L: int, c) -> np.ndarray:
    """Real-basis coefficients of a real spin-s field from its complex-basis coefficients."""
    c = np.atleast_2d(np.asarray(c, dtype=complex))
    r = np.zeros(c.shape)
    h = math.sqrt(2.0)
    for j, l in spin_labels(s, L):
        o = spin_offset(s, j, l) + j
        blk = c[:, o - j:o + j + 1]
        if _label_sigma(s, j, l) < 0:
            blk = 1j * blk
        r[:, o] = blk[:, j].real
        for m in range(1, j + 1):
            r[:, o + m] = h * blk[:, j - m].real
            r[:, o - m] = h * blk[:, j - m].imag
    return r


SPIN_OUTPUT_PHASE = {0: 1.0, 1: 1j, 2: 1.0}


def spin_tp_real(s: int, L: int, r1, r2, threads: int = 0) -> np.ndarray:
    """(s, s, s) product of real-basis rows: labels up to l = L in, up to 2L out, all in the real basis."""
    c1, c2 = spin_to_complex(s, L, r1), spin_to_complex(s, L, r2)
    f = lambda a, b: spin_tp(s, L, a, b, threads)
    z = (f(c1.real, c2.real) - f(c1.imag, c2.imag)) + 1j * (f(c1.real, c2.imag) + f(c1.imag, c2.real))
    return spin_to_real(s, 2 * L, SPIN_OUTPUT_PHASE[s] * z)


def gaunt_tp_real_vjp(L: int, r1, r2, g, threads: int = 0):
    """Gradients of sum(g * gaunt_tp_real(r1, r2)) w.r.t. r1 and r2, by the plain definition of a bilinear
    map's derivatives (``gaunt_tp_real`` on unit rows, one pair at a time)."""
    a = _rows(r1, gaunt_size(L))
    b = _rows(r2, gaunt_size(L))
    gg = _rows(g, gaunt_size(2 * L))
    eye = np.eye(gaunt_size(L))
    g1 = np.zeros_like(a)
    g2 = np.zeros_like(b)
    for n in range(a.shape[0]):
        g1[n] = gaunt_tp_real(L, eye, np.repeat(b[n:n + 1], gaunt_size(L), 0), threads) @ gg[n]
        g2[n] = gaunt_tp_real(L, np.repeat(a[n:n + 1], gaunt_size(L), 0), eye, threads) @ gg[n]
    return g1, g2


def channel_product_vjp(spin: int, L: int, x1, x2, g, w1=None, w2=None, wo=None, threads: int = 0):
    """Gradients of sum(g * channel_product(x1, x2, w1, w2, wo)) w.r.t. x1 and x2 (x2 per channel, [N, C, n_in]):
    the chain rule through the label weights around ``product_vjp``."""
    a = np.asarray(x1, dtype=np.float64)
    b = np.asarray(x2, dtype=np.float64)
    gg = np.asarray(g, dtype=np.float64)
    n, c, nin = a.shape

    def col_weights(w, Lx):
        if w is None:
            return np.ones((n, c, spin_size(spin, Lx)))
        wt = np.asarray(w, dtype=np.float64)
        if wt.ndim == 2:
            wt = np.broadcast_to(wt, (n, c, wt.shape[1]))
        return wt[:, :, column_labels(spin, Lx)]

    s1, s2, so = col_weights(w1, L), col_weights(w2, L), col_weights(wo, 2 * L)
    r1, r2 = product_vjp(spin, L, (s1 * a).reshape(n * c, nin), (s2 * b).reshape(n * c, nin),
                         (so * gg).reshape(n * c, -1), threads)
    return s1 * r1.reshape(n, c, nin), s2 * r2.reshape(n, c, nin)

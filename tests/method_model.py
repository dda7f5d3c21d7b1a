"""fp64 numpy model of the GPU method, for tests only.

It follows the kernel's steps with the plan's own host math (Gauss-Legendre
nodes, normalised Legendre values, vector-coupling coefficients, 1/K from
Theorem 4.2 via ``cgtp_path_norm``) and ``numpy.fft`` in place of the LDS FFT:

  lift (Definition 4.1, l = j, s = 0 and s = 1) -> two real series packed per
  complex transform -> longitude synthesis -> unpack -> pointwise products
  (scalar-scalar, and the 1 (x) 1 -> 1 coupling, i.e. the cross product;
  or, for the alternate cover, scalar-vector and dot) -> longitude analysis ->
  Legendre projection on the northern rings with parity folding ->
  recombination with C^{j3 m3}_{l3, m3-q, 1, q} -> division by K.

It never imports the oracle; tests compare the two.  Checking it against the
oracle pins the plan's conventions (phases, K, grid exactness) on the CPU.
"""
from __future__ import annotations

import numpy as np

import paper_2602_21466_amd as lib


def _unpack(F):
    """Two Hermitian signals packed as F = fA + i fB -> (fA, fB)."""
    Fr = np.roll(F[:, ::-1], 1, axis=1)   # F at -k
    fa = 0.5 * (F + np.conj(Fr))
    fb = -0.5j * (F - np.conj(Fr))
    return fa, fb


def model_cgtp(L: int, x1: np.ndarray, x2: np.ndarray, cover: int = 0, n_theta: int = 0, n_phi: int = 0):
    x1 = np.atleast_2d(np.asarray(x1, dtype=np.float64))
    x2 = np.atleast_2d(np.asarray(x2, dtype=np.float64))
    N = x1.shape[0]
    out = np.zeros((N, (L + 1) ** 4))
    grid = lib._grid(n_theta, n_phi, "fp64", 0)
    for j1 in range(L + 1):
        for j2 in range(L + 1):
            nt, Phi = lib.cgtp_block_grid(L, j1, j2, grid)
            J, d = j1 + j2, abs(j1 - j2)
            R = nt // 2
            xs, ws = lib.cgtp_gauss_legendre(nt)
            xs, ws = xs[:R], 2.0 * ws[:R]            # northern rings, south folded in
            lmax = max(J, 0)
            pb = [lib.cgtp_legendre(lmax, x) for x in xs]

            def P(i, l, m):
                am = abs(m)
                if am > l:
                    return 0.0
                v = pb[i][l * (l + 1) // 2 + am]
                return -v if (m < 0 and am % 2) else v

            def lifts(x, j, i):
                """Coefficient series (index m mod Phi) of the scalar and q = -1, 0, +1 lifts."""
                a = {c: np.zeros((N, Phi)) for c in ("s", -1, 0, 1)}
                for m in range(-j, j + 1):
                    pv = P(i, j, m)
                    a["s"][:, m % Phi] = x[:, j * j + j + m] * pv
                    for q in (-1, 0, 1):
                        mj = m + q
                        if abs(mj) <= j:
                            a[q][:, m % Phi] = lib.cgtp_cg_vector(j, m, q, j, mj) * x[:, j * j + j + mj] * pv
                return a

            B = {c: np.zeros((N, J + 1, 2 * J + 1)) for c in ("s", "dot", -1, 0, 1)}
            for i in range(R):
                a1, a2 = lifts(x1, j1, i), lifts(x2, j2, i)
                f1, f2 = {}, {}
                for a, f in ((a1, f1), (a2, f2)):
                    f["s"], f[0] = _unpack(np.fft.ifft(a["s"] + 1j * a[0], axis=1) * Phi)
                    f[-1], f[1] = _unpack(np.fft.ifft(a[-1] + 1j * a[1], axis=1) * Phi)
                g = {"s": f1["s"] * f2["s"]}
                for q in (-1, 0, 1):
                    g[q] = sum(lib.cgtp_cg_vector(1, q1, q - q1, 1, q) * f1[q1] * f2[q - q1]
                               for q1 in (-1, 0, 1) if abs(q - q1) <= 1)
                if cover == 1:
                    g["dot"] = sum(lib.cgtp_cg_vector(1, q, -q, 0, 0) * f1[q] * f2[-q] for q in (-1, 0, 1))
                    g["sv"] = {q: f1["s"] * f2[q] for q in (-1, 0, 1)}
                z1 = np.fft.fft(g["s"] + 1j * g[0], axis=1) * (2 * np.pi / Phi)
                z2 = np.fft.fft(g[-1] + 1j * g[1], axis=1) * (2 * np.pi / Phi)
                spec = {"s": z1.real, 0: z1.imag, -1: z2.real, 1: z2.imag}
                if cover == 1:
                    spec["dot"] = (np.fft.fft(g["dot"], axis=1) * (2 * np.pi / Phi)).real
                    spec["sv"] = {q: (np.fft.fft(g["sv"][q], axis=1) * (2 * np.pi / Phi)).real for q in (-1, 0, 1)}
                for l3 in range(d, J + 1, 2):
                    for m in range(-l3, l3 + 1):
                        w = ws[i] * P(i, l3, m)
                        for c in ("s", -1, 0, 1):
                            B[c][:, l3, m + J] += w * spec[c][:, m % Phi]
                        if cover == 1:
                            B["dot"][:, l3, m + J] += w * spec["dot"][:, m % Phi]
                            for q in (-1, 0, 1):
                                B.setdefault(("sv", q), np.zeros((N, J + 1, 2 * J + 1)))
                                B[("sv", q)][:, l3, m + J] += w * spec["sv"][q][:, m % Phi]
            off = lib.cgtp_path_offset(L, j1, j2, d)
            for j3 in range(d, J + 1):
                K, kind = lib.cgtp_path_norm(j1, j2, j3, cover)
                zz = np.zeros((N, 2 * j3 + 1))
                for m3 in range(-j3, j3 + 1):
                    if kind == 0:
                        zz[:, m3 + j3] = B["s"][:, j3, m3 + J]
                    elif kind == 3:
                        zz[:, m3 + j3] = B["dot"][:, j3, m3 + J]
                    else:
                        l3 = j3 - 1
                        for q in (-1, 0, 1):
                            m = m3 - q
                            if abs(m) <= l3:
                                src = B[q] if kind == 1 else B[("sv", q)]
                                zz[:, m3 + j3] += lib.cgtp_cg_vector(l3, m, q, j3, m3) * src[:, l3, m + J]
                base = off + j3 * j3 - d * d
                out[:, base:base + 2 * j3 + 1] = zz / K
    return out

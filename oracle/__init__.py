"""Oracle for the full Clebsch-Gordan tensor product: TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never imports, links or
calls it; the two share no code.

The numerical work is in ``cgtp_oracle.c`` (plain C, fp64, Racah-formula
Clebsch-Gordan coefficients in long double, naive O(L^6) double sum over
(m1, m2)).  This module only marshals numpy arrays through ctypes.

Complex inputs (used by the rotation-equivariance pins) are handled by
bilinearity: (a + ib) (x) (c + id) = a(x)c - b(x)d + i (a(x)d + b(x)c).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cgtp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compiles the oracle shared library with gcc (portable x86-64 code)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=False)
    lib = ctypes.CDLL(_LIB)
    lib.oracle_cg.restype = ctypes.c_double
    lib.oracle_cg.argtypes = [ctypes.c_int] * 6
    lib.oracle_cgtp.restype = ctypes.c_int
    lib.oracle_cgtp.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_int]
    lib.oracle_cg_block.restype = ctypes.c_int
    lib.oracle_cg_block.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    lib.oracle_num_outputs.restype = ctypes.c_int64
    lib.oracle_num_outputs.argtypes = [ctypes.c_int]
    lib.oracle_path_offset.restype = ctypes.c_int64
    lib.oracle_path_offset.argtypes = [ctypes.c_int] * 4
    lib.oracle_cgtp_backward.restype = ctypes.c_int
    lib.oracle_cgtp_backward.argtypes = [ctypes.c_int, ctypes.c_int64] + [ctypes.c_void_p] * 5 + [ctypes.c_int]
    lib.oracle_table_build_seconds.restype = ctypes.c_double
    lib.oracle_table_build_seconds.argtypes = []
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_max_threads.argtypes = []
    _lib = lib
    return lib


def cg(j1: int, m1: int, j2: int, m2: int, j: int, m: int) -> float:
    """C^{j m}_{j1 m1 j2 m2} (Condon-Shortley), Racah formula."""
    return _load().oracle_cg(j1, m1, j2, m2, j, m)


def cg_block(l1: int, l2: int, l3: int) -> np.ndarray:
    """Array [2 l3 + 1, 2 l1 + 1] of C^{l3 m3}_{l1 m1 l2 (m3 - m1)}."""
    out = np.zeros((2 * l3 + 1, 2 * l1 + 1), dtype=np.float64)
    rc = _load().oracle_cg_block(l1, l2, l3, out.ctypes.data)
    if rc != 0:
        raise ValueError("invalid triple (%d, %d, %d)" % (l1, l2, l3))
    return out


def num_outputs(L: int) -> int:
    return (L + 1) ** 4


def path_offset(L: int, l1: int, l2: int, l3: int) -> int:
    """Offset of path (l1, l2, l3) within one pair's output, -1 if not a path."""
    return int(_load().oracle_path_offset(L, l1, l2, l3))


def cgtp(L: int, x1, x2, threads: int = 0) -> np.ndarray:
    """Full CGTP in fp64.  x1, x2: [N, (L+1)^2] real; returns [N, (L+1)^4]."""
    a = np.ascontiguousarray(np.asarray(x1, dtype=np.float64))
    b = np.ascontiguousarray(np.asarray(x2, dtype=np.float64))
    if a.ndim == 1:
        a = a[None]
    if b.ndim == 1:
        b = b[None]
    if a.shape != b.shape or a.shape[1] != (L + 1) ** 2:
        raise ValueError("inputs must both be [N, (L+1)^2]")
    n = a.shape[0]
    out = np.empty((n, num_outputs(L)), dtype=np.float64)
    rc = _load().oracle_cgtp(L, n, a.ctypes.data, b.ctypes.data, out.ctypes.data, int(threads))
    if rc != 0:
        raise RuntimeError("oracle_cgtp failed (L=%d, N=%d)" % (L, n))
    return out


def cgtp_backward(L: int, x1, x2, g, threads: int = 0):
    """Gradients (gx1, gx2) of sum(g * cgtp(L, x1, x2)) in fp64: the derivative of the bilinear map by its
    definition, written out term by term (cgtp_oracle.c).  x1, x2: [N, (L+1)^2]; g: [N, (L+1)^4]."""
    a = np.ascontiguousarray(np.asarray(x1, dtype=np.float64))
    b = np.ascontiguousarray(np.asarray(x2, dtype=np.float64))
    gz = np.ascontiguousarray(np.asarray(g, dtype=np.float64))
    if a.ndim == 1:
        a, b, gz = a[None], b[None], gz[None]
    n = a.shape[0]
    if a.shape != b.shape or a.shape[1] != (L + 1) ** 2 or gz.shape != (n, num_outputs(L)):
        raise ValueError("x1, x2 must be [N, (L+1)^2] and g [N, (L+1)^4]")
    ga = np.empty_like(a)
    gb = np.empty_like(b)
    rc = _load().oracle_cgtp_backward(L, n, a.ctypes.data, b.ctypes.data, gz.ctypes.data, ga.ctypes.data,
                                      gb.ctypes.data, int(threads))
    if rc != 0:
        raise RuntimeError("oracle_cgtp_backward failed (L=%d, N=%d)" % (L, n))
    return ga, gb


def cgtp_complex(L: int, x1, x2, threads: int = 0) -> np.ndarray:
    """CGTP of complex inputs, by bilinearity of the real oracle."""
    x1 = np.asarray(x1, dtype=np.complex128)
    x2 = np.asarray(x2, dtype=np.complex128)
    rr = cgtp(L, x1.real, x2.real, threads)
    ii = cgtp(L, x1.imag, x2.imag, threads)
    ri = cgtp(L, x1.real, x2.imag, threads)
    ir = cgtp(L, x1.imag, x2.real, threads)
    return (rr - ii) + 1j * (ri + ir)


def _degree_to_real(l: int, c) -> np.ndarray:
    """Real-basis coefficients [N, 2l + 1] of a real function's degree-l complex coefficients c [N, 2l + 1]:
    r_0 = Re c_0, r_m = sqrt(2) Re c_{-m}, r_{-m} = sqrt(2) Im c_{-m} (m > 0), for the real harmonics
    Y^R_{l,m} = sqrt(2) (-1)^m Re Y_l^m (m > 0), Y_l^0 (m = 0), sqrt(2) (-1)^m Im Y_l^|m| (m < 0)."""
    r = np.zeros(c.shape)
    r[:, l] = c[:, l].real
    for m in range(1, l + 1):
        r[:, l + m] = math.sqrt(2.0) * c[:, l - m].real
        r[:, l - m] = math.sqrt(2.0) * c[:, l - m].imag
    return r


def cgtp_real(L: int, r1, r2, threads: int = 0) -> np.ndarray:
    """Full CGTP of real-basis rows r1, r2 [N, (L+1)^2], every path read back in the real basis; [N, (L+1)^4]
    in cgtp's layout.

    The inputs' complex-basis coefficients c = to_complex(r) are Hermitian.  With real Clebsch-Gordan
    coefficients, path (l1, l2, l3) of two Hermitian inputs is Hermitian when l1 + l2 + l3 is even and
    anti-Hermitian when it is odd (C^{l3,-m3}_{l1,-m1,l2,-m2} = (-1)^{l1+l2-l3} C^{l3 m3}_{l1 m1 l2 m2}); the
    even paths are read back as they are, the odd ones after multiplication by i, which makes them Hermitian
    (and the degree-1 path (1, 1, 1) the cross product over sqrt(2) in the real basis' (y, z, x) order).
    """
    from .istp import to_complex
    c1 = to_complex(L, r1)
    c2 = to_complex(L, r2)
    z = cgtp_complex(L, c1, c2, threads)
    out = np.empty(z.shape)
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                off = path_offset(L, l1, l2, l3)
                blk = z[:, off:off + 2 * l3 + 1]
                if (l1 + l2 + l3) % 2:
                    blk = 1j * blk
                out[:, off:off + 2 * l3 + 1] = _degree_to_real(l3, blk)
    return out


def table_build_seconds() -> float:
    return float(_load().oracle_table_build_seconds())


def max_threads() -> int:
    return int(_load().oracle_max_threads())

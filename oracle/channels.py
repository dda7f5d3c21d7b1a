"""Oracle for the channel-wise, path-weighted CGTP: TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The GPU library never imports or calls
it.

A network layer holds C copies (channels) of the (0 + 1 + ... + L) feature
and puts an equivariant linear map around the tensor product.  By Schur's
lemma such a map can only scale each path (l1, l2, l3) of the CGTP by a
scalar (the degrees-of-freedom count of Appendix E).  The plain definition,
channel by channel:

    out[n, c, path (l1, l2, l3)] = w[(n,) c, p(l1, l2, l3)] * z^(l1,l2,l3)(x1[n, c], y)

with y = x2[n, c], or x2[n] when the second input is shared by the channels
of pair n, z the CGTP (``oracle.cgtp``) and p the position of the path when
all paths are listed in (l1, l2, l3) order.
"""
from __future__ import annotations

import numpy as np

from . import cgtp as _cgtp
from . import num_outputs as _num_outputs
from . import path_offset as _path_offset


def paths(L: int):
    """Every path (l1, l2, l3) of degree L, in (l1, l2, l3) order."""
    return [(l1, l2, l3) for l1 in range(L + 1) for l2 in range(L + 1) for l3 in range(abs(l1 - l2), l1 + l2 + 1)]


def num_paths(L: int) -> int:
    return len(paths(L))


def cgtp_channels(L: int, x1, x2, w=None, threads: int = 0) -> np.ndarray:
    """x1: [N, C, (L+1)^2]; x2: [N, C, (L+1)^2] or [N, (L+1)^2] (shared by the channels);
    w: None (all ones), [C, P] or [N, C, P] with P = num_paths(L).  Returns [N, C, (L+1)^4] in fp64."""
    nin = (L + 1) ** 2
    a = np.asarray(x1, dtype=np.float64)
    if a.ndim != 3 or a.shape[2] != nin:
        raise ValueError("x1 must be [N, C, %d]" % nin)
    n, c = a.shape[:2]
    b = np.asarray(x2, dtype=np.float64)
    if b.shape == (n, nin):
        b = np.repeat(b[:, None, :], c, axis=1)
    elif b.shape != (n, c, nin):
        raise ValueError("x2 must be [N, C, %d] or [N, %d]" % (nin, nin))
    z = _cgtp(L, a.reshape(n * c, nin), b.reshape(n * c, nin), threads).reshape(n, c, _num_outputs(L))
    if w is None:
        return z
    plist = paths(L)
    wt = np.asarray(w, dtype=np.float64)
    if wt.shape == (c, len(plist)):
        wt = np.broadcast_to(wt, (n, c, len(plist)))
    elif wt.shape != (n, c, len(plist)):
        raise ValueError("w must be [C, %d] or [N, C, %d]" % (len(plist), len(plist)))
    out = np.empty_like(z)
    for k, (l1, l2, l3) in enumerate(plist):
        off = _path_offset(L, l1, l2, l3)
        out[:, :, off:off + 2 * l3 + 1] = wt[:, :, k:k + 1] * z[:, :, off:off + 2 * l3 + 1]
    return out

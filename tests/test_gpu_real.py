"""GPU parity of the real-basis full CGTP (cgtp_forward_real through the C
ABI) against the fp64 oracle's real-basis CGTP (oracle.cgtp_real).

Bar: per-path relative L2 error (over every checked pair and component of the
path) <= 1e-4 for fp32 and <= 1e-10 for fp64, as for the complex basis.  Every
pair for L <= 8 (ragged N); L = 16 and 32 on a seeded subsample, plus the
norm identity of the real CG tensor (each (l1, l2) block keeps
|x1^(l1)|^2 |x2^(l2)|^2) on every pair, which holds at any size.
"""
import ctypes

import numpy as np
import pytest

import cgtp_inputs as wl
import oracle

from test_gpu_parity import per_path_rel_err, TOL

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _lib():
    import paper_2602_21466_amd as lib
    return lib


def _run(L, N, dtype, seed, same=False, **grid):
    torch = _torch()
    x1, x2 = wl.draw(L, N, dtype, seed=seed)
    if same:
        x2 = x1
    plan = _lib().Plan(L, dtype=dtype, **grid)
    a = x1.to("cuda")
    b = a if same else x2.to("cuda")
    out = plan.forward_real(a, b)
    torch.cuda.synchronize()
    return plan, x1, x2, out


def _check(L, x1, x2, out, dtype, idx=None, what=""):
    a, b, got = x1.double().numpy(), x2.double().numpy(), out.cpu().double().numpy()
    if idx is not None:
        a, b, got = a[idx], b[idx], got[idx]
    ref = oracle.cgtp_real(L, a, b)
    err, path = per_path_rel_err(L, got, ref)
    print("%s L=%d dtype=%s checked=%d worst per-path rel L2 %.3e at %s" % (what, L, dtype, a.shape[0], err, path),
          flush=True)
    assert err <= TOL[dtype], (err, path)


@pytest.mark.parametrize("L,N,dtype", [(0, 7, "fp32"), (1, 33, "fp32"), (2, 37, "fp32"), (3, 29, "fp32"),
                                       (4, 37, "fp32"), (5, 19, "fp32"), (8, 13, "fp32"),
                                       (1, 9, "fp64"), (4, 11, "fp64"), (8, 5, "fp64")])
def test_real_all_pairs(L, N, dtype):
    _, x1, x2, out = _run(L, N, dtype, seed=600 + L)
    _check(L, x1, x2, out, dtype, what="all pairs")


def test_real_alternate_cover_and_aliased_inputs():
    _, x1, x2, out = _run(5, 17, "fp32", seed=700, cover=1)
    _check(5, x1, x2, out, "fp32", what="alternate cover")
    _, x1, x2, out = _run(4, 9, "fp32", seed=701, same=True)
    _check(4, x1, x2, out, "fp32", what="x1 == x2")


@pytest.mark.parametrize("L,N,rows", [(16, 512, 8), (32, 64, 3)])
def test_real_large_subsample_and_norm_identity(L, N, rows):
    torch = _torch()
    _, x1, x2, out = _run(L, N, "fp32", seed=800 + L)
    idx = np.sort(np.random.default_rng(L + 5).choice(N, rows, replace=False))
    _check(L, x1, x2, out, "fp32", idx=idx, what="subsample")
    # every pair: sum over l3 of |z(l1, l2, l3)|^2 = |x1^(l1)|^2 |x2^(l2)|^2
    z = out.double()
    a, b = x1.double().to("cuda"), x2.double().to("cuda")
    worst = 0.0
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            lo = _lib().cgtp_path_offset(L, l1, l2, abs(l1 - l2))
            hi = lo + (2 * l1 + 1) * (2 * l2 + 1)
            got = (z[:, lo:hi] ** 2).sum(1)
            want = (a[:, wl.block_slice(l1)] ** 2).sum(1) * (b[:, wl.block_slice(l2)] ** 2).sum(1)
            worst = max(worst, float(((got - want).abs() / want).max()))
    print("L=%d norm identity over %d pairs, every block: max rel err %.3e" % (L, N, worst), flush=True)
    assert worst <= 1e-4


def test_real_argument_errors_and_no_workspace():
    """The fused kernel needs no workspace (0 bytes); bad pointers, misalignment, negative sizes and outputs that
    overlap an input are rejected before anything is launched."""
    torch = _torch()
    lib = _lib()
    L, N = 3, 8
    plan = lib.Plan(L)
    f = lib._load()
    assert lib.cgtp_real_workspace_bytes(plan._h, N) == 0
    assert lib.cgtp_real_workspace_bytes(plan._h, -1) == -1
    x = torch.randn(N, 16, device="cuda")
    big = torch.randn(N * 256 + 64, device="cuda")
    out = torch.full((N, 256), 7.0, device="cuda")
    P = lambda t, off=0: ctypes.c_void_p(t.data_ptr() + off)
    for args in [(None, P(x), P(out), N, None, 0),          # missing input
                 (P(x), P(x), None, N, None, 0),            # missing output
                 (P(x), P(x), P(out, 4), N, None, 0),       # misaligned output
                 (P(x), P(x), P(out), -1, None, 0),         # negative N
                 (P(x), P(x), P(out), N, None, -1),         # negative workspace size
                 (P(big), P(x), P(big, 64), N, None, 0)]:   # output overlapping an input
        assert f.cgtp_forward_real(plan._h, *args, None) == lib.CGTP_EINVAL, args
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # a call without workspace works (and N = 0 is a no-op)
    assert f.cgtp_forward_real(plan._h, P(x), P(x), P(out), 0, None, 0, None) == lib.CGTP_OK
    assert f.cgtp_forward_real(plan._h, P(x), P(x), P(out), N, None, 0, None) == lib.CGTP_OK
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all()) and not bool((out == 7.0).all())

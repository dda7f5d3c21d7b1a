"""GPU parity of the CGTP gradients (cgtp_backward through the C ABI) against
the fp64 CPU oracle's gradients (oracle.cgtp_backward, the transposed double
sum).

Bar: per-degree relative L2 error of each gradient (over every checked pair
and the 2l + 1 components of degree l) <= 1e-4 for fp32 and <= 1e-10 for
fp64.  Degrees L <= 8 (and L = 12, 16 in fp64) are compared on every pair (N
ragged: not a multiple of any tile); L = 16 and 32 in fp32 on a seeded
subsample of pairs, plus the adjoint
identity <grad_x1, d> = <grad_out, forward(d, x2)> on every pair, which holds
at any size.
"""
import ctypes

import numpy as np
import pytest

import cgtp_inputs as wl
import oracle

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "fp64": 1e-10}


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _lib():
    import paper_2602_21466_amd as lib
    return lib


def per_degree_rel_err(L, got, ref):
    worst, at = 0.0, -1
    for l in range(L + 1):
        sl = wl.block_slice(l)
        den = float((ref[:, sl] ** 2).sum())
        num = float(((got[:, sl] - ref[:, sl]) ** 2).sum())
        rel = np.sqrt(num / den) if den > 0 else np.sqrt(num)
        if rel > worst:
            worst, at = rel, l
    return worst, at


def _grads(L, N, dtype, seed, **grid):
    """Seeded x1, x2, grad_out; the GPU gradients; the plan and device tensors."""
    torch = _torch()
    x1, x2 = wl.draw(L, N, dtype, seed=seed)
    g = wl.draw_rows((L + 1) ** 4, N, dtype, seed=seed + 7919)[0]
    plan = _lib().Plan(L, dtype=dtype, **grid)
    a, b, gg = x1.to("cuda"), x2.to("cuda"), g.to("cuda")
    g1, g2 = plan.backward(a, b, gg)
    torch.cuda.synchronize()
    return plan, (x1, x2, g), (a, b, gg), (g1.cpu().double().numpy(), g2.cpu().double().numpy())


def _check(L, host, got, dtype, idx=None, what=""):
    x1, x2, g = (t.double().numpy() for t in host)
    if idx is not None:
        x1, x2, g = x1[idx], x2[idx], g[idx]
        got = tuple(a[idx] for a in got)
    r1, r2 = oracle.cgtp_backward(L, x1, x2, g)
    e1, l1 = per_degree_rel_err(L, got[0], r1)
    e2, l2 = per_degree_rel_err(L, got[1], r2)
    print("%s L=%d dtype=%s checked=%d worst per-degree rel L2: gx1 %.3e (l=%d) gx2 %.3e (l=%d)"
          % (what, L, dtype, x1.shape[0], e1, l1, e2, l2), flush=True)
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype], (e1, l1, e2, l2)


@pytest.mark.parametrize("L,N,dtype", [(0, 5, "fp32"), (1, 37, "fp32"), (2, 37, "fp32"), (3, 29, "fp32"),
                                       (4, 37, "fp32"), (5, 21, "fp32"), (8, 19, "fp32"),
                                       (1, 9, "fp64"), (3, 17, "fp64"), (4, 13, "fp64"), (8, 7, "fp64"),
                                       # grids of more rings than one group holds, in both variants
                                       (12, 7, "fp64"), (16, 5, "fp64")])
def test_backward_all_pairs(L, N, dtype):
    _, host, _, got = _grads(L, N, dtype, seed=100 + L)
    _check(L, host, got, dtype, what="all pairs")


@pytest.mark.parametrize("L,dtype", [(3, "fp32"), (5, "fp32"), (6, "fp64")])
def test_backward_alternate_cover(L, dtype):
    _, host, _, got = _grads(L, 11, dtype, seed=200 + L, cover=1)
    _check(L, host, got, dtype, what="alternate cover")


def test_backward_global_grid():
    L = 4
    _, host, _, got = _grads(L, 9, "fp32", seed=300, n_theta=2 * L + 4, n_phi=27)
    _check(L, host, got, "fp32", what="global grid")


@pytest.mark.parametrize("L,N,rows", [(16, 512, 12), (32, 48, 6)])
def test_backward_large_subsample(L, N, rows):
    torch = _torch()
    plan, host, dev, got = _grads(L, N, "fp32", seed=400 + L)
    idx = np.sort(np.random.default_rng(L).choice(N, rows, replace=False))
    _check(L, host, got, "fp32", idx=idx, what="subsample")
    # adjoint identity on every pair: <gx1, d> = <g, z(d, x2)>, <gx2, d> = <g, z(x1, d)>
    a, b, gg = dev
    d = torch.from_numpy(np.random.default_rng(L + 1).standard_normal(a.shape)).to(a.dtype).to("cuda")
    g = gg.double()
    lhs1 = (torch.from_numpy(got[0]).to("cuda") * d.double()).sum(1)
    rhs1 = (g * plan.forward(d, b).double()).sum(1)
    lhs2 = (torch.from_numpy(got[1]).to("cuda") * d.double()).sum(1)
    rhs2 = (g * plan.forward(a, d).double()).sum(1)
    torch.cuda.synchronize()
    for lhs, rhs in ((lhs1, rhs1), (lhs2, rhs2)):
        scale = float(rhs.abs().max())
        err = float((lhs - rhs).abs().max()) / scale
        print("L=%d adjoint identity over %d pairs: max |lhs - rhs| / max |rhs| = %.3e" % (L, N, err), flush=True)
        assert err <= 1e-4


def test_backward_one_gradient_and_determinism():
    torch = _torch()
    L, N = 5, 23
    plan, host, (a, b, gg), (f1, f2) = _grads(L, N, "fp32", seed=500)
    g1, none2 = plan.backward(a, b, gg, need_x2=False)
    none1, g2 = plan.backward(a, b, gg, need_x1=False)
    torch.cuda.synchronize()
    assert none1 is None and none2 is None
    assert np.array_equal(g1.cpu().double().numpy(), f1)
    assert np.array_equal(g2.cpu().double().numpy(), f2)


def test_backward_zero_pairs():
    torch = _torch()
    lib = _lib()
    plan = lib.Plan(3)
    e = torch.empty((0, 16), device="cuda")
    g1, g2 = plan.backward(e, e, torch.empty((0, 256), device="cuda"))
    assert g1.shape == (0, 16) and g2.shape == (0, 16)


def test_backward_rejects_bad_arguments():
    torch = _torch()
    lib = _lib()
    L, N = 3, 8
    plan = lib.Plan(L)
    f = lib._load()
    x = torch.randn(N, 16, device="cuda")
    g = torch.randn(N, 256, device="cuda")
    gx = torch.full((N, 16), 7.0, device="cuda")
    need = lib.cgtp_backward_workspace_bytes(plan._h, N)
    assert need == 2 * (L + 1) ** 3 * N * 4
    ws = torch.empty(need + 512, dtype=torch.uint8, device="cuda")
    P = lambda t, off=0: ctypes.c_void_p(t.data_ptr() + off)
    h = plan._h
    cases = [
        (P(x), P(x), P(g), None, None, N, P(ws), need),            # no gradient asked for
        (P(x), P(x), P(g), P(gx), None, N, P(ws), need - 1),       # workspace too short
        (P(x), P(x), P(g), P(gx), None, N, P(ws, 16), need),       # workspace not 256-byte aligned
        (P(x), P(x), P(g), P(gx), None, N, None, need),            # no workspace
        (P(x), P(x), P(g), P(x), None, N, P(ws), need),            # gradient overlaps an input
        (P(x), P(x), P(g), P(gx), P(gx), N, P(ws), need),          # the two gradients overlap
        (P(x), P(x), P(g), P(gx, 4), None, N, P(ws), need),        # gradient misaligned
        (P(x), None, P(g), P(gx), None, N, P(ws), need),           # NULL input
        (P(x), P(x), P(g), P(gx), None, -1, P(ws), need),          # negative N
    ]
    for args in cases:
        assert f.cgtp_backward(h, *args, None) == lib.CGTP_EINVAL, args
    torch.cuda.synchronize()
    assert bool((gx == 7.0).all())

"""The no-allocation entry point istp_forward_real_static against istp_forward_real
(same kernels, caller-allocated workspace), through the C ABI, on two calls in a
row (the second with fewer pairs, reusing the static scratch the first one left
behind), and its size limit.  Spin 2 uses the scratch (three products); spins
0 and 1 run the real-basis kernel, which needs none."""
import ctypes

import numpy as np
import pytest

import cgtp_inputs
import oracle.istp as oi

pytestmark = pytest.mark.gpu


def _setup():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_21466_amd as lib
    return torch, lib


def _rel(a, b):
    a = a.double().cpu().numpy()
    b = b.double().cpu().numpy()
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.mark.parametrize("L,N1,N2,dtype", [(16, 2000, 500, "fp32"), (5, 300, 37, "fp32"), (4, 50, 9, "fp64")])
def test_static_scratch_matches_workspace_entry_point(L, N1, N2, dtype):
    torch, lib = _setup()
    plan = lib.IstpPlan(L, lib.ISTP_GAUNT, dtype)
    tdt = torch.float32 if dtype == "fp32" else torch.float64
    s = torch.cuda.current_stream().cuda_stream
    for n, seed in ((N1, 11), (N2, 12)):
        x1, x2 = cgtp_inputs.draw_rows(oi.gaunt_size(L), n, dtype, seed=seed + L)
        a, b = x1.cuda(), x2.cuda()
        ref = plan.forward_real(a, b)
        out = torch.full((n, plan.nout), float("nan"), dtype=tdt, device="cuda")
        lib.istp_forward_real_static(plan._h, a.data_ptr(), b.data_ptr(), out.data_ptr(), n, s)
        torch.cuda.synchronize()
        err = _rel(out, ref)
        print("L=%d N=%d %s: static vs workspace entry point rel L2 %.3e, identical %s"
              % (L, n, dtype, err, torch.equal(out, ref)), flush=True)
        assert torch.isfinite(out).all().item()
        assert err <= (1e-6 if dtype == "fp32" else 1e-13)
        # and the oracle on a few rows, at the parity bar of the real-basis product
        k = min(n, 3)
        want = oi.gaunt_tp_real(L, x1[:k].double().numpy(), x2[:k].double().numpy())
        got = out[:k].double().cpu().numpy()
        assert np.linalg.norm(got - want) / np.linalg.norm(want) <= (1e-4 if dtype == "fp32" else 1e-10)


def test_static_scratch_size_limit():
    """Spin 2 (three products through the scratch): the largest N whose workspace fits the static array runs,
    one more is refused with CGTP_ESCRATCH and nothing is written.  Spin 0 runs the real-basis kernel, which
    needs no workspace: the static entry point takes any N."""
    torch, lib = _setup()
    L = 8
    plan = lib.IstpPlan(L, lib.ISTP_TENSOR, "fp32")
    cap = 64 << 20
    lo, hi = 1, 1 << 20
    while lo < hi:   # the largest n with workspace <= cap
        mid = (lo + hi + 1) // 2
        if lib.istp_real_workspace_bytes(plan._h, mid) <= cap:
            lo = mid
        else:
            hi = mid - 1
    limit = lo
    assert lib.istp_real_workspace_bytes(plan._h, limit + 1) > cap
    f = lib._load()
    x = torch.zeros(limit + 1, plan.nin, device="cuda")
    out = torch.full((limit + 1, plan.nout), 5.0, device="cuda")
    rc = f.istp_forward_real_static(plan._h, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(x.data_ptr()),
                                    ctypes.c_void_p(out.data_ptr()), limit + 1, None)
    assert rc == lib.CGTP_ESCRATCH
    assert lib.cgtp_strerror(rc)
    torch.cuda.synchronize()
    assert (out == 5.0).all().item()
    rc = f.istp_forward_real_static(plan._h, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(x.data_ptr()),
                                    ctypes.c_void_p(out.data_ptr()), limit, None)
    assert rc == lib.CGTP_OK
    torch.cuda.synchronize()
    assert (out[:limit] == 0.0).all().item() and (out[limit] == 5.0).all().item()
    # spin 0: no workspace, so no limit
    p0 = lib.IstpPlan(16, lib.ISTP_GAUNT, "fp32")
    assert lib.istp_real_workspace_bytes(p0._h, 100000) == 0
    n = 6000
    x0 = torch.zeros(n, p0.nin, device="cuda")
    o0 = torch.full((n, p0.nout), 5.0, device="cuda")
    assert f.istp_forward_real_static(p0._h, ctypes.c_void_p(x0.data_ptr()), ctypes.c_void_p(x0.data_ptr()),
                                      ctypes.c_void_p(o0.data_ptr()), n, None) == lib.CGTP_OK
    torch.cuda.synchronize()
    assert (o0 == 0.0).all().item()


@pytest.mark.parametrize("spin,L,N1,N2", [(1, 6, 400, 41), (2, 3, 120, 7)])
def test_static_scratch_spin_products(spin, L, N1, N2):
    """The spin-1 and spin-2 real-basis products through the static scratch, two calls in a row."""
    torch, lib = _setup()
    plan = lib.IstpPlan(L, spin, "fp32")
    s = torch.cuda.current_stream().cuda_stream
    for n, seed in ((N1, 21), (N2, 22)):
        x1, x2 = cgtp_inputs.draw_rows(oi.spin_size(spin, L), n, "fp32", seed=seed + L)
        a, b = x1.cuda(), x2.cuda()
        ref = plan.forward_real(a, b)
        out = torch.full((n, plan.nout), float("nan"), device="cuda")
        rc = lib._load().istp_forward_real_static(plan._h, ctypes.c_void_p(a.data_ptr()), ctypes.c_void_p(b.data_ptr()),
                                                 ctypes.c_void_p(out.data_ptr()), n, ctypes.c_void_p(s))
        assert rc == lib.CGTP_OK
        torch.cuda.synchronize()
        err = _rel(out, ref)
        print("spin %d L=%d N=%d: static vs workspace entry point rel L2 %.3e" % (spin, L, n, err), flush=True)
        assert torch.isfinite(out).all().item() and err <= 1e-6
        want = oi.spin_tp_real(spin, L, x1[:2].double().numpy(), x2[:2].double().numpy())
        got = out[:2].double().cpu().numpy()
        assert np.linalg.norm(got - want) / np.linalg.norm(want) <= 1e-4

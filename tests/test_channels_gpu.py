"""GPU parity of the channel-wise, path-weighted CGTP (cgtp_forward_weighted)
against the fp64 oracle, through the C ABI.

Bar: per-path relative L2 error over the checked (pair, channel) rows <= 1e-4
(fp32) or 1e-10 (fp64), as for the plain CGTP."""
import numpy as np
import pytest

import cgtp_inputs as wl
import oracle.channels as oc
from test_gpu_parity import TOL, _lib, _torch, path_ids, per_path_rel_err

pytestmark = pytest.mark.gpu

# (L, pairs N, channels C, x2 shared, weights, dtype): ragged row counts against the
# pairs per work-group, channel counts that do not divide them, both weight layouts
CASES = [
    (4, 13, 3, True, "channel", "fp32"),
    (4, 13, 3, False, "pair", "fp32"),
    (5, 9, 5, True, "none", "fp32"),
    (3, 7, 4, True, "pair", "fp32"),
    (8, 10, 7, True, "channel", "fp32"),
    (2, 11, 3, True, "channel", "fp64"),
    (3, 5, 6, False, "channel", "fp64"),
    (1, 3, 1, False, "channel", "fp32"),
]


def _run(L, N, C, shared, weights, dtype, seed):
    torch = _torch()
    x1, x2, w = wl.channel_inputs(L, N, C, shared, weights, dtype, seed)
    plan = _lib().Plan(L, dtype=dtype)
    out = plan.forward_weighted(x1.cuda(), x2.cuda(), None if w is None else w.cuda())
    torch.cuda.synchronize()
    return plan, x1, x2, w, out.cpu()


@pytest.mark.parametrize("L,N,C,shared,weights,dtype", CASES)
def test_weighted_channels_match_oracle(L, N, C, shared, weights, dtype):
    print("case L=%d N=%d C=%d shared=%s weights=%s %s" % (L, N, C, shared, weights, dtype), flush=True)
    plan, x1, x2, w, got = _run(L, N, C, shared, weights, dtype, seed=L + 200)
    ref = oc.cgtp_channels(L, x1.double().numpy(), x2.double().numpy(), None if w is None else w.double().numpy())
    nout = (L + 1) ** 4
    err, path = per_path_rel_err(L, got.double().numpy().reshape(N * C, nout), ref.reshape(N * C, nout))
    print("  worst per-path rel L2 %.3e at %s" % (err, path), flush=True)
    assert err <= TOL[dtype], (err, path)
    plan.close()


def test_unweighted_single_channel_is_the_plain_forward():
    """C = 1, no weights, x2 not shared: bit-identical to cgtp_forward (the same kernel path)."""
    torch = _torch()
    L, N = 6, 21
    x1, x2 = wl.draw_rows((L + 1) ** 2, N, "fp32", seed=3)
    plan = _lib().Plan(L)
    a, b = x1.cuda(), x2.cuda()
    plain = plan.forward(a, b)
    ch = plan.forward_weighted(a[:, None].contiguous(), b[:, None].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(plain, ch[:, 0])
    plan.close()


def test_weights_scale_paths_of_the_unweighted_result():
    """Weighted output = weight x unweighted output, path by path (one rounding apart)."""
    torch = _torch()
    L, N, C = 7, 6, 5
    x1, x2, w = wl.channel_inputs(L, N, C, True, "pair", "fp32", seed=11)
    plan = _lib().Plan(L)
    a, b, wc = x1.cuda(), x2.cuda(), w.cuda()
    zw = plan.forward_weighted(a, b, wc)
    z = plan.forward_weighted(a, b)
    torch.cuda.synchronize()
    pid, _ = path_ids(L)
    scale = wc[:, :, torch.as_tensor(pid, device="cuda")]
    torch.testing.assert_close(zw, z * scale, rtol=2e-6, atol=1e-6 * float(z.abs().max()))
    plan.close()


def test_channel_workload_sampled():
    """The benchmark's channel workload in its launch configuration, checked on a seeded subsample of rows."""
    torch = _torch()
    wk = wl.CHANNEL_WORKLOADS[0]
    print("workload %s" % wk.name, flush=True)
    plan, x1, x2, w, got = _run(wk.L, wk.N, wk.C, wk.x2_shared, wk.weights, wk.dtype, wk.seed)
    rows = wl.channel_check_rows(wk)
    n_idx = [r // wk.C for r in rows]
    c_idx = [r % wk.C for r in rows]
    nin, nout = (wk.L + 1) ** 2, (wk.L + 1) ** 4
    x1r = x1.double().numpy()[n_idx, c_idx][:, None]
    x2r = (x2.double().numpy()[n_idx] if wk.x2_shared else x2.double().numpy()[n_idx, c_idx])
    wr = w.double().numpy()[c_idx][:, None] if wk.weights == "channel" else w.double().numpy()[n_idx, c_idx][:, None]
    ref = oc.cgtp_channels(wk.L, x1r, x2r if wk.x2_shared else x2r[:, None], wr).reshape(len(rows), nout)
    sub = got.reshape(wk.N * wk.C, nout)[rows].double().numpy()
    err, path = per_path_rel_err(wk.L, sub, ref)
    print("  rows checked %d, worst per-path rel L2 %.3e at %s" % (len(rows), err, path), flush=True)
    assert err <= TOL[wk.dtype], (err, path)
    assert torch.isfinite(got).all()
    plan.close()


def test_rejects_bad_channel_arguments():
    torch = _torch()
    lib = _lib()
    L, N, C = 3, 4, 2
    plan = lib.Plan(L)
    nin, nout, P = (L + 1) ** 2, (L + 1) ** 4, lib.cgtp_num_paths(L)
    x1 = torch.zeros(N, C, nin, device="cuda")
    x2 = torch.zeros(N, nin, device="cuda")
    out = torch.zeros(N, C, nout, device="cuda")
    w = torch.zeros(C, P, device="cuda")
    h = plan._h
    call = lambda **k: lib.cgtp_forward_weighted(h, x1.data_ptr(), x2.data_ptr(), k.get("w", w.data_ptr()),
                                                 k.get("out", out.data_ptr()), k.get("N", N), k.get("C", C),
                                                 True, False, None)
    for bad in ({"C": 0}, {"C": -3}, {"N": -1}, {"out": x1.data_ptr()}, {"w": out.data_ptr() + 4}):
        with pytest.raises(lib.CgtpError) as e:
            call(**bad)
        assert e.value.args[0].endswith("(-1)"), bad
    rc = lib._load().cgtp_forward_weighted(h, x1.data_ptr(), x2.data_ptr(), None, out.data_ptr(), N,
                                           lib.ctypes.byref(lib.cgtp_channels(C, 1, 0, 5)), None)
    assert rc == lib.CGTP_EINVAL
    rc = lib._load().cgtp_forward_weighted(h, x1.data_ptr(), x2.data_ptr(), None, out.data_ptr(), N,
                                           lib.ctypes.byref(lib.cgtp_channels(C, 2, 0, 0)), None)
    assert rc == lib.CGTP_EINVAL
    call(N=0)   # nothing to do
    torch.cuda.synchronize()
    plan.close()


@pytest.mark.parametrize("grid", [{"cover": 1}, {"n_theta": 12, "n_phi": 24}], ids=["alternate-cover", "global-grid"])
def test_weighted_channels_other_plans(grid):
    """The channel kernel on plans with the alternate product cover and with one forced global grid."""
    torch = _torch()
    L, N, C = 5, 6, 3
    x1, x2, w = wl.channel_inputs(L, N, C, True, "pair", "fp32", seed=31)
    plan = _lib().Plan(L, **grid)
    got = plan.forward_weighted(x1.cuda(), x2.cuda(), w.cuda())
    torch.cuda.synchronize()
    ref = oc.cgtp_channels(L, x1.double().numpy(), x2.double().numpy(), w.double().numpy())
    nout = (L + 1) ** 4
    err, path = per_path_rel_err(L, got.cpu().double().numpy().reshape(N * C, nout), ref.reshape(N * C, nout))
    print("%s worst per-path rel L2 %.3e at %s" % (grid, err, path), flush=True)
    assert err <= TOL["fp32"], (err, path)
    plan.close()

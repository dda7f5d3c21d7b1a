"""GPU parity of the channel-wise, label-weighted signal products
(istp_forward_weighted) against the fp64 oracle, through the C ABI.

Bar as for the signal products: per-output-label relative L2 error over the
checked (pair, channel) rows <= 1e-4 (fp32) or 1e-10 (fp64)."""
import numpy as np
import pytest

import cgtp_inputs as wl
import oracle.istp as oi
from test_istp_gpu import TOL, _lib, _torch, per_label_rel_err

pytestmark = pytest.mark.gpu

# (spin, L, pairs N, channels C, x2 shared, weights, dtype); row counts ragged against the
# pairs per work-group, channel counts that do not divide them, both weight layouts
CASES = [
    (0, 4, 11, 3, True, "channel", "fp32"),
    (1, 4, 11, 3, True, "channel", "fp32"),
    (1, 5, 7, 5, False, "pair", "fp32"),
    (0, 6, 9, 2, False, "none", "fp32"),
    (1, 3, 6, 4, True, "pair", "fp32"),
    (1, 8, 5, 7, True, "channel", "fp32"),
    (0, 3, 5, 3, True, "channel", "fp64"),
    (1, 2, 4, 6, False, "pair", "fp64"),
    (2, 3, 5, 3, True, "channel", "fp32"),
    (2, 2, 3, 2, False, "pair", "fp64"),
]


def _run(spin, L, N, C, shared, weights, dtype, seed, drop=()):
    torch = _torch()
    x1, x2, w1, w2, wo = wl.istp_channel_inputs(spin, L, N, C, shared, weights, dtype, seed)
    ws = [None if (w is None or k in drop) else w for k, w in enumerate((w1, w2, wo))]
    plan = _lib().IstpPlan(L, spin, dtype)
    cu = lambda t: None if t is None else t.cuda()
    out = plan.forward_weighted(x1.cuda(), x2.cuda(), *[cu(w) for w in ws])
    torch.cuda.synchronize()
    return plan, x1, x2, ws, out.cpu()


def _ref(spin, L, x1, x2, ws):
    d = lambda t: None if t is None else t.double().numpy()
    return oi.channel_product(spin, L, d(x1), d(x2), *[d(w) for w in ws])


@pytest.mark.parametrize("spin,L,N,C,shared,weights,dtype", CASES)
def test_weighted_channels_match_oracle(spin, L, N, C, shared, weights, dtype):
    print("case spin=%d L=%d N=%d C=%d shared=%s weights=%s %s" % (spin, L, N, C, shared, weights, dtype),
          flush=True)
    plan, x1, x2, ws, got = _run(spin, L, N, C, shared, weights, dtype, seed=L + 300 + spin)
    ref = _ref(spin, L, x1, x2, ws)
    err, lab = per_label_rel_err(2 * L, spin, got.double().numpy().reshape(N * C, -1), ref.reshape(N * C, -1))
    print("  worst per-label rel L2 %.3e at %s" % (err, lab), flush=True)
    assert err <= TOL[dtype], (err, lab)
    plan.close()


def test_partial_weights():
    """Any of w1, w2, wo may be absent (all ones)."""
    spin, L, N, C = 1, 4, 6, 3
    for drop in ((0,), (1, 2), (0, 2)):
        plan, x1, x2, ws, got = _run(spin, L, N, C, True, "channel", "fp32", seed=5, drop=drop)
        ref = _ref(spin, L, x1, x2, ws)
        err, lab = per_label_rel_err(2 * L, spin, got.double().numpy().reshape(N * C, -1), ref.reshape(N * C, -1))
        print("drop %s: worst per-label rel L2 %.3e at %s" % (drop, err, lab), flush=True)
        assert err <= TOL["fp32"], (drop, err, lab)
        plan.close()


def test_unweighted_channels_equal_the_plain_forward():
    """x2 not shared, no weights: the rows are independent products, as istp_forward computes them."""
    torch = _torch()
    spin, L, N, C = 1, 6, 5, 4
    x1, x2, *_ = wl.istp_channel_inputs(spin, L, N, C, False, "none", "fp32", seed=9)
    plan = _lib().IstpPlan(L, spin)
    a, b = x1.cuda(), x2.cuda()
    ch = plan.forward_weighted(a, b)
    plain = plan.forward(a.view(N * C, -1), b.view(N * C, -1))
    torch.cuda.synchronize()
    assert torch.equal(ch.view(N * C, -1), plain)
    plan.close()


def test_channel_workload_sampled():
    """The benchmark's channel workload in its launch configuration, checked on sampled rows."""
    torch = _torch()
    wk = wl.ISTP_CHANNEL_WORKLOADS[0]
    print("workload %s" % wk.name, flush=True)
    plan, x1, x2, ws, got = _run(wk.spin, wk.L, wk.N, wk.C, wk.x2_shared, wk.weights, wk.dtype, wk.seed)
    rows = wl.istp_channel_check_rows(wk)
    n_idx = [r // wk.C for r in rows]
    c_idx = [r % wk.C for r in rows]
    d = lambda t: t.double().numpy()
    x1r = d(x1)[n_idx, c_idx][:, None]
    x2r = d(x2)[n_idx] if wk.x2_shared else d(x2)[n_idx, c_idx]
    wr = [None if w is None else (d(w)[c_idx] if wk.weights == "channel" else d(w)[n_idx, c_idx])[:, None]
          for w in ws]
    ref = oi.channel_product(wk.spin, wk.L, x1r, x2r if wk.x2_shared else x2r[:, None], *wr)
    sub = got.reshape(wk.N * wk.C, -1)[rows].double().numpy()
    err, lab = per_label_rel_err(2 * wk.L, wk.spin, sub, ref.reshape(len(rows), -1))
    print("  rows checked %d, worst per-label rel L2 %.3e at %s" % (len(rows), err, lab), flush=True)
    assert err <= TOL[wk.dtype], (err, lab)
    assert torch.isfinite(got).all()
    plan.close()


def test_rejects_bad_channel_arguments():
    torch = _torch()
    lib = _lib()
    L, spin, N, C = 3, 1, 4, 2
    plan = lib.IstpPlan(L, spin)
    x1 = torch.zeros(N, C, plan.nin, device="cuda")
    x2 = torch.zeros(N, plan.nin, device="cuda")
    out = torch.zeros(N, C, plan.nout, device="cuda")
    h = plan._h
    call = lambda **k: lib.istp_forward_weighted(h, x1.data_ptr(), x2.data_ptr(), None, None,
                                                 k.get("wo", None), k.get("out", out.data_ptr()), k.get("N", N),
                                                 k.get("C", C), True, False, None)
    for bad in ({"C": 0}, {"N": -1}, {"out": x1.data_ptr()}, {"wo": out.data_ptr() + 4}):
        with pytest.raises(lib.CgtpError) as e:
            call(**bad)
        assert e.value.args[0].endswith("(-1)"), bad
    call(N=0)
    torch.cuda.synchronize()
    plan.close()


@pytest.mark.parametrize("spin,L,N,C,weights,dtype", [(0, 3, 5, 3, "channel", "fp32"), (1, 4, 4, 2, "pair", "fp32"),
                                                      (1, 2, 3, 3, "channel", "fp64"), (2, 2, 3, 2, "channel", "fp32")])
def test_weighted_channel_gradients(spin, L, N, C, weights, dtype):
    """istp_backward_weighted against the oracle's chain rule through the label weights (x2 per channel)."""
    torch = _torch()
    x1, x2, w1, w2, wo = wl.istp_channel_inputs(spin, L, N, C, False, weights, dtype, seed=40 + L + spin)
    g = torch.randn(N, C, (2 * spin + 1) * (2 * L + 1) ** 2, generator=torch.Generator().manual_seed(50 + L),
                    dtype=torch.float64).to(x1.dtype)
    plan = _lib().IstpPlan(L, spin, dtype)
    cu = lambda t: None if t is None else t.cuda()
    g1, g2 = plan.backward_weighted(x1.cuda(), x2.cuda(), g.cuda(), cu(w1), cu(w2), cu(wo))
    torch.cuda.synchronize()
    d = lambda t: None if t is None else t.double().numpy()
    r1, r2 = oi.channel_product_vjp(spin, L, d(x1), d(x2), d(g), d(w1), d(w2), d(wo))
    e1, l1 = per_label_rel_err(L, spin, g1.cpu().double().numpy().reshape(N * C, -1), r1.reshape(N * C, -1))
    e2, l2 = per_label_rel_err(L, spin, g2.cpu().double().numpy().reshape(N * C, -1), r2.reshape(N * C, -1))
    print("weighted gradients spin=%d L=%d %s: %s %.3e, %s %.3e" % (spin, L, dtype, l1, e1, l2, e2), flush=True)
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype], (l1, e1, l2, e2)
    plan.close()

"""GPU parity of the MIMO Gaunt (spin 0) and vector (spin 1) signal products
against the fp64 CPU oracle, through the C ABI of include/istp.h.

Bar: per-output-label relative L2 error (over every checked pair and
component of the label) <= 1e-4 for fp32 and <= 1e-10 for fp64.  A label
whose reference is exactly zero (a selection rule) is held to the scale of a
typical label.  The full-size workloads run in the benchmark's launch
configuration and are compared on a seeded subsample of pairs.
"""

import numpy as np
import pytest

import cgtp_inputs as wl
import oracle.istp as oi

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


def _labels(L, spin):
    """Label id of every column of a row with degrees <= L, and the (j, l) list."""
    if spin == 0:
        labels = [(l, l) for l in range(L + 1)]
        sizes = [2 * l + 1 for l in range(L + 1)]
    else:
        labels = oi.vector_labels(L) if spin == 1 else oi.spin_labels(spin, L)
        sizes = [2 * j + 1 for j, l in labels]
    return np.repeat(np.arange(len(labels)), sizes), labels


def per_label_rel_err(L_out, spin, got, ref):
    lid, labels = _labels(L_out, spin)
    num = np.bincount(lid, weights=((got - ref) ** 2).sum(0), minlength=len(labels))
    den = np.bincount(lid, weights=(ref ** 2).sum(0), minlength=len(labels))
    typical = np.median(den[den > 0]) if (den > 0).any() else 1.0
    rel = np.sqrt(num / np.where(den > 1e-20 * typical, den, typical))
    worst = int(np.argmax(rel))
    return float(rel[worst]), labels[worst]


def reference(L, spin, x1, x2):
    a, b = np.asarray(x1, dtype=np.float64), np.asarray(x2, dtype=np.float64)
    if spin == 2:
        return oi.spin_tp(2, L, a, b)
    return (oi.gaunt_tp if spin == 0 else oi.vector_tp)(L, a, b)


def run_gpu(L, spin, x1, x2, dtype):
    torch = _torch()
    plan = _lib().IstpPlan(L, spin, dtype)
    a, b = x1.to("cuda"), x2.to("cuda")
    out = plan.forward(a, b)
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


CASES = [(0, 0, 5, "fp32"), (0, 1, 5, "fp64"), (1, 0, 17, "fp64"), (1, 1, 9, "fp32"), (2, 1, 64, "fp64"),
         (2, 0, 64, "fp32"), (3, 1, 33, "fp32"), (4, 0, 100, "fp32"), (5, 1, 19, "fp64"), (6, 1, 21, "fp32"),
         (8, 0, 37, "fp64"), (8, 1, 40, "fp32"), (12, 1, 7, "fp64"), (12, 0, 9, "fp32"),
         # spin 2 (rank-2 tensor harmonics): one pair per work-group
         (0, 2, 5, "fp32"), (1, 2, 7, "fp32"), (2, 2, 9, "fp64"), (3, 2, 11, "fp32"), (5, 2, 6, "fp32"),
         (6, 2, 4, "fp64"), (8, 2, 3, "fp32")]


@pytest.mark.parametrize("L,spin,N,dtype", CASES)
def test_parity_small(L, spin, N, dtype):
    """Every pair, ragged N (not a multiple of the pairs per work-group)."""
    x1, x2 = wl.draw_rows((2 * spin + 1) * (L + 1) ** 2, N, dtype, seed=1000 + 10 * L + spin)
    got = run_gpu(L, spin, x1, x2, dtype)
    ref = reference(L, spin, x1, x2)
    err, lab = per_label_rel_err(2 * L, spin, got, ref)
    print("L=%d spin=%d N=%d %s worst label %s rel err %.3e" % (L, spin, N, dtype, lab, err))
    assert err <= TOL[dtype], (lab, err)


@pytest.mark.parametrize("w", wl.ISTP_WORKLOADS, ids=lambda w: w.name)
def test_parity_workloads(w):
    """Full-size workloads in the benchmark's launch configuration, on a seeded subsample of pairs."""
    x1, x2 = wl.istp_inputs(w)
    got = run_gpu(w.L, w.spin, x1, x2, w.dtype)
    idx = wl.istp_check_indices(w).numpy()
    ref = reference(w.L, w.spin, x1[idx], x2[idx])
    err, lab = per_label_rel_err(2 * w.L, w.spin, got[idx], ref)
    print("%s worst label %s rel err %.3e" % (w.name, lab, err))
    assert err <= TOL[w.dtype], (lab, err)
    assert np.isfinite(got).all()


def test_same_input_twice_and_symmetry():
    """x1 == x2 (one buffer) is allowed; the Gaunt product is symmetric, the vector one antisymmetric."""
    torch = _torch()
    L = 6
    for spin, sign in ((0, 1.0), (1, -1.0), (2, 1.0)):
        x1, x2 = wl.draw_rows((2 * spin + 1) * (L + 1) ** 2, 11, "fp64", seed=77 + spin)
        plan = _lib().IstpPlan(L, spin, "fp64")
        a, b = x1.cuda(), x2.cuda()
        ab, ba, aa = plan.forward(a, b), plan.forward(b, a), plan.forward(a, a)
        torch.cuda.synchronize()
        scale = np.abs(ab.cpu().numpy()).max()
        np.testing.assert_allclose(ba.cpu().numpy(), sign * ab.cpu().numpy(), atol=1e-12 * scale)
        # x1 (x) x1: the Gaunt product against the oracle, the vector product vanishes
        np.testing.assert_allclose(aa.cpu().numpy(), reference(L, spin, x1, x1), atol=1e-12 * scale)
        if spin == 1:
            assert np.abs(aa.cpu().numpy()).max() < 1e-12 * scale


def test_empty_and_errors():
    torch = _torch()
    lib = _lib()
    plan = lib.IstpPlan(3, 1, "fp32")
    nin, nout = plan.nin, plan.nout
    x = torch.zeros((4, nin), device="cuda")
    out = torch.zeros((4, nout), device="cuda")
    lib.istp_forward(plan._h, x.data_ptr(), x.data_ptr(), out.data_ptr(), 0, None)   # N == 0: no launch
    with pytest.raises(lib.CgtpError) as e:
        lib.istp_forward(plan._h, x.data_ptr() + 4, x.data_ptr(), out.data_ptr(), 4, None)
    assert e.value.code == lib.CGTP_EINVAL
    with pytest.raises(lib.CgtpError) as e:
        lib.istp_forward(plan._h, x.data_ptr(), x.data_ptr(), x.data_ptr(), 1, None)   # out overlaps x1
    assert e.value.code == lib.CGTP_EINVAL
    with pytest.raises(lib.CgtpError) as e:
        lib.istp_forward(plan._h, x.data_ptr(), x.data_ptr(), out.data_ptr(), -1, None)
    assert e.value.code == lib.CGTP_EINVAL
    for L, spin, dtype, code in [(34, 0, "fp32", lib.CGTP_EUNSUP), (13, 1, "fp64", lib.CGTP_EUNSUP),
                                 (21, 2, "fp32", lib.CGTP_EUNSUP), (13, 2, "fp64", lib.CGTP_EUNSUP),
                                 (-1, 0, "fp32", lib.CGTP_EINVAL), (2, 3, "fp32", lib.CGTP_EINVAL),
                                 (2, 0, 7, lib.CGTP_EDTYPE)]:
        with pytest.raises(lib.CgtpError) as e:
            lib.istp_plan(L, spin, dtype)
        assert e.value.code == code
    q = plan.query()
    assert q["n_theta"] == 8 and q["n_phi"] == 16 and q["pairs_per_group"] >= 1
    torch.cuda.synchronize()


def test_largest_sizes():
    """The largest L of each precision (fp32 at L = 33 on a few pairs, fp64 at L = 12)."""
    for L, spin, N, dtype in ((33, 1, 2, "fp32"), (33, 0, 3, "fp32"), (12, 1, 3, "fp64"), (20, 2, 2, "fp32"),
                              (12, 2, 2, "fp64")):
        x1, x2 = wl.draw_rows((2 * spin + 1) * (L + 1) ** 2, N, dtype, seed=500 + L + spin)
        got = run_gpu(L, spin, x1, x2, dtype)
        err, lab = per_label_rel_err(2 * L, spin, got, reference(L, spin, x1, x2))
        print("L=%d spin=%d %s worst %s %.3e" % (L, spin, dtype, lab, err))
        assert err <= TOL[dtype], (lab, err)


# ---------------------------------------------------------------- gradients

BACKWARD_CASES = [(1, 0, 5, "fp64"), (2, 1, 7, "fp64"), (3, 0, 9, "fp32"), (4, 1, 6, "fp32"), (6, 1, 5, "fp64"),
                  (8, 0, 4, "fp32"), (5, 0, 3, "fp64"), (7, 1, 3, "fp32"),
                  # spin 2: symmetric coupling, the same time reversal
                  (1, 2, 5, "fp32"), (2, 2, 4, "fp64"), (4, 2, 3, "fp32"), (6, 2, 2, "fp32")]


def run_backward(L, spin, x1, x2, g, dtype):
    torch = _torch()
    plan = _lib().IstpPlan(L, spin, dtype)
    a, b, gg = x1.to("cuda"), x2.to("cuda"), g.to("cuda")
    g1, g2 = plan.backward(a, b, gg)
    torch.cuda.synchronize()
    return g1.cpu().double().numpy(), g2.cpu().double().numpy()


@pytest.mark.parametrize("L,spin,N,dtype", BACKWARD_CASES)
def test_backward_small(L, spin, N, dtype):
    """Both gradients against the oracle's derivative of the bilinear map, every pair."""
    nin, nout = (2 * spin + 1) * (L + 1) ** 2, (2 * spin + 1) * (2 * L + 1) ** 2
    x1, x2 = wl.draw_rows(nin, N, dtype, seed=2000 + 10 * L + spin)
    g, _ = wl.draw_rows(nout, N, dtype, seed=3000 + 10 * L + spin)
    got1, got2 = run_backward(L, spin, x1, x2, g, dtype)
    ref1, ref2 = oi.product_vjp(spin, L, x1.double().numpy(), x2.double().numpy(), g.double().numpy())
    e1, l1 = per_label_rel_err(L, spin, got1, ref1)
    e2, l2 = per_label_rel_err(L, spin, got2, ref2)
    print("backward L=%d spin=%d N=%d %s worst labels %s %.3e, %s %.3e" % (L, spin, N, dtype, l1, e1, l2, e2))
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype], (l1, e1, l2, e2)


@pytest.mark.parametrize("L,spin", [(18, 1), (31, 0), (16, 1), (11, 2)])
def test_backward_largest(L, spin):
    """The largest fp32 gradient products: <g, z(x1, x2)> = <grad_x1, x1> = <grad_x2, x2> with the GPU forward,
    and (where the oracle's degree range allows) the time-reversed product of the oracle on one pair."""
    torch = _torch()
    nin, nout = (2 * spin + 1) * (L + 1) ** 2, (2 * spin + 1) * (2 * L + 1) ** 2
    x1, x2 = wl.draw_rows(nin, 6, "fp32", seed=4000 + L)
    g, _ = wl.draw_rows(nout, 6, "fp32", seed=4100 + L)
    plan = _lib().IstpPlan(L, spin, "fp32")
    a, b, gg = x1.cuda(), x2.cuda(), g.cuda()
    z = plan.forward(a, b)
    g1, g2 = plan.backward(a, b, gg)
    torch.cuda.synchronize()
    z, g1, g2 = (t.double().cpu().numpy() for t in (z, g1, g2))
    want = (g.double().numpy() * z).sum(1)
    scale = np.abs(g.double().numpy()).sum(1) * np.abs(z).max(1)
    assert np.all(np.abs((g1 * x1.double().numpy()).sum(1) - want) <= 1e-5 * scale)
    assert np.all(np.abs((g2 * x2.double().numpy()).sum(1) - want) <= 1e-5 * scale)
    if 2 * L <= 36:
        fn = {0: oi.gaunt_tp, 1: oi.vector_tp}.get(spin, lambda *a, **k: oi.spin_tp(spin, *a, **k))
        from test_istp_oracle import _reverse
        ref1 = fn(2 * L, g[:1].double().numpy(), _reverse(spin, L, x2[:1].double().numpy()), L2=L, Lo=L)
        e1, lab = per_label_rel_err(L, spin, g1[:1], ref1)
        print("backward L=%d spin=%d worst label %s rel err %.3e" % (L, spin, lab, e1))
        assert e1 <= TOL["fp32"], (lab, e1)


def test_backward_errors():
    torch = _torch()
    lib = _lib()
    plan = lib.IstpPlan(3, 1, "fp32")
    x = torch.zeros((4, plan.nin), device="cuda")
    g = torch.zeros((4, plan.nout), device="cuda")
    gx = torch.zeros((4, plan.nin), device="cuda")
    lib.istp_backward(plan._h, x.data_ptr(), x.data_ptr(), g.data_ptr(), gx.data_ptr(), None, 0, None)
    with pytest.raises(lib.CgtpError) as e:   # no gradient asked for
        lib.istp_backward(plan._h, x.data_ptr(), x.data_ptr(), g.data_ptr(), None, None, 4, None)
    assert e.value.code == lib.CGTP_EINVAL
    with pytest.raises(lib.CgtpError) as e:   # a gradient over an input
        lib.istp_backward(plan._h, x.data_ptr(), x.data_ptr(), g.data_ptr(), x.data_ptr(), None, 4, None)
    assert e.value.code == lib.CGTP_EINVAL
    with pytest.raises(lib.CgtpError) as e:   # the two gradients overlap
        lib.istp_backward(plan._h, x.data_ptr(), x.data_ptr(), g.data_ptr(), gx.data_ptr(), gx.data_ptr(), 4, None)
    assert e.value.code == lib.CGTP_EINVAL
    big = lib.IstpPlan(24, 1, "fp32")   # forward only: the degree-48 lift does not fit
    with pytest.raises(lib.CgtpError) as e:
        big.backward_query()
    assert e.value.code == lib.CGTP_EUNSUP
    q = plan.backward_query()
    assert q["flops_per_pair"] > 0 and q["pairs_per_group"] >= 1
    torch.cuda.synchronize()


def test_spin_two_gradient_limit():
    """Spin-2 gradient products exist up to L = 11 (fp32); beyond, istp_backward reports CGTP_EUNSUP and
    launches nothing."""
    torch = _torch()
    lib = _lib()
    assert lib.IstpPlan(11, 2, "fp32").backward_query()["flops_per_pair"] > 0
    plan = lib.IstpPlan(12, 2, "fp32")
    x = torch.zeros((2, plan.nin), device="cuda")
    g = torch.zeros((2, plan.nout), device="cuda")
    gx = torch.zeros((2, plan.nin), device="cuda")
    with pytest.raises(lib.CgtpError) as e:
        lib.istp_backward(plan._h, x.data_ptr(), x.data_ptr(), g.data_ptr(), gx.data_ptr(), None, 2, None)
    assert e.value.code == lib.CGTP_EUNSUP
    torch.cuda.synchronize()



# ---------------------------------------------------------------- real basis

REAL_CASES = [(0, 5, "fp32"), (1, 7, "fp32"), (2, 9, "fp64"), (3, 11, "fp32"), (5, 6, "fp64"), (8, 13, "fp32"),
              (16, 3, "fp32")]


@pytest.mark.parametrize("L,N,dtype", REAL_CASES)
def test_real_basis_gaunt(L, N, dtype):
    """istp_forward_real against the real-basis oracle on every pair (ragged N)."""
    torch = _torch()
    x1, x2 = wl.draw_rows((L + 1) ** 2, N, dtype, seed=700 + L)
    plan = _lib().IstpPlan(L, 0, dtype)
    got = plan.forward_real(x1.cuda(), x2.cuda())
    torch.cuda.synchronize()
    ref = oi.gaunt_tp_real(L, x1.double().numpy(), x2.double().numpy())
    err, lab = per_label_rel_err(2 * L, 0, got.cpu().double().numpy(), ref)
    print("real basis L=%d N=%d %s worst label %s rel err %.3e" % (L, N, dtype, lab, err), flush=True)
    assert err <= TOL[dtype], (lab, err)
    plan.close()


@pytest.mark.parametrize("w", wl.REAL_WORKLOADS, ids=lambda w: w.name)
def test_real_basis_bench_workload_subsample(w):
    """istp_forward_real at the benchmark's sizes (L = 16, N = 65536) on their seeded subsamples of pairs."""
    torch = _torch()
    x1, x2 = wl.istp_inputs(w)
    plan = _lib().IstpPlan(w.L, w.spin, w.dtype)
    got = plan.forward_real(x1.cuda(), x2.cuda())
    torch.cuda.synchronize()
    idx = wl.istp_check_indices(w).numpy()
    ref = oi.spin_tp_real(w.spin, w.L, x1.double().numpy()[idx], x2.double().numpy()[idx])
    err, lab = per_label_rel_err(2 * w.L, w.spin, got.cpu().double().numpy()[idx], ref)
    print("real basis %s: %d sampled pairs, worst label %s rel err %.3e" % (w.name, len(idx), lab, err), flush=True)
    assert err <= TOL[w.dtype], (lab, err)
    plan.close()


def test_real_basis_largest_degree():
    """istp_forward_real at the largest fp32 degree the plans accept, every pair."""
    torch = _torch()
    lib = _lib()
    L, N = 33, 3
    x1, x2 = wl.draw_rows((L + 1) ** 2, N, "fp32", seed=733)
    plan = lib.IstpPlan(L, 0, "fp32")
    got = plan.forward_real(x1.cuda(), x2.cuda())
    torch.cuda.synchronize()
    ref = oi.gaunt_tp_real(L, x1.double().numpy(), x2.double().numpy())
    err, lab = per_label_rel_err(2 * L, 0, got.cpu().double().numpy(), ref)
    print("real basis L=%d (largest fp32) worst label %s rel err %.3e" % (L, lab, err), flush=True)
    assert err <= TOL["fp32"], (lab, err)
    plan.close()


def test_real_basis_gradients_largest_degree():
    """istp_backward_real at the largest degree whose plan has the gradient product, every pair, checked
    through directional derivatives against the forward oracle: <grad_x1, d> = <g, z(d, x2)> and
    <grad_x2, d> = <g, z(x1, d)> for three seeded directions d (the unit-row derivative costs
    (L + 1)^2 oracle products per pair at this degree)."""
    torch = _torch()
    lib = _lib()
    L = None
    for cand in range(33, 0, -1):
        plan = lib.IstpPlan(cand, 0, "fp32")
        if lib.istp_real_backward_workspace_bytes(plan._h, 2) >= 0:   # -1: no gradient product
            L = cand
            break
        plan.close()
    assert L is not None
    print("largest degree with real-basis gradients: L=%d" % L, flush=True)
    N = 2
    x1, x2 = wl.draw_rows((L + 1) ** 2, N, "fp32", seed=834)
    g, _ = wl.draw_rows((2 * L + 1) ** 2, N, "fp32", seed=934)
    g1, g2 = plan.backward_real(x1.cuda(), x2.cuda(), g.cuda())
    torch.cuda.synchronize()
    a, b, gg = x1.double().numpy(), x2.double().numpy(), g.double().numpy()
    G1, G2 = g1.cpu().double().numpy(), g2.cpu().double().numpy()
    rng = np.random.default_rng(L)
    for k in range(3):
        d = rng.standard_normal(a.shape)
        lhs1, rhs1 = (G1 * d).sum(1), (gg * oi.gaunt_tp_real(L, d, b)).sum(1)
        lhs2, rhs2 = (G2 * d).sum(1), (gg * oi.gaunt_tp_real(L, a, d)).sum(1)
        e1 = float(np.abs(lhs1 - rhs1).max() / np.abs(rhs1).max())
        e2 = float(np.abs(lhs2 - rhs2).max() / np.abs(rhs2).max())
        print("L=%d direction %d: rel err %.3e (x1), %.3e (x2)" % (L, k, e1, e2), flush=True)
        assert e1 <= 1e-4 and e2 <= 1e-4, (k, e1, e2)
    plan.close()


def test_real_basis_errors():
    torch = _torch()
    lib = _lib()
    plan = lib.IstpPlan(3, 0, "fp32")
    N = 4
    # spin 0 runs the real-basis kernel: no workspace (gradients likewise)
    assert lib.istp_real_workspace_bytes(plan._h, N) == 0 and lib.istp_real_workspace_bytes(plan._h, -1) == -1
    assert lib.istp_real_backward_workspace_bytes(plan._h, N) == 0
    x = torch.zeros((N, plan.nin), device="cuda")
    out = torch.full((N, plan.nout), 3.0, device="cuda")
    lib.istp_forward_real(plan._h, x.data_ptr(), x.data_ptr(), out.data_ptr(), 0, None, 0, None)
    big = torch.zeros(N * plan.nout + 64, device="cuda")
    for args in [(x.data_ptr(), x.data_ptr(), out.data_ptr() + 4, N, None, 0),       # misaligned output
                 (x.data_ptr(), x.data_ptr(), out.data_ptr(), N, None, -1),          # negative workspace size
                 (big.data_ptr(), x.data_ptr(), big.data_ptr() + 64, N, None, 0)]:   # output overlapping an input
        with pytest.raises(lib.CgtpError) as e:
            lib.istp_forward_real(plan._h, *args, None)
        assert e.value.code == lib.CGTP_EINVAL, args
    torch.cuda.synchronize()
    assert (out == 3.0).all().item()
    lib.istp_forward_real(plan._h, x.data_ptr(), x.data_ptr(), out.data_ptr(), N, None, 0, None)
    torch.cuda.synchronize()
    assert (out == 0.0).all().item()
    assert lib.istp_real_workspace_bytes(lib.IstpPlan(3, 1, "fp32")._h, N) == 0   # spin 1: real-basis kernel too
    vplan = lib.IstpPlan(3, 2, "fp32")
    vneed = lib.istp_real_workspace_bytes(vplan._h, N)
    assert vneed > 0
    vx = torch.zeros((N, vplan.nin), device="cuda")
    vout = torch.zeros((N, vplan.nout), device="cuda")
    vws = torch.zeros(vneed, dtype=torch.uint8, device="cuda")
    with pytest.raises(lib.CgtpError) as e:   # a spin-2 workspace too small
        lib.istp_forward_real(vplan._h, vx.data_ptr(), vx.data_ptr(), vout.data_ptr(), N, vws.data_ptr(),
                              vneed - 1, None)
    assert e.value.code == lib.CGTP_EINVAL
    torch.cuda.synchronize()
    plan.close()
    vplan.close()


SPIN_REAL_CASES = [(1, 1, 7, "fp32"), (1, 3, 9, "fp32"), (1, 8, 5, "fp32"), (1, 4, 6, "fp64"), (1, 16, 2, "fp32"),
                   (2, 1, 5, "fp32"), (2, 3, 6, "fp32"), (2, 2, 4, "fp64"), (2, 8, 3, "fp32")]


@pytest.mark.parametrize("spin,L,N,dtype", SPIN_REAL_CASES)
def test_real_basis_spin_products(spin, L, N, dtype):
    """istp_forward_real for the vector (spin 1) and rank-2 (spin 2) products against the real-basis oracle,
    every pair (ragged N)."""
    torch = _torch()
    x1, x2 = wl.draw_rows(oi.spin_size(spin, L), N, dtype, seed=1000 + 10 * spin + L)
    plan = _lib().IstpPlan(L, spin, dtype)
    got = plan.forward_real(x1.cuda(), x2.cuda())
    torch.cuda.synchronize()
    ref = oi.spin_tp_real(spin, L, x1.double().numpy(), x2.double().numpy())
    err, lab = per_label_rel_err(2 * L, spin, got.cpu().double().numpy(), ref)
    print("real basis spin %d L=%d N=%d %s worst label %s rel err %.3e" % (spin, L, N, dtype, lab, err), flush=True)
    assert err <= TOL[dtype], (lab, err)
    plan.close()


@pytest.mark.parametrize("L,N,dtype", [(1, 5, "fp32"), (3, 7, "fp64"), (6, 4, "fp32"), (10, 3, "fp32")])
def test_real_basis_gradients(L, N, dtype):
    """istp_backward_real against the oracle's derivative of the real-basis product, every pair."""
    torch = _torch()
    x1, x2 = wl.draw_rows((L + 1) ** 2, N, dtype, seed=800 + L)
    g, _ = wl.draw_rows((2 * L + 1) ** 2, N, dtype, seed=900 + L)
    plan = _lib().IstpPlan(L, 0, dtype)
    g1, g2 = plan.backward_real(x1.cuda(), x2.cuda(), g.cuda())
    torch.cuda.synchronize()
    r1, r2 = oi.gaunt_tp_real_vjp(L, x1.double().numpy(), x2.double().numpy(), g.double().numpy())
    e1, l1 = per_label_rel_err(L, 0, g1.cpu().double().numpy(), r1)
    e2, l2 = per_label_rel_err(L, 0, g2.cpu().double().numpy(), r2)
    print("real-basis gradients L=%d %s worst %s %.3e, %s %.3e" % (L, dtype, l1, e1, l2, e2), flush=True)
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype], (l1, e1, l2, e2)
    lib = _lib()
    vplan = lib.IstpPlan(2, 1, dtype)
    assert lib.istp_real_backward_workspace_bytes(vplan._h, N) == -1
    plan.close()
    vplan.close()

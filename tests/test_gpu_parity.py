"""GPU parity: the HIP path through the C ABI against the fp64 CPU oracle.

Bar: per-path relative L2 error (over every checked pair and component of the
path) <= 1e-4 for fp32 workloads and <= 1e-10 for fp64 ones.  The L = 2, 4
and 8 workloads are compared with the oracle on every pair; the L = 16 and 32
ones, in the benchmark's launch configuration, on a seeded subsample of pairs,
plus identities checked on every pair.
"""
import ctypes
import math

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


def path_ids(L):
    """Path index of every output column, and the list of (l1, l2, l3)."""
    pid = np.empty((L + 1) ** 4, dtype=np.int64)
    paths = []
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                off = oracle.path_offset(L, l1, l2, l3)
                pid[off:off + 2 * l3 + 1] = len(paths)
                paths.append((l1, l2, l3))
    return pid, paths


def per_path_rel_err(L, got, ref):
    pid, paths = path_ids(L)
    num = np.bincount(pid, weights=((got - ref) ** 2).sum(0), minlength=len(paths))
    den = np.bincount(pid, weights=(ref ** 2).sum(0), minlength=len(paths))
    # a path that is exactly zero (x1 = x2, l1 = l2, odd l3) is held to the scale of a typical path
    typical = np.median(den[den > 0]) if (den > 0).any() else 1.0
    rel = np.sqrt(num / np.where(den > 1e-20 * typical, den, typical))
    worst = int(np.argmax(rel))
    return float(rel[worst]), paths[worst]


def run_gpu(L, x1, x2, dtype, **grid):
    torch = _torch()
    plan = _lib().Plan(L, dtype=dtype, **grid)
    a = x1.to("cuda")
    b = x2.to("cuda") if x2 is not x1 else a
    out = plan.forward(a, b)
    torch.cuda.synchronize()
    return plan, a, b, out


def check_against_oracle(L, x1, x2, got, dtype, idx=None):
    x1d = x1.double().numpy()
    x2d = x2.double().numpy()
    if idx is not None:
        x1d, x2d = x1d[idx], x2d[idx]
    ref = oracle.cgtp(L, x1d, x2d)
    err, path = per_path_rel_err(L, got, ref)
    print("L=%d dtype=%s checked=%d worst per-path rel L2 %.3e at %s" % (L, dtype, ref.shape[0], err, path),
          flush=True)
    assert err <= TOL[dtype], (err, path)
    return err


def block_energy_check(L, a, b, out, rtol):
    """sum_l3 |z^(l1,l2,l3)|^2 = |x1^(l1)|^2 |x2^(l2)|^2 on every pair (CG unitarity)."""
    torch = _torch()
    N = out.shape[0]
    blk_of_col = torch.empty((L + 1) ** 4, dtype=torch.long)
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            off = oracle.path_offset(L, l1, l2, abs(l1 - l2))
            blk_of_col[off:off + (2 * l1 + 1) * (2 * l2 + 1)] = l1 * (L + 1) + l2
    blk_of_col = blk_of_col.cuda()
    deg_of_in = torch.tensor([l for l in range(L + 1) for _ in range(2 * l + 1)], device="cuda")
    worst = 0.0
    step = max(1, int(2e8 // out.shape[1]))
    for s in range(0, N, step):
        z = out[s:s + step].double()
        e = torch.zeros(z.shape[0], (L + 1) ** 2, dtype=torch.float64, device="cuda")
        e.index_add_(1, blk_of_col, z * z)
        n1 = torch.zeros(z.shape[0], L + 1, dtype=torch.float64, device="cuda").index_add_(
            1, deg_of_in, a[s:s + step].double() ** 2)
        n2 = torch.zeros(z.shape[0], L + 1, dtype=torch.float64, device="cuda").index_add_(
            1, deg_of_in, b[s:s + step].double() ** 2)
        want = (n1[:, :, None] * n2[:, None, :]).reshape(z.shape[0], -1)
        rel = ((e - want).abs() / want.clamp_min(1e-30)).max().item()
        worst = max(worst, rel)
    print("block energy: worst relative deviation %.3e over %d pairs" % (worst, N), flush=True)
    assert worst <= rtol


# ------------------------------------------------------------ full workloads

CHUNK = 4096   # pairs per oracle call when every pair of a workload is checked


def check_all_pairs(L, x1, x2, out, dtype):
    """Every pair against the oracle, in chunks; per-path sums of squares are
    accumulated over all chunks, so the bar is the same per-path relative L2."""
    pid, paths = path_ids(L)
    num = np.zeros(len(paths))
    den = np.zeros(len(paths))
    x1d, x2d = x1.double().numpy(), x2.double().numpy()
    N = x1d.shape[0]
    for s in range(0, N, CHUNK):
        e = min(N, s + CHUNK)
        ref = oracle.cgtp(L, x1d[s:e], x2d[s:e])
        got = out[s:e].double().cpu().numpy()
        num += np.bincount(pid, weights=((got - ref) ** 2).sum(0), minlength=len(paths))
        den += np.bincount(pid, weights=(ref ** 2).sum(0), minlength=len(paths))
    typical = np.median(den[den > 0])
    rel = np.sqrt(num / np.where(den > 1e-20 * typical, den, typical))
    worst = int(np.argmax(rel))
    print("L=%d dtype=%s checked=%d (all pairs) worst per-path rel L2 %.3e at %s"
          % (L, dtype, N, rel[worst], paths[worst]), flush=True)
    assert rel[worst] <= TOL[dtype], (rel[worst], paths[worst])


@pytest.mark.parametrize("w", wl.WORKLOADS, ids=[w.name for w in wl.WORKLOADS])
def test_workload_parity(w):
    torch = _torch()
    print("workload %s L=%d N=%d %s" % (w.name, w.L, w.N, w.dtype), flush=True)
    x1, x2 = wl.workload_inputs(w)
    plan, a, b, out = run_gpu(w.L, x1, x2, w.dtype)
    if w.check_pairs:
        idx = wl.check_indices(w).numpy()
        got = out[torch.as_tensor(idx, device="cuda")].double().cpu().numpy()
        check_against_oracle(w.L, x1, x2, got, w.dtype, idx)
    else:
        check_all_pairs(w.L, x1, x2, out, w.dtype)
    block_energy_check(w.L, a, b, out, 1e-4 if w.dtype == "fp32" else 1e-11)
    assert torch.isfinite(out).all().item()


# ------------------------------------------------------------ small cases, every element

@pytest.mark.parametrize("L,N,dtype", [(0, 5, "fp32"), (1, 1, "fp32"), (2, 33, "fp64"), (3, 37, "fp32"),
                                       (5, 1000, "fp32"), (6, 130, "fp64"), (12, 41, "fp32"), (20, 7, "fp32")])
def test_small_parity(L, N, dtype):
    torch = _torch()
    x1, x2 = wl.draw(L, N, dtype, seed=1000 + L)
    _, _, _, out = run_gpu(L, x1, x2, dtype)
    check_against_oracle(L, x1, x2, out.double().cpu().numpy(), dtype)


@pytest.mark.parametrize("L,N,dtype", [(2, 17, "fp64"), (5, 33, "fp64"), (6, 300, "fp32"), (12, 19, "fp32")])
def test_alternate_cover_parity(L, N, dtype):
    """Dot and scalar-vector products (with the per-block fall-backs; L >= 5 holds block
    (3, 5)) reach the same CGTP as the oracle, and agree with the default cover."""
    _torch()
    x1, x2 = wl.draw(L, N, dtype, seed=1000 + L)
    _, _, _, out_alt = run_gpu(L, x1, x2, dtype, cover=1)
    alt = out_alt.double().cpu().numpy()
    check_against_oracle(L, x1, x2, alt, dtype)
    _, _, _, out_dflt = run_gpu(L, x1, x2, dtype)
    err, path = per_path_rel_err(L, alt, out_dflt.double().cpu().numpy())
    print("alternate vs default cover: worst per-path rel L2 %.3e at %s" % (err, path), flush=True)
    assert err <= 2 * TOL[dtype], (err, path)


def test_fp64_size_limit():
    """fp64 plans hold fewer accumulator tiles per work-group: the largest degree that
    fits plans and passes parity; one more is refused cleanly with CGTP_EUNSUP."""
    _torch()
    lib = _lib()
    largest = None
    for L in range(16, 33):
        try:
            plan = lib.Plan(L, dtype="fp64")
        except lib.CgtpError as e:
            assert e.code == lib.CGTP_EUNSUP, e.code
            break
        plan.close()
        largest = L
    print("largest fp64 degree: %s" % largest, flush=True)
    assert largest is not None and largest >= 19
    x1, x2 = wl.draw(largest, 3, "fp64", seed=1000 + largest)
    _, _, _, out = run_gpu(largest, x1, x2, "fp64")
    check_against_oracle(largest, x1, x2, out.double().cpu().numpy(), "fp64")


def test_zero_pairs_launches_nothing():
    torch = _torch()
    lib = _lib()
    plan = lib.Plan(3)
    x = torch.zeros(0, 16, device="cuda")
    out = torch.full((0, 256), 7.0, device="cuda")
    plan.forward(x, x, out)
    torch.cuda.synchronize()


def test_aliased_inputs():
    """x1 == x2 (one buffer): odd paths with l1 = l2 vanish."""
    torch = _torch()
    L = 6
    x1, _ = wl.draw(L, 50, "fp32", seed=77)
    _, a, _, out = run_gpu(L, x1, x1, "fp32")
    got = out.double().cpu().numpy()
    check_against_oracle(L, x1, x1, got, "fp32")
    for l in range(L + 1):
        for l3 in range(1, 2 * l + 1, 2):
            off = oracle.path_offset(L, l, l, l3)
            assert np.abs(got[:, off:off + 2 * l3 + 1]).max() < 1e-4


def test_global_grid_agrees():
    torch = _torch()
    L = 7
    x1, x2 = wl.draw(L, 64, "fp32", seed=5)
    _, _, _, out = run_gpu(L, x1, x2, "fp32", n_theta=2 * L + 4, n_phi=36)
    check_against_oracle(L, x1, x2, out.double().cpu().numpy(), "fp32")


def test_deterministic_and_stream():
    torch = _torch()
    lib = _lib()
    L = 9
    x1, x2 = wl.draw(L, 300, "fp32", seed=9)
    plan = lib.Plan(L)
    a, b = x1.cuda(), x2.cuda()
    o1 = plan.forward(a, b)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        o2 = plan.forward(a, b, stream=s)
    s.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def test_forward_rejects_overlap_and_misalignment():
    torch = _torch()
    lib = _lib()
    L = 2
    plan = lib.Plan(L)
    buf = torch.zeros(4 * 81 + 64, device="cuda")
    x = buf[:4 * 9].view(4, 9)
    with pytest.raises(lib.CgtpError) as e:
        lib.cgtp_forward(plan._h, x.data_ptr(), x.data_ptr(), buf.data_ptr(), 4, None)
    assert e.value.code == lib.CGTP_EINVAL
    with pytest.raises(lib.CgtpError) as e:
        lib.cgtp_forward(plan._h, x.data_ptr() + 4, x.data_ptr(), buf.data_ptr() + 4 * 200, 1, None)
    assert e.value.code == lib.CGTP_EINVAL


def test_forward_rejects_bad_arguments():
    """N < 0 and NULL pointers are refused with CGTP_EINVAL before any launch; the output is untouched."""
    torch = _torch()
    lib = _lib()
    plan = lib.Plan(2)
    x = torch.zeros(4, 9, device="cuda")
    out = torch.full((4, 81), 3.0, device="cuda")
    f = lib._load()
    xp, op = ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(out.data_ptr())
    cases = [(xp, xp, op, -1), (None, xp, op, 4), (xp, None, op, 4), (xp, xp, None, 4)]
    for a, b, o, n in cases:
        assert f.cgtp_forward(plan._h, a, b, o, n, None) == lib.CGTP_EINVAL, (a, b, o, n)
        assert f.cgtp_forward_weighted(plan._h, a, b, None, o, n, None, None) == lib.CGTP_EINVAL, (a, b, o, n)
    torch.cuda.synchronize()
    assert (out == 3.0).all().item()


def _exchange_index(L):
    """Column of path (l2, l1, l3) for every column of path (l1, l2, l3), and the sign (-1)^(l1+l2-l3)."""
    n = (L + 1) ** 4
    idx = np.empty(n, dtype=np.int64)
    sign = np.empty(n)
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                a = oracle.path_offset(L, l1, l2, l3)
                b = oracle.path_offset(L, l2, l1, l3)
                idx[a:a + 2 * l3 + 1] = np.arange(b, b + 2 * l3 + 1)
                sign[a:a + 2 * l3 + 1] = (-1.0) ** ((l1 + l2 - l3) % 2)
    return idx, sign


def test_exchange_symmetry_full_workload():
    """Every pair of the L = 8 workload: z^(l2,l1,l3)(x2, x1) = (-1)^(l1+l2-l3) z^(l1,l2,l3)(x1, x2) (CG symmetry),
    per-path relative L2 <= 1e-4; and the alternate cover (dot / scalar-vector products) agrees with the default."""
    torch = _torch()
    w = wl.BY_L[8]
    x1, x2 = wl.workload_inputs(w)
    lib = _lib()
    plan = lib.Plan(w.L, dtype=w.dtype)
    alt = lib.Plan(w.L, dtype=w.dtype, cover=lib.CGTP_COVER_ALTERNATE)
    a, b = x1.cuda(), x2.cuda()
    z = plan.forward(a, b)
    zs = plan.forward(b, a)
    idx, sign = _exchange_index(w.L)
    zs = zs[:, torch.as_tensor(idx, device="cuda")] * torch.as_tensor(sign, device="cuda", dtype=zs.dtype)
    pid, paths = path_ids(w.L)
    pid_t = torch.as_tensor(pid, device="cuda")
    for other, what in ((zs, "exchange"), (alt.forward(a, b), "alternate cover")):
        num = torch.zeros(len(paths), device="cuda", dtype=torch.float64).index_add_(
            0, pid_t, ((other - z).double() ** 2).sum(0))
        den = torch.zeros(len(paths), device="cuda", dtype=torch.float64).index_add_(0, pid_t, (z.double() ** 2).sum(0))
        rel = (num / den.clamp_min(1e-30)).sqrt().max().item()
        print("%s: worst per-path relative L2 %.3e over %d pairs" % (what, rel, w.N), flush=True)
        assert rel <= 1e-4, what
    torch.cuda.synchronize()

"""Benchmark: full-CGTP pairs/s on one MI355X, with roofline and CPU-oracle baseline.

One step = one cgtp_forward over the whole batch (every (l1, l2) block of every
pair: lift, products, lower, per-path recovery), inputs already resident in
HBM.  The headline workload is L = 32, N = 1024 pairs, fp32; L = 16,
N = 8192 is reported beside it, each with the time of both gradients
(cgtp_backward: the block adjoint kernel and the fixed-order sums, timed
together as one step) under "backward" and of the real-basis CGTP
(cgtp_forward_real, its roofline against one CGTP's model work) under "real".  The multiple-input, multiple-output Gaunt
and vector signal products (istp_forward) are timed after it, each with its
own roofline and oracle baseline, under "istp" (with the gradients,
istp_backward, where the plan supports them).  Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "full-CGTP pairs/sec at L=16 and L=32 + % of HBM/MFMA roofline"
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector (and dense fp32 MFMA) peak
PEAK_FP64_TFLOPS = 78.6
PEAK_HBM_GBS = 8000.0


# HBM traffic of each timed step from rocprofv3 counter runs (FETCH_SIZE and
# WRITE_SIZE over a whole bench run, KiB summed over a step's launches, median
# over the timed steps), each scaled by the ratio of known bytes to the same
# counter over a plain device copy (--copy-probe).  Keyed by a digest of the
# kernel and plan sources: once they change, the figures no longer describe the
# kernel and traffic is null.
MEASURED_TRAFFIC = {
    "e0592f17ebf6f287": {
        "cgtp_L32_N1024_fp32": {"fetch_kib": 213816.3, "fetch_scale": 1.999956, "write_kib": 5726851.8, "write_scale": 1.000000},
        "cgtp_L16_N8192_fp32": {"fetch_kib": 40231.1, "fetch_scale": 1.999956, "write_kib": 3175600.4, "write_scale": 1.000000},
    },
    "2bb8a257d38c4263": {
        "cgtp_L32_N1024_fp32:backward": {"fetch_kib": 2961045.2, "fetch_scale": 1.999956, "write_kib": 300568.0, "write_scale": 1.000000},
        "cgtp_L16_N8192_fp32:backward": {"fetch_kib": 2115206.8, "fetch_scale": 1.999956, "write_kib": 342208.0, "write_scale": 1.000000},
    },
    "1b33802ce775416c": {
        "cgtp_L32_N1024_fp32:real": {"fetch_kib": 214700.0, "fetch_scale": 1.999956, "write_kib": 5877975.5, "write_scale": 1.000000},
        "cgtp_L16_N8192_fp32:real": {"fetch_kib": 40535.3, "fetch_scale": 1.999956, "write_kib": 3288884.6, "write_scale": 1.000000},
    },
    "fe115111045573c6": {
        "cgtp_L16_N512_C16_fp32_x2shared_weighted": {"fetch_kib": 30048.7, "fetch_scale": 1.999956, "write_kib": 3125639.0, "write_scale": 1.000000},
    },
    "c7165dffef5eff6e": {
        "vstp_L32_N16384_fp32": {"fetch_kib": 217106.9, "fetch_scale": 1.999956, "write_kib": 986776.2, "write_scale": 1.000000},
        "gtp_L32_N65536_fp32": {"fetch_kib": 286868.4, "fetch_scale": 1.999956, "write_kib": 1327525.3, "write_scale": 1.000000},
        "vstp_L16_N65536_fp32": {"fetch_kib": 227504.5, "fetch_scale": 1.999956, "write_kib": 1011543.4, "write_scale": 1.000000},
        "vstp_L16_N65536_fp32:backward": {"fetch_kib": 1068316.0, "fetch_scale": 1.999956, "write_kib": 522281.5, "write_scale": 1.000000},
        "tstp_L16_N16384_fp32": {"fetch_kib": 97086.0, "fetch_scale": 1.999956, "write_kib": 428170.1, "write_scale": 1.000000},
    },
    "8f1e51cd32a343ae": {
        "gtp_real_L16_N65536_fp32": {"fetch_kib": 76038.7, "fetch_scale": 1.999956, "write_kib": 347086.7, "write_scale": 1.000000},
        "gtp_real_L16_N65536_fp32:backward": {"fetch_kib": 355974.0, "fetch_scale": 1.999956, "write_kib": 176640.0, "write_scale": 1.000000},
        "vstp_real_L16_N65536_fp32": {"fetch_kib": 228015.0, "fetch_scale": 1.999956, "write_kib": 1004179.2, "write_scale": 1.000000},
    },
    "636ee2db894d691d": {
        "vstp_L16_N4096_C16_fp32_x2shared_weighted": {"fetch_kib": 170283.2, "fetch_scale": 1.999956, "write_kib": 962724.6, "write_scale": 1.000000},
    },
}


DIGEST_SOURCES = {
    "cgtp": ("cgtp_kernels.hip", "cgtp_plan.cpp", "cgtp_internal.h", "device_common.h"),
    "cgtp_backward": ("cgtp_backward.hip", "cgtp_plan.cpp", "cgtp_internal.h", "device_common.h"),
    "cgtp_real": ("cgtp_kernels_real.hip", "cgtp_kernels.hip", "cgtp_plan.cpp", "cgtp_internal.h", "device_common.h"),
    "istp": ("istp_kernels.hip", "istp_kernels_tensor.hip", "istp_plan.cpp", "istp_internal.h", "device_common.h"),
    "channels": ("cgtp_kernels.hip", "cgtp_kernels_channels.hip", "cgtp_plan.cpp", "cgtp_internal.h",
                 "device_common.h"),
    "istp_real": ("istp_kernels.hip", "istp_kernels_tensor.hip", "istp_kernels_real.hip", "istp_real.hip",
                  "istp_plan.cpp", "istp_internal.h", "device_common.h"),
    "istp_channels": ("istp_kernels.hip", "istp_kernels_channels.hip", "istp_kernels_channels_tensor.hip",
                      "istp_plan.cpp", "istp_internal.h", "device_common.h"),
}


def code_only(text):
    """C/C++ source without its comments, whitespace runs collapsed to one space:
    what the compiler sees, so that edits to comments keep a kernel's digest."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c == "/" and text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif c == "/" and text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_digest(kind="cgtp"):
    h = hashlib.sha256()
    for name in DIGEST_SOURCES[kind]:
        with open(os.path.join(ROOT, "paper_2602_21466_amd", "csrc", name), encoding="utf-8") as f:
            h.update(code_only(f.read()).encode())
    return h.hexdigest()[:16]


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def _time_launches(forward, N, steps, warmup):
    """Times `steps` launches of forward(stream) after `warmup`: HIP events on the launch stream."""
    import torch

    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        forward(stream)
    torch.cuda.synchronize()
    # per-launch events on the launch stream bracket exactly one kernel each
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(steps):
        ev[i][0].record(stream)
        forward(stream)
        ev[i][1].record(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    launch_ms = sorted(s.elapsed_time(e) for s, e in ev)
    return {"ms_per_step": total_ms / steps, "value": N * steps / (total_ms / 1e3),
            "avg_launch_ms": sum(launch_ms) / len(launch_ms), "median_launch_ms": launch_ms[len(launch_ms) // 2],
            "wall_s": wall}


def time_workload(w, steps, warmup, backward=True):
    import torch

    import cgtp_inputs
    import paper_2602_21466_amd as lib

    x1, x2 = cgtp_inputs.workload_inputs(w)
    plan = lib.Plan(w.L, dtype=w.dtype)
    a, b = x1.cuda(), x2.cuda()
    out = torch.empty((w.N, w.n_outputs), dtype=a.dtype, device="cuda")
    res = {"workload": w.name, "L": w.L, "N": w.N, "dtype": w.dtype, "plan": plan.query(), "kind": "cgtp"}
    res.update(_time_launches(lambda st: plan.forward(a, b, out, st), w.N, steps, warmup))
    if backward:
        # both gradients (block kernel and the fixed-order sums) for a seeded grad_out
        g = torch.randn(out.shape, generator=torch.Generator("cpu").manual_seed(w.seed + 2),
                        dtype=torch.float64).to(out.dtype).cuda()
        del out
        g1, g2 = torch.empty_like(a), torch.empty_like(b)
        need = lib.cgtp_backward_workspace_bytes(plan._h, w.N)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        bwd = {"workload": w.name + ":backward", "L": w.L, "N": w.N, "dtype": w.dtype,
               "plan": plan.backward_query(), "kind": "cgtp_backward"}
        bwd.update(_time_launches(lambda st: lib.cgtp_backward(plan._h, a.data_ptr(), b.data_ptr(), g.data_ptr(),
                                                               g1.data_ptr(), g2.data_ptr(), w.N, ws.data_ptr(),
                                                               need, st.cuda_stream),
                                  w.N, steps, warmup))
        res["backward"] = bwd
        del g, g1, g2, ws
        # the real spherical-harmonic basis (cgtp_forward_real: the block kernel's real-basis variant)
        out = torch.empty((w.N, w.n_outputs), dtype=a.dtype, device="cuda")
        need = lib.cgtp_real_workspace_bytes(plan._h, w.N)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        real = {"workload": w.name + ":real", "L": w.L, "N": w.N, "dtype": w.dtype, "plan": plan.query(),
                "kind": "cgtp_real"}
        real.update(_time_launches(lambda st: lib.cgtp_forward_real(plan._h, a.data_ptr(), b.data_ptr(),
                                                                    out.data_ptr(), w.N, ws.data_ptr(), need,
                                                                    st.cuda_stream),
                                   w.N, steps, warmup))
        res["real"] = real
        del out, ws
    else:
        del out
    plan.close()
    del a, b
    torch.cuda.empty_cache()
    return res


def time_istp(w, steps, warmup):
    import torch

    import cgtp_inputs
    import paper_2602_21466_amd as lib

    x1, x2 = cgtp_inputs.istp_inputs(w)
    plan = lib.IstpPlan(w.L, w.spin, w.dtype)
    a, b = x1.cuda(), x2.cuda()
    out = torch.empty((w.N, w.n_outputs), dtype=a.dtype, device="cuda")
    res = {"workload": w.name, "L": w.L, "N": w.N, "dtype": w.dtype, "plan": plan.query(), "kind": "istp"}
    res.update(_time_launches(lambda st: plan.forward(a, b, out, st), w.N, steps, warmup))
    # both gradients (two launches of the adjoint product), where the plan has it
    try:
        bq = plan.backward_query()
    except lib.CgtpError:
        bq = None
    if bq is not None:
        g = torch.randn(out.shape, generator=torch.Generator("cpu").manual_seed(w.seed + 2),
                        dtype=torch.float64).to(out.dtype).cuda()
        g1, g2 = torch.empty_like(a), torch.empty_like(b)
        bwd = {"workload": w.name + ":backward", "L": w.L, "N": w.N, "dtype": w.dtype, "plan": bq, "kind": "istp"}
        bwd.update(_time_launches(lambda st: lib.istp_backward(plan._h, a.data_ptr(), b.data_ptr(), g.data_ptr(),
                                                               g1.data_ptr(), g2.data_ptr(), w.N, st.cuda_stream),
                                  w.N, steps, warmup))
        res["backward"] = bwd
        del g, g1, g2
    plan.close()
    del out, a, b
    torch.cuda.empty_cache()
    return res


def time_channels(w, steps, warmup):
    """Channel-wise CGTP with path weights: N pairs x C channels = N C rows per launch."""
    import torch

    import cgtp_inputs
    import paper_2602_21466_amd as lib

    x1, x2, wt = cgtp_inputs.channel_inputs(w.L, w.N, w.C, w.x2_shared, w.weights, w.dtype, w.seed)
    plan = lib.Plan(w.L, dtype=w.dtype)
    a, b = x1.cuda(), x2.cuda()
    wc = wt.cuda() if wt is not None else None
    rows = w.N * w.C
    nout = (w.L + 1) ** 4
    out = torch.empty((w.N, w.C, nout), dtype=a.dtype, device="cuda")
    q = dict(plan.query())
    # compulsory bytes per row: x1 row, the x2 row (shared by C rows), weights, output row
    esz = a.element_size()
    nin = (w.L + 1) ** 2
    wbytes = 0 if wc is None else wc.numel() * esz / rows
    q["bytes_per_pair"] = esz * (nin * (1 + (1 / w.C if w.x2_shared else 1)) + nout) + wbytes
    res = {"workload": w.name, "L": w.L, "N": rows, "dtype": w.dtype, "plan": q, "kind": "channels"}
    res.update(_time_launches(lambda st: plan.forward_weighted(a, b, wc, out, st), rows, steps, warmup))
    plan.close()
    del out, a, b, wc
    torch.cuda.empty_cache()
    return res


def time_istp_real(w, steps, warmup):
    """A signal product in the real basis: spin 0 one launch of the real-basis kernel (no workspace); spins 1
    and 2 two conversions, three products and the read-back per step."""
    import torch

    import paper_2602_21466_amd as lib

    x1, x2 = draw_rows_for(w, 400)
    plan = lib.IstpPlan(w.L, w.spin, w.dtype)
    a, b = x1.cuda(), x2.cuda()
    out = torch.empty((w.N, plan.nout), dtype=a.dtype, device="cuda")
    need = lib.istp_real_workspace_bytes(plan._h, w.N)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    q = dict(plan.query())
    # the method's work: one product's (the real-basis kernel) or three products; compulsory bytes: the
    # inputs and the output once
    nprod = 1 if need == 0 else 3
    q["flops_per_pair"] = nprod * q["flops_per_pair"]
    res = {"workload": w.name, "L": w.L, "N": w.N, "dtype": w.dtype, "plan": q, "kind": "istp_real"}
    res.update(_time_launches(lambda st: plan.forward_real(a, b, out, ws, st), w.N, steps, warmup))
    # both gradients in the real basis: one real-basis gradient product each, or three plus conversions
    nbw = lib.istp_real_backward_workspace_bytes(plan._h, w.N)
    if nbw >= 0:
        bq = dict(plan.backward_query())
        bq["flops_per_pair"] = (1 if nbw == 0 else 3) * bq["flops_per_pair"]
        g = torch.randn(out.shape, generator=torch.Generator("cpu").manual_seed(w.seed + 2),
                        dtype=torch.float64).to(out.dtype).cuda()
        g1, g2 = torch.empty_like(a), torch.empty_like(b)
        wsb = torch.empty(nbw, dtype=torch.uint8, device="cuda")
        bwd = {"workload": w.name + ":backward", "L": w.L, "N": w.N, "dtype": w.dtype, "plan": bq,
               "kind": "istp_real"}
        bwd.update(_time_launches(lambda st: lib.istp_backward_real(plan._h, a.data_ptr(), b.data_ptr(), g.data_ptr(),
                                                                    g1.data_ptr(), g2.data_ptr(), w.N, wsb.data_ptr(),
                                                                    nbw, st.cuda_stream),
                                  w.N, steps, warmup))
        res["backward"] = bwd
        del g, g1, g2, wsb
    plan.close()
    del out, a, b, ws
    torch.cuda.empty_cache()
    return res


def draw_rows_for(w, seed_offset):
    import cgtp_inputs
    return cgtp_inputs.draw_rows(w.n_coeffs, w.N, w.dtype, w.L + seed_offset)


def time_istp_channels(w, steps, warmup):
    """Channel-wise signal product with label weights: N pairs x C channels = N C rows per launch."""
    import torch

    import cgtp_inputs
    import paper_2602_21466_amd as lib

    x1, x2, w1, w2, wo = cgtp_inputs.istp_channel_inputs(w.spin, w.L, w.N, w.C, w.x2_shared, w.weights, w.dtype,
                                                          w.seed)
    plan = lib.IstpPlan(w.L, w.spin, w.dtype)
    a, b = x1.cuda(), x2.cuda()
    ws = [None if t is None else t.cuda() for t in (w1, w2, wo)]
    rows = w.N * w.C
    out = torch.empty((w.N, w.C, plan.nout), dtype=a.dtype, device="cuda")
    q = dict(plan.query())
    esz = a.element_size()
    wbytes = sum(t.numel() for t in ws if t is not None) * esz / rows
    q["bytes_per_pair"] = esz * (plan.nin * (1 + (1 / w.C if w.x2_shared else 1)) + plan.nout) + wbytes
    res = {"workload": w.name, "L": w.L, "N": rows, "dtype": w.dtype, "plan": q, "kind": "istp_channels"}
    res.update(_time_launches(lambda st: plan.forward_weighted(a, b, *ws, out=out, stream=st), rows, steps, warmup))
    plan.close()
    del out, a, b, ws
    torch.cuda.empty_cache()
    return res


def global_grid_flops_per_pair(L):
    """Algorithmic flops per pair of the full CGTP on one global exact grid
    (n_theta = 2L + 2, Phi = 4L + 1, lifts once per input degree, FFT cost
    2.5 Phi log2 Phi): lift, products, longitude analysis, Legendre projection
    and recombination, summed over all (l1, l2) blocks."""
    import math
    R, Phi, H = L + 1, 4 * L + 1, 2 * L + 1
    f = 2.5 * Phi * math.log2(Phi) if Phi > 1 else 0.0
    total = 4 * R * (L + 1) ** 2 + 4 * R * (L + 1) * f
    T = rec = 0
    for j1 in range(L + 1):
        for j2 in range(L + 1):
            vec = 1 if j1 * j2 > 0 else 0
            total += R * H * (6 + 60 * vec) + (1 + 3 * vec) * R * f
            for j3 in range(abs(j1 - j2), j1 + j2 + 1):
                if (j1 + j2 + j3) % 2 == 0:
                    T += 2 * j3 + 1
                    rec += 2 * j3 + 1
                else:
                    T += 3 * (2 * j3 - 1)
                    rec += 7 * (2 * j3 + 1)
    return total + 2 * R * T + rec


def roofline(res):
    flops = res["plan"]["flops_per_pair"] * res["N"]
    t = res["avg_launch_ms"] / 1e3
    achieved = flops / t / 1e12
    peak = PEAK_FP32_TFLOPS if res["dtype"] == "fp32" else PEAK_FP64_TFLOPS
    compulsory = res["plan"]["bytes_per_pair"] * res["N"]
    hbm = compulsory / t / 1e9
    # the bound of the algorithmic work: arithmetic or HBM time at peak, whichever is longer
    bound = "alu" if flops / (peak * 1e12) >= compulsory / (PEAK_HBM_GBS * 1e9) else "hbm"
    digest = kernel_digest(res["kind"])
    m = MEASURED_TRAFFIC.get(digest, {}).get(res["workload"])
    traffic = None
    if m is not None:
        traffic = int(m["fetch_kib"] * 1024 * m["fetch_scale"] + m["write_kib"] * 1024 * m["write_scale"])
    out = {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
           "frac": round(achieved / peak, 4), "traffic": traffic,
            "flops_per_launch": flops, "compulsory_bytes_per_launch": int(compulsory),
            "hbm_gbs_compulsory": round(hbm, 1), "hbm_frac_compulsory": round(hbm / PEAK_HBM_GBS, 4),
            "avg_launch_ms": round(res["avg_launch_ms"], 4), "median_launch_ms": round(res["median_launch_ms"], 4),
            "kernel_digest": digest}
    if res["kind"] == "cgtp":
        # the same launch against the work of the method on one global grid
        fs = global_grid_flops_per_pair(res["L"]) * res["N"]
        out["flops_per_launch_global_grid"] = fs
        out["achieved_global_grid"] = round(fs / t / 1e12, 3)
        out["frac_global_grid"] = round(fs / t / 1e12 / peak, 4)
    return out


def backward_entry(rb):
    log("  backward (both gradients) %.4f ms/step, %.4g pairs/s" % (rb["ms_per_step"], rb["value"]))
    return {"value": round(rb["value"], 1), "unit": "pairs/s", "ms_per_step": round(rb["ms_per_step"], 4),
            "roofline": roofline(rb)}


def real_entry(rr):
    log("  real basis (conversions + three products) %.4f ms/step, %.4g pairs/s" % (rr["ms_per_step"], rr["value"]))
    return {"value": round(rr["value"], 1), "unit": "pairs/s", "basis": "real",
            "ms_per_step": round(rr["ms_per_step"], 4), "roofline": roofline(rr)}


def copy_probe(nbytes, reps=10):
    """Plain device-to-device copy of nbytes: the calibration for the HBM counters."""
    import torch

    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        dst.copy_(src)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    print(json.dumps({"copy_probe_bytes": nbytes, "read_kib": nbytes / 1024, "write_kib": nbytes / 1024,
                      "ms": round(ms, 4), "gbs": round(2 * nbytes / ms / 1e6, 1)}), flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, budget_s, budget_1t_s=5.0):
    import numpy as np

    import cgtp_inputs
    import oracle

    x1, x2 = cgtp_inputs.workload_inputs(w)
    a = x1.double().numpy()
    b = x2.double().numpy()
    oracle.cgtp(w.L, a[:1], b[:1])          # builds the coefficient table (reported separately)
    table_s = oracle.table_build_seconds()
    t0 = time.perf_counter()
    oracle.cgtp(w.L, a[:1], b[:1])
    t1 = max(time.perf_counter() - t0, 1e-6)
    k = int(max(1, min(w.N, budget_s / t1)))
    t0 = time.perf_counter()
    oracle.cgtp(w.L, a[:k], b[:k])
    dt = time.perf_counter() - t0
    cores = oracle.max_threads()
    # one thread, on a smaller sample (the thread count persists, so this runs last)
    t0 = time.perf_counter()
    oracle.cgtp(w.L, a[:1], b[:1], threads=1)
    t1s = max(time.perf_counter() - t0, 1e-6)
    k1 = int(max(1, min(w.N, budget_1t_s / t1s)))
    t0 = time.perf_counter()
    oracle.cgtp(w.L, a[:k1], b[:k1], threads=1)
    dt1 = time.perf_counter() - t0
    return {"value": round(k / dt, 4), "unit": "pairs/s", "cores": cores, "kind": "oracle",
            "sample": "first %d of the %d pairs of %s (naive O(L^6) fp64 oracle, OpenMP over pairs x l1; "
                      "coefficient table built beforehand in %.2f s, not timed)" % (k, w.N, w.name, table_s),
            "seconds": round(dt, 2), "value_1_thread": round(k1 / dt1, 4), "sample_1_thread": "first %d pairs" % k1,
            "host_cpu": cpu_model(), "host_threads": os.cpu_count()}


def cpu_baseline_istp(w, budget_s):
    import cgtp_inputs
    import oracle
    import oracle.istp as oi

    x1, x2 = cgtp_inputs.istp_inputs(w)
    a = x1.double().numpy()
    b = x2.double().numpy()
    fn = oi.gaunt_tp if w.spin == 0 else (oi.vector_tp if w.spin == 1 else (lambda L, x, y: oi.spin_tp(2, L, x, y)))
    fn(w.L, a[:1], b[:1])                    # coefficient table of the CGTP oracle it builds on
    t0 = time.perf_counter()
    fn(w.L, a[:1], b[:1])
    t1 = max(time.perf_counter() - t0, 1e-6)
    k = int(max(1, min(w.N, budget_s / t1)))
    t0 = time.perf_counter()
    fn(w.L, a[:k], b[:k])
    dt = time.perf_counter() - t0
    return {"value": round(k / dt, 4), "unit": "pairs/s", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": "first %d of the %d pairs of %s (coefficient-space fp64 oracle on the naive CGTP oracle)"
                      % (k, w.N, w.name), "seconds": round(dt, 2)}


def main():
    import cgtp_inputs

    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="cgtp_L32_N1024_fp32")
    ap.add_argument("--secondary", default="cgtp_L16_N8192_fp32")
    ap.add_argument("--istp", default=",".join(x.name for x in cgtp_inputs.ISTP_WORKLOADS),
                    help="comma-separated signal-product workloads, or 'none'")
    ap.add_argument("--channels", default=",".join(x.name for x in cgtp_inputs.CHANNEL_WORKLOADS),
                    help="comma-separated channel-wise (path-weighted) CGTP workloads, or 'none'")
    ap.add_argument("--istp-channels", default=",".join(x.name for x in cgtp_inputs.ISTP_CHANNEL_WORKLOADS),
                    help="comma-separated channel-wise (label-weighted) signal-product workloads, or 'none'")
    ap.add_argument("--istp-real", default=",".join(x.name for x in cgtp_inputs.REAL_WORKLOADS),
                    help="comma-separated real-basis Gaunt workloads, or 'none'")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--istp-cpu-seconds", type=float, default=4.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only; --gpus %d is not supported "
              "(pairs are independent: shard N across GPUs and run one process each)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    by_name = {w.name: w for w in cgtp_inputs.WORKLOADS}
    w = by_name[args.workload]
    log("timing %s: %d warmup, %d steps" % (w.name, args.warmup, args.steps))
    main_res = time_workload(w, args.steps, args.warmup)
    log("  %.4f ms/step, %.4g pairs/s" % (main_res["ms_per_step"], main_res["value"]))
    secondary = []
    if args.secondary and args.secondary != "none":
        for name in args.secondary.split(","):
            w2 = by_name[name]
            log("timing %s" % w2.name)
            r2 = time_workload(w2, args.steps, args.warmup)
            log("  %.4f ms/step, %.4g pairs/s" % (r2["ms_per_step"], r2["value"]))
            entry = {"workload": r2["workload"], "value": round(r2["value"], 1), "unit": "pairs/s",
                     "ms_per_step": round(r2["ms_per_step"], 4), "roofline": roofline(r2)}
            if "backward" in r2:
                entry["backward"] = backward_entry(r2["backward"])
            if "real" in r2:
                entry["real"] = real_entry(r2["real"])
            secondary.append(entry)
    channels = []
    if args.channels and args.channels != "none":
        by_ch = {x.name: x for x in cgtp_inputs.CHANNEL_WORKLOADS}
        for name in args.channels.split(","):
            wc = by_ch[name]
            log("timing %s" % wc.name)
            rc = time_channels(wc, args.steps, args.warmup)
            log("  %.4f ms/step, %.4g rows/s" % (rc["ms_per_step"], rc["value"]))
            channels.append({"workload": wc.name, "value": round(rc["value"], 1), "unit": "rows/s",
                             "rows": rc["N"], "pairs": wc.N, "channels": wc.C, "x2_shared": wc.x2_shared,
                             "weights": wc.weights, "ms_per_step": round(rc["ms_per_step"], 4),
                             "roofline": roofline(rc)})
    istp = []
    if args.istp and args.istp != "none":
        by_istp = {x.name: x for x in cgtp_inputs.ISTP_WORKLOADS}
        for name in args.istp.split(","):
            wi = by_istp[name]
            log("timing %s" % wi.name)
            ri = time_istp(wi, args.steps, args.warmup)
            log("  %.4f ms/step, %.4g pairs/s" % (ri["ms_per_step"], ri["value"]))
            entry = {"workload": wi.name, "value": round(ri["value"], 1), "unit": "pairs/s",
                     "ms_per_step": round(ri["ms_per_step"], 4), "roofline": roofline(ri)}
            if "backward" in ri:
                rb = ri["backward"]
                log("  backward (both gradients) %.4f ms/step, %.4g pairs/s" % (rb["ms_per_step"], rb["value"]))
                entry["backward"] = {"value": round(rb["value"], 1), "unit": "pairs/s",
                                     "ms_per_step": round(rb["ms_per_step"], 4), "roofline": roofline(rb)}
            istp.append(entry)
    if args.istp_real and args.istp_real != "none":
        by_re = {x.name: x for x in cgtp_inputs.REAL_WORKLOADS}
        for name in args.istp_real.split(","):
            wr = by_re[name]
            log("timing %s" % wr.name)
            rr = time_istp_real(wr, args.steps, args.warmup)
            log("  %.4f ms/step, %.4g pairs/s" % (rr["ms_per_step"], rr["value"]))
            entry = {"workload": wr.name, "value": round(rr["value"], 1), "unit": "pairs/s",
                     "basis": "real", "ms_per_step": round(rr["ms_per_step"], 4), "roofline": roofline(rr)}
            if "backward" in rr:
                rb = rr["backward"]
                log("  backward (both gradients) %.4f ms/step, %.4g pairs/s" % (rb["ms_per_step"], rb["value"]))
                entry["backward"] = {"value": round(rb["value"], 1), "unit": "pairs/s",
                                     "ms_per_step": round(rb["ms_per_step"], 4), "roofline": roofline(rb)}
            istp.append(entry)
    if args.istp_channels and args.istp_channels != "none":
        by_ic = {x.name: x for x in cgtp_inputs.ISTP_CHANNEL_WORKLOADS}
        for name in args.istp_channels.split(","):
            wc = by_ic[name]
            log("timing %s" % wc.name)
            rc = time_istp_channels(wc, args.steps, args.warmup)
            log("  %.4f ms/step, %.4g rows/s" % (rc["ms_per_step"], rc["value"]))
            istp.append({"workload": wc.name, "value": round(rc["value"], 1), "unit": "rows/s",
                         "rows": rc["N"], "pairs": wc.N, "channels": wc.C, "x2_shared": wc.x2_shared,
                         "weights": wc.weights, "ms_per_step": round(rc["ms_per_step"], 4),
                         "roofline": roofline(rc)})
    line = {
        "metric": METRIC, "value": round(main_res["value"], 1), "unit": "pairs/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(main_res["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if w.dtype == "fp32" else "f64", "data": "synthetic",
        "config": {"workload": w.name, "L": w.L, "pairs": w.N, "outputs_per_pair": w.n_outputs,
                   "grid": "per-block minimal exact Gauss-Legendre x FFT", "cover": "scalar-scalar + cross"},
        "roofline": roofline(main_res),
        "backward": backward_entry(main_res["backward"]) if "backward" in main_res else None,
        "real": real_entry(main_res["real"]) if "real" in main_res else None,
        "secondary": secondary,
        "channels": channels,
        "istp": istp,
    }
    if not args.no_cpu_baseline:
        # the signal-product baselines first: the CGTP baseline's one-thread leg
        # leaves the oracle's thread count at one
        for entry in istp:
            wi = {x.name: x for x in cgtp_inputs.ISTP_WORKLOADS}.get(entry["workload"])
            if wi is None:
                continue   # channel workloads: the row products' baseline stands for them
            log("timing the CPU oracle on %s (budget %.0f s)" % (wi.name, args.istp_cpu_seconds))
            entry["cpu_baseline"] = cpu_baseline_istp(wi, args.istp_cpu_seconds)
        log("timing the CPU oracle (budget %.0f s)" % args.cpu_seconds)
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

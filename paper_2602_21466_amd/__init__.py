"""Python binding of the MI355X CGTP library (libcgtp.so): argument marshalling only.

Every step of the tensor products runs in the HIP kernels behind the C ABI
declared in ``include/cgtp.h`` (full CGTP) and ``include/istp.h`` (the MIMO
Gaunt and vector signal products); this module passes raw device pointers and
a HIP stream through ctypes.  PyTorch is used for device memory and streams.
There is no CPU fallback: if the shared library is missing or the GPU is
absent, the calls raise.

The functions carry the C names (``cgtp_plan``, ``cgtp_forward``,
``istp_plan``, ...); ``Plan`` and ``IstpPlan`` are small convenience wrappers
around them.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from ._build import LIB as _LIB_PATH

CGTP_OK, CGTP_EINVAL, CGTP_EGRID, CGTP_EDTYPE, CGTP_ENOMEM, CGTP_EHIP, CGTP_EUNSUP = 0, -1, -2, -3, -4, -5, -6
CGTP_ESCRATCH = -7
CGTP_FP32, CGTP_FP64 = 0, 1
CGTP_COVER_DEFAULT, CGTP_COVER_ALTERNATE = 0, 1
CGTP_MAX_L = 32
KIND_NAMES = {0: "scalar-scalar", 1: "cross", 2: "scalar-vector", 3: "dot"}
ISTP_GAUNT, ISTP_VECTOR, ISTP_TENSOR = 0, 1, 2
ISTP_MAX_L = {"fp32": 33, "fp64": 12}
ISTP_TENSOR_MAX_L = {"fp32": 20, "fp64": 12}
ISTP_DESC_FIELDS = ("L", "L2", "Lo", "spin", "C", "R", "G", "Phi", "A", "B", "pairs", "nin", "nin2", "nout",
                    "n_lift", "n_proj", "acoef_len", "hc_len", "lw_len", "pw_len", "wrow", "lds_bytes", "n_bcol",
                    "flags")

_lib = None


class CgtpError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = "%s failed: %s (%d)" % (where, cgtp_strerror(code), code)
        if code == CGTP_EHIP:
            msg += ", HIP error %d" % _load().cgtp_last_hip_error()
        super().__init__(msg)


class cgtp_grid(ctypes.Structure):
    _fields_ = [("n_theta", ctypes.c_int32), ("n_phi", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("cover", ctypes.c_int32)]


class cgtp_channels(ctypes.Structure):
    _fields_ = [("channels", ctypes.c_int32), ("x2_shared", ctypes.c_int32),
                ("weights_per_pair", ctypes.c_int32), ("reserved", ctypes.c_int32)]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from ._build import build
        build(force=False)
    lib = ctypes.CDLL(_LIB_PATH)
    i32, i64, vp, dp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)
    sig = {
        "cgtp_plan": (ctypes.c_int, [i32, ctypes.POINTER(cgtp_grid), ctypes.POINTER(vp)]),
        "cgtp_forward": (ctypes.c_int, [vp, vp, vp, vp, i64, vp]),
        "cgtp_forward_weighted": (ctypes.c_int, [vp, vp, vp, vp, vp, i64, ctypes.POINTER(cgtp_channels), vp]),
        "cgtp_backward": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, i64, vp, i64, vp]),
        "cgtp_backward_workspace_bytes": (i64, [vp, i64]),
        "cgtp_backward_query": (ctypes.c_int, [vp, dp, dp]),
        "cgtp_forward_real": (ctypes.c_int, [vp, vp, vp, vp, i64, vp, i64, vp]),
        "cgtp_real_workspace_bytes": (i64, [vp, i64]),
        "cgtp_num_paths": (i64, [i32]),
        "cgtp_path_index": (i64, [i32, i32, i32, i32]),
        "cgtp_destroy": (ctypes.c_int, [vp]),
        "cgtp_num_outputs": (i64, [i32]),
        "cgtp_path_offset": (i64, [i32, i32, i32, i32]),
        "cgtp_plan_query": (ctypes.c_int, [vp, ctypes.POINTER(i32), ctypes.POINTER(i32), dp, dp, dp]),
        "cgtp_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "cgtp_last_hip_error": (ctypes.c_int, []),
        "cgtp_path_norm": (ctypes.c_int, [i32, i32, i32, i32, dp, ctypes.POINTER(i32)]),
        "cgtp_wigner_9j": (ctypes.c_double, [i32] * 9),
        "cgtp_cg_vector": (ctypes.c_double, [i32] * 5),
        "cgtp_cg_zero": (ctypes.c_double, [i32] * 3),
        "cgtp_gauss_legendre": (ctypes.c_int, [i32, vp, vp]),
        "cgtp_legendre": (ctypes.c_int, [i32, ctypes.c_double, vp]),
        "cgtp_block_grid": (ctypes.c_int, [i32, ctypes.POINTER(cgtp_grid), i32, i32,
                                           ctypes.POINTER(i32), ctypes.POINTER(i32)]),
        "istp_plan": (ctypes.c_int, [i32, i32, i32, ctypes.POINTER(vp)]),
        "istp_forward": (ctypes.c_int, [vp, vp, vp, vp, i64, vp]),
        "istp_forward_weighted": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, vp, i64, ctypes.POINTER(cgtp_channels), vp]),
        "istp_num_labels": (i64, [i32, i32]),
        "istp_forward_real": (ctypes.c_int, [vp, vp, vp, vp, i64, vp, i64, vp]),
        "istp_real_workspace_bytes": (i64, [vp, i64]),
        "istp_forward_real_static": (ctypes.c_int, [vp, vp, vp, vp, i64, vp]),
        "istp_backward_real": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, i64, vp, i64, vp]),
        "istp_real_backward_workspace_bytes": (i64, [vp, i64]),
        "istp_backward_weighted": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64,
                                                  ctypes.POINTER(cgtp_channels), vp]),
        "istp_label_index": (i64, [i32, i32, i32]),
        "istp_destroy": (ctypes.c_int, [vp]),
        "istp_num_inputs": (i64, [i32, i32]),
        "istp_num_outputs": (i64, [i32, i32]),
        "istp_label_offset": (i64, [i32, i32, i32]),
        "istp_plan_query": (ctypes.c_int, [vp, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32), dp, dp]),
        "istp_plan_describe": (ctypes.c_int, [i32, i32, i32, vp]),
        "istp_backward": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, i64, vp]),
        "istp_backward_query": (ctypes.c_int, [vp, ctypes.POINTER(i32), dp, dp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def exported_symbols():
    """Names of the C ABI entry points this binding expects."""
    return ["cgtp_plan", "cgtp_forward", "cgtp_forward_weighted", "cgtp_backward", "cgtp_backward_workspace_bytes",
            "cgtp_backward_query", "cgtp_forward_real", "cgtp_real_workspace_bytes",
            "cgtp_num_paths", "cgtp_path_index", "cgtp_destroy", "cgtp_num_outputs", "cgtp_path_offset",
            "cgtp_plan_query", "cgtp_strerror", "cgtp_last_hip_error", "cgtp_path_norm", "cgtp_wigner_9j",
            "cgtp_cg_vector", "cgtp_cg_zero", "cgtp_gauss_legendre", "cgtp_legendre", "cgtp_block_grid",
            "istp_plan", "istp_forward", "istp_forward_weighted", "istp_num_labels", "istp_label_index",
            "istp_forward_real", "istp_real_workspace_bytes", "istp_forward_real_static", "istp_backward_real",
            "istp_real_backward_workspace_bytes", "istp_backward_weighted", "istp_destroy", "istp_num_inputs", "istp_num_outputs", "istp_label_offset",
            "istp_plan_query", "istp_plan_describe", "istp_backward", "istp_backward_query"]


def _check(rc: int, where: str):
    if rc != CGTP_OK:
        raise CgtpError(rc, where)


def _grid(n_theta=0, n_phi=0, dtype="fp32", cover=0) -> cgtp_grid:
    dt = {"fp32": CGTP_FP32, "fp64": CGTP_FP64}.get(dtype, dtype)
    return cgtp_grid(int(n_theta), int(n_phi), int(dt), int(cover))


# ---------------------------------------------------------------- C names

def cgtp_strerror(code: int) -> str:
    return _load().cgtp_strerror(int(code)).decode()


def cgtp_plan(L: int, grid: cgtp_grid | None = None) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    rc = _load().cgtp_plan(int(L), ctypes.byref(grid) if grid is not None else None, ctypes.byref(h))
    _check(rc, "cgtp_plan(L=%d)" % L)
    return h


def cgtp_forward(plan, x1_ptr: int, x2_ptr: int, out_ptr: int, N: int, stream_ptr: int | None) -> None:
    rc = _load().cgtp_forward(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), ctypes.c_void_p(out_ptr),
                              int(N), ctypes.c_void_p(stream_ptr) if stream_ptr else None)
    _check(rc, "cgtp_forward")


def cgtp_forward_weighted(plan, x1_ptr: int, x2_ptr: int, w_ptr: int | None, out_ptr: int, N: int,
                          channels: int = 1, x2_shared: bool = False, weights_per_pair: bool = False,
                          stream_ptr: int | None = None) -> None:
    ch = cgtp_channels(int(channels), int(bool(x2_shared)), int(bool(weights_per_pair)), 0)
    rc = _load().cgtp_forward_weighted(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr),
                                       ctypes.c_void_p(w_ptr) if w_ptr else None, ctypes.c_void_p(out_ptr),
                                       int(N), ctypes.byref(ch), ctypes.c_void_p(stream_ptr) if stream_ptr else None)
    _check(rc, "cgtp_forward_weighted")


def cgtp_backward(plan, x1_ptr: int, x2_ptr: int, g_ptr: int, gx1_ptr: int | None, gx2_ptr: int | None, N: int,
                  ws_ptr: int, ws_bytes: int, stream_ptr: int | None = None) -> None:
    vpn = lambda p: ctypes.c_void_p(p) if p else None
    rc = _load().cgtp_backward(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), ctypes.c_void_p(g_ptr),
                               vpn(gx1_ptr), vpn(gx2_ptr), int(N), vpn(ws_ptr), int(ws_bytes), vpn(stream_ptr))
    _check(rc, "cgtp_backward")


def cgtp_backward_workspace_bytes(plan, N: int) -> int:
    return int(_load().cgtp_backward_workspace_bytes(plan, int(N)))


def cgtp_forward_real(plan, x1_ptr: int, x2_ptr: int, out_ptr: int, N: int, ws_ptr: int, ws_bytes: int,
                      stream_ptr: int | None = None) -> None:
    vpn = lambda p: ctypes.c_void_p(p) if p else None
    rc = _load().cgtp_forward_real(plan, vpn(x1_ptr), vpn(x2_ptr), vpn(out_ptr), int(N), vpn(ws_ptr), int(ws_bytes),
                                   vpn(stream_ptr))
    _check(rc, "cgtp_forward_real")


def cgtp_real_workspace_bytes(plan, N: int) -> int:
    return int(_load().cgtp_real_workspace_bytes(plan, int(N)))


def cgtp_backward_query(plan) -> dict:
    fl, by = ctypes.c_double(), ctypes.c_double()
    _check(_load().cgtp_backward_query(plan, ctypes.byref(fl), ctypes.byref(by)), "cgtp_backward_query")
    return {"flops_per_pair": fl.value, "bytes_per_pair": by.value}


def cgtp_num_paths(L: int) -> int:
    return int(_load().cgtp_num_paths(int(L)))


def cgtp_path_index(L: int, l1: int, l2: int, l3: int) -> int:
    return int(_load().cgtp_path_index(int(L), int(l1), int(l2), int(l3)))


def cgtp_destroy(plan) -> None:
    _check(_load().cgtp_destroy(plan), "cgtp_destroy")


def cgtp_num_outputs(L: int) -> int:
    return int(_load().cgtp_num_outputs(int(L)))


def cgtp_path_offset(L: int, l1: int, l2: int, l3: int) -> int:
    return int(_load().cgtp_path_offset(int(L), int(l1), int(l2), int(l3)))


def cgtp_plan_query(plan) -> dict:
    nt, nph = ctypes.c_int32(), ctypes.c_int32()
    k, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(_load().cgtp_plan_query(plan, ctypes.byref(nt), ctypes.byref(nph), ctypes.byref(k), ctypes.byref(fl),
                                   ctypes.byref(by)), "cgtp_plan_query")
    return {"n_theta": nt.value, "n_phi": nph.value, "min_abs_K": k.value,
            "flops_per_pair": fl.value, "bytes_per_pair": by.value}


def cgtp_path_norm(j1: int, j2: int, j3: int, cover: int = 0):
    K, kind = ctypes.c_double(), ctypes.c_int32()
    _check(_load().cgtp_path_norm(j1, j2, j3, cover, ctypes.byref(K), ctypes.byref(kind)), "cgtp_path_norm")
    return K.value, kind.value


def cgtp_wigner_9j(*args) -> float:
    return float(_load().cgtp_wigner_9j(*[int(a) for a in args]))


def cgtp_cg_vector(j1, m1, q, j, m) -> float:
    return float(_load().cgtp_cg_vector(j1, m1, q, j, m))


def cgtp_cg_zero(l1, l2, l3) -> float:
    return float(_load().cgtp_cg_zero(l1, l2, l3))


def cgtp_gauss_legendre(n: int):
    x = np.zeros(n)
    w = np.zeros(n)
    _check(_load().cgtp_gauss_legendre(n, x.ctypes.data, w.ctypes.data), "cgtp_gauss_legendre")
    return x, w


def cgtp_legendre(lmax: int, x: float) -> np.ndarray:
    out = np.zeros((lmax + 1) * (lmax + 2) // 2)
    _check(_load().cgtp_legendre(lmax, float(x), out.ctypes.data), "cgtp_legendre")
    return out


def cgtp_block_grid(L: int, l1: int, l2: int, grid: cgtp_grid | None = None):
    nt, nph = ctypes.c_int32(), ctypes.c_int32()
    _check(_load().cgtp_block_grid(L, ctypes.byref(grid) if grid is not None else None, l1, l2,
                                   ctypes.byref(nt), ctypes.byref(nph)), "cgtp_block_grid")
    return nt.value, nph.value


def _dtype_code(dtype) -> int:
    return {"fp32": CGTP_FP32, "fp64": CGTP_FP64}.get(dtype, dtype)


def istp_plan(L: int, spin: int, dtype="fp32") -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    rc = _load().istp_plan(int(L), int(spin), int(_dtype_code(dtype)), ctypes.byref(h))
    _check(rc, "istp_plan(L=%d, spin=%d)" % (L, spin))
    return h


def istp_forward(plan, x1_ptr: int, x2_ptr: int, out_ptr: int, N: int, stream_ptr: int | None) -> None:
    rc = _load().istp_forward(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), ctypes.c_void_p(out_ptr),
                              int(N), ctypes.c_void_p(stream_ptr) if stream_ptr else None)
    _check(rc, "istp_forward")


def istp_destroy(plan) -> None:
    _check(_load().istp_destroy(plan), "istp_destroy")


def istp_num_inputs(L: int, spin: int) -> int:
    return int(_load().istp_num_inputs(int(L), int(spin)))


def istp_num_outputs(L: int, spin: int) -> int:
    return int(_load().istp_num_outputs(int(L), int(spin)))


def istp_label_offset(spin: int, j: int, l: int) -> int:
    return int(_load().istp_label_offset(int(spin), int(j), int(l)))


def istp_forward_real(plan, x1_ptr: int, x2_ptr: int, out_ptr: int, N: int, ws_ptr: int, ws_bytes: int,
                      stream_ptr: int | None = None) -> None:
    rc = _load().istp_forward_real(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), ctypes.c_void_p(out_ptr),
                                   int(N), ctypes.c_void_p(ws_ptr) if ws_ptr else None, int(ws_bytes),
                                   ctypes.c_void_p(stream_ptr) if stream_ptr else None)
    _check(rc, "istp_forward_real")


def istp_forward_real_static(plan, x1_ptr: int, x2_ptr: int, out_ptr: int, N: int,
                             stream_ptr: int | None = None) -> None:
    rc = _load().istp_forward_real_static(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr),
                                          ctypes.c_void_p(out_ptr), int(N),
                                          ctypes.c_void_p(stream_ptr) if stream_ptr else None)
    _check(rc, "istp_forward_real_static")


def istp_real_workspace_bytes(plan, N: int) -> int:
    return int(_load().istp_real_workspace_bytes(plan, int(N)))


def istp_backward_real(plan, x1_ptr: int, x2_ptr: int, g_ptr: int, gx1_ptr: int | None, gx2_ptr: int | None,
                       N: int, ws_ptr: int, ws_bytes: int, stream_ptr: int | None = None) -> None:
    vpn = lambda p: ctypes.c_void_p(p) if p else None
    rc = _load().istp_backward_real(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), ctypes.c_void_p(g_ptr),
                                    vpn(gx1_ptr), vpn(gx2_ptr), int(N), vpn(ws_ptr), int(ws_bytes), vpn(stream_ptr))
    _check(rc, "istp_backward_real")


def istp_real_backward_workspace_bytes(plan, N: int) -> int:
    return int(_load().istp_real_backward_workspace_bytes(plan, int(N)))


def istp_backward_weighted(plan, x1_ptr: int, x2_ptr: int, w1_ptr, w2_ptr, wo_ptr, g_ptr: int, gx1_ptr, gx2_ptr,
                           N: int, channels: int = 1, weights_per_pair: bool = False,
                           stream_ptr: int | None = None) -> None:
    ch = cgtp_channels(int(channels), 0, int(bool(weights_per_pair)), 0)
    vpn = lambda p: ctypes.c_void_p(p) if p else None
    rc = _load().istp_backward_weighted(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), vpn(w1_ptr),
                                        vpn(w2_ptr), vpn(wo_ptr), ctypes.c_void_p(g_ptr), vpn(gx1_ptr), vpn(gx2_ptr),
                                        int(N), ctypes.byref(ch), vpn(stream_ptr))
    _check(rc, "istp_backward_weighted")


def istp_num_labels(L: int, spin: int) -> int:
    return int(_load().istp_num_labels(int(L), int(spin)))


def istp_label_index(spin: int, j: int, l: int) -> int:
    return int(_load().istp_label_index(int(spin), int(j), int(l)))


def istp_forward_weighted(plan, x1_ptr: int, x2_ptr: int, w1_ptr, w2_ptr, wo_ptr, out_ptr: int, N: int,
                          channels: int = 1, x2_shared: bool = False, weights_per_pair: bool = False,
                          stream_ptr: int | None = None) -> None:
    # istp_channels has the layout of cgtp_channels
    ch = cgtp_channels(int(channels), int(bool(x2_shared)), int(bool(weights_per_pair)), 0)
    vpn = lambda p: ctypes.c_void_p(p) if p else None
    rc = _load().istp_forward_weighted(plan, ctypes.c_void_p(x1_ptr), ctypes.c_void_p(x2_ptr), vpn(w1_ptr),
                                       vpn(w2_ptr), vpn(wo_ptr), ctypes.c_void_p(out_ptr), int(N), ctypes.byref(ch),
                                       vpn(stream_ptr))
    _check(rc, "istp_forward_weighted")


def istp_plan_query(plan) -> dict:
    nt, nph, pp = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    fl, by = ctypes.c_double(), ctypes.c_double()
    _check(_load().istp_plan_query(plan, ctypes.byref(nt), ctypes.byref(nph), ctypes.byref(pp), ctypes.byref(fl),
                                   ctypes.byref(by)), "istp_plan_query")
    return {"n_theta": nt.value, "n_phi": nph.value, "pairs_per_group": pp.value,
            "flops_per_pair": fl.value, "bytes_per_pair": by.value}


def istp_plan_describe(L: int, spin: int, dtype="fp32") -> dict:
    """Forward product's geometry; its gradient product's under "backward" (None outside the limits)."""
    out = np.zeros(48, dtype=np.int32)
    _check(_load().istp_plan_describe(int(L), int(spin), int(_dtype_code(dtype)), out.ctypes.data),
           "istp_plan_describe")
    d = dict(zip(ISTP_DESC_FIELDS, (int(v) for v in out[:24])))
    d["backward"] = dict(zip(ISTP_DESC_FIELDS, (int(v) for v in out[24:]))) if out[24:].any() else None
    return d


def istp_backward(plan, x1_ptr: int, x2_ptr: int, g_ptr: int, gx1_ptr: int | None, gx2_ptr: int | None, N: int,
                  stream_ptr: int | None) -> None:
    vp = ctypes.c_void_p
    rc = _load().istp_backward(plan, vp(x1_ptr), vp(x2_ptr), vp(g_ptr), vp(gx1_ptr) if gx1_ptr else None,
                               vp(gx2_ptr) if gx2_ptr else None, int(N), vp(stream_ptr) if stream_ptr else None)
    _check(rc, "istp_backward")


def istp_backward_query(plan) -> dict:
    pp, fl, by = ctypes.c_int32(), ctypes.c_double(), ctypes.c_double()
    _check(_load().istp_backward_query(plan, ctypes.byref(pp), ctypes.byref(fl), ctypes.byref(by)),
           "istp_backward_query")
    return {"pairs_per_group": pp.value, "flops_per_pair": fl.value, "bytes_per_pair": by.value}


# ---------------------------------------------------------------- convenience

class Plan:
    """Owns a cgtp plan; forward() takes and returns CUDA (HIP) torch tensors."""

    def __init__(self, L: int, n_theta: int = 0, n_phi: int = 0, dtype: str = "fp32", cover: int = 0):
        self.L = int(L)
        self.dtype = dtype
        self.grid = _grid(n_theta, n_phi, dtype, cover)
        self._h = cgtp_plan(self.L, self.grid)

    def query(self) -> dict:
        return cgtp_plan_query(self._h)

    def forward(self, x1, x2, out=None, stream=None):
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        nin = (self.L + 1) ** 2
        for t in (x1, x2):
            if not t.is_cuda or t.dtype != tdt or t.dim() != 2 or t.shape[1] != nin or not t.is_contiguous():
                raise ValueError("inputs must be contiguous %s CUDA tensors [N, %d]" % (tdt, nin))
        if x1.shape[0] != x2.shape[0]:
            raise ValueError("x1 and x2 must hold the same number of pairs")
        N = x1.shape[0]
        if out is None:
            out = torch.empty((N, cgtp_num_outputs(self.L)), dtype=tdt, device=x1.device)
        elif out.dtype != tdt or not out.is_contiguous() or tuple(out.shape) != (N, cgtp_num_outputs(self.L)):
            raise ValueError("out must be a contiguous %s tensor [N, (L+1)^4]" % tdt)
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        cgtp_forward(self._h, x1.data_ptr(), x2.data_ptr(), out.data_ptr(), N, s.cuda_stream)
        return out

    def forward_weighted(self, x1, x2, weights=None, out=None, stream=None):
        """x1: [N, C, (L+1)^2]; x2: [N, C, (L+1)^2] or [N, (L+1)^2] (shared by the channels);
        weights: None, [C, P] or [N, C, P] with P = cgtp_num_paths(L).  Returns [N, C, (L+1)^4]."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        nin, npaths = (self.L + 1) ** 2, cgtp_num_paths(self.L)
        if not x1.is_cuda or x1.dtype != tdt or x1.dim() != 3 or x1.shape[2] != nin or not x1.is_contiguous():
            raise ValueError("x1 must be a contiguous %s CUDA tensor [N, C, %d]" % (tdt, nin))
        N, C = x1.shape[0], x1.shape[1]
        if x2.dtype != tdt or not x2.is_cuda or not x2.is_contiguous() or tuple(x2.shape) not in ((N, C, nin), (N, nin)):
            raise ValueError("x2 must be a contiguous %s CUDA tensor [N, C, %d] or [N, %d]" % (tdt, nin, nin))
        shared = x2.dim() == 2
        per_pair = False
        if weights is not None:
            if weights.dtype != tdt or not weights.is_cuda or not weights.is_contiguous() or \
                    tuple(weights.shape) not in ((C, npaths), (N, C, npaths)):
                raise ValueError("weights must be a contiguous %s CUDA tensor [C, %d] or [N, C, %d]" % (tdt, npaths, npaths))
            per_pair = weights.dim() == 3
        if out is None:
            out = torch.empty((N, C, cgtp_num_outputs(self.L)), dtype=tdt, device=x1.device)
        elif out.dtype != tdt or not out.is_contiguous() or tuple(out.shape) != (N, C, cgtp_num_outputs(self.L)):
            raise ValueError("out must be a contiguous %s tensor [N, C, (L+1)^4]" % tdt)
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        cgtp_forward_weighted(self._h, x1.data_ptr(), x2.data_ptr(), weights.data_ptr() if weights is not None else None,
                              out.data_ptr(), N, C, shared, per_pair, s.cuda_stream)
        return out

    def forward_real(self, x1, x2, out=None, workspace=None, stream=None):
        """Full CGTP of real-basis inputs [N, (L+1)^2], every path in the real basis [N, (L+1)^4]."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        nin, nout = (self.L + 1) ** 2, cgtp_num_outputs(self.L)
        N = x1.shape[0]
        for t, what in ((x1, "x1"), (x2, "x2")):
            if not t.is_cuda or t.dtype != tdt or tuple(t.shape) != (N, nin) or not t.is_contiguous():
                raise ValueError("%s must be a contiguous %s CUDA tensor [N, %d]" % (what, tdt, nin))
        if out is None:
            out = torch.empty((N, nout), dtype=tdt, device=x1.device)
        elif out.dtype != tdt or not out.is_contiguous() or tuple(out.shape) != (N, nout):
            raise ValueError("out must be a contiguous %s tensor [N, (L+1)^4]" % tdt)
        # (the fused kernel needs no workspace: `workspace` is accepted and unused)
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        cgtp_forward_real(self._h, x1.data_ptr(), x2.data_ptr(), out.data_ptr(), N, None, 0, s.cuda_stream)
        return out

    def backward_query(self) -> dict:
        return cgtp_backward_query(self._h)

    def backward(self, x1, x2, grad_out, need_x1=True, need_x2=True, workspace=None, stream=None):
        """(grad_x1, grad_x2) of sum(grad_out * forward(x1, x2)); a gradient not asked for is None.
        workspace: optional uint8 CUDA tensor of at least cgtp_backward_workspace_bytes(plan, N) bytes."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        nin, nout = (self.L + 1) ** 2, cgtp_num_outputs(self.L)
        N = x1.shape[0]
        for t, n, what in ((x1, nin, "x1"), (x2, nin, "x2"), (grad_out, nout, "grad_out")):
            if not t.is_cuda or t.dtype != tdt or tuple(t.shape) != (N, n) or not t.is_contiguous():
                raise ValueError("%s must be a contiguous %s CUDA tensor [N, %d]" % (what, tdt, n))
        if not (need_x1 or need_x2):
            return None, None
        need = cgtp_backward_workspace_bytes(self._h, N)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x1.device)
        elif workspace.dtype != torch.uint8 or not workspace.is_cuda or workspace.numel() < need:
            raise ValueError("workspace must be a uint8 CUDA tensor of at least %d bytes" % need)
        g1 = torch.empty_like(x1) if need_x1 else None
        g2 = torch.empty_like(x2) if need_x2 else None
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        cgtp_backward(self._h, x1.data_ptr(), x2.data_ptr(), grad_out.data_ptr(),
                      g1.data_ptr() if g1 is not None else None, g2.data_ptr() if g2 is not None else None, N,
                      workspace.data_ptr(), workspace.numel(), s.cuda_stream)
        return g1, g2

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            cgtp_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class IstpPlan:
    """Owns an istp plan (spin 0: Gaunt product, spin 1: vector product); forward() takes CUDA (HIP) tensors."""

    def __init__(self, L: int, spin: int, dtype: str = "fp32"):
        self.L, self.spin, self.dtype = int(L), int(spin), dtype
        self._h = istp_plan(self.L, self.spin, dtype)
        self.nin = istp_num_inputs(self.L, self.spin)
        self.nout = istp_num_outputs(self.L, self.spin)

    def query(self) -> dict:
        return istp_plan_query(self._h)

    def forward(self, x1, x2, out=None, stream=None):
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        for t in (x1, x2):
            if not t.is_cuda or t.dtype != tdt or t.dim() != 2 or t.shape[1] != self.nin or not t.is_contiguous():
                raise ValueError("inputs must be contiguous %s CUDA tensors [N, %d]" % (tdt, self.nin))
        if x1.shape[0] != x2.shape[0]:
            raise ValueError("x1 and x2 must hold the same number of pairs")
        N = x1.shape[0]
        if out is None:
            out = torch.empty((N, self.nout), dtype=tdt, device=x1.device)
        elif out.dtype != tdt or not out.is_contiguous() or tuple(out.shape) != (N, self.nout):
            raise ValueError("out must be a contiguous %s tensor [N, %d]" % (tdt, self.nout))
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        istp_forward(self._h, x1.data_ptr(), x2.data_ptr(), out.data_ptr(), N, s.cuda_stream)
        return out

    def forward_weighted(self, x1, x2, w1=None, w2=None, wo=None, out=None, stream=None):
        """x1: [N, C, nin]; x2: [N, C, nin] or [N, nin] (shared by the channels); w1, w2: None, [C, nl] or
        [N, C, nl] with nl = istp_num_labels(L, spin); wo: None, [C, nlo] or [N, C, nlo] with
        nlo = istp_num_labels(2L, spin).  Returns [N, C, nout]."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        if not x1.is_cuda or x1.dtype != tdt or x1.dim() != 3 or x1.shape[2] != self.nin or not x1.is_contiguous():
            raise ValueError("x1 must be a contiguous %s CUDA tensor [N, C, %d]" % (tdt, self.nin))
        N, C = x1.shape[0], x1.shape[1]
        if x2.dtype != tdt or not x2.is_cuda or not x2.is_contiguous() or \
                tuple(x2.shape) not in ((N, C, self.nin), (N, self.nin)):
            raise ValueError("x2 must be a contiguous %s CUDA tensor [N, C, %d] or [N, %d]" % (tdt, self.nin, self.nin))
        nl, nlo = istp_num_labels(self.L, self.spin), istp_num_labels(2 * self.L, self.spin)
        given = [w for w in (w1, w2, wo) if w is not None]
        per_pair = bool(given) and given[0].dim() == 3
        for w, n in ((w1, nl), (w2, nl), (wo, nlo)):
            if w is None:
                continue
            want = (N, C, n) if per_pair else (C, n)
            if w.dtype != tdt or not w.is_cuda or not w.is_contiguous() or tuple(w.shape) != want:
                raise ValueError("weights must be contiguous %s CUDA tensors %s (all per channel or all per pair)"
                                 % (tdt, want))
        if out is None:
            out = torch.empty((N, C, self.nout), dtype=tdt, device=x1.device)
        elif out.dtype != tdt or not out.is_contiguous() or tuple(out.shape) != (N, C, self.nout):
            raise ValueError("out must be a contiguous %s tensor [N, C, %d]" % (tdt, self.nout))
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        ptr = lambda w: w.data_ptr() if w is not None else None
        istp_forward_weighted(self._h, x1.data_ptr(), x2.data_ptr(), ptr(w1), ptr(w2), ptr(wo), out.data_ptr(), N,
                              C, x2.dim() == 2, per_pair, s.cuda_stream)
        return out

    def forward_real(self, x1, x2, out=None, workspace=None, stream=None):
        """The signal product in the real spherical-harmonic basis: x1, x2 [N, nin] real-basis rows (spin 0:
        [N, (L+1)^2]); returns [N, nout].  The workspace (a uint8 CUDA tensor of istp_real_workspace_bytes bytes)
        is allocated here when not given."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        for t in (x1, x2):
            if not t.is_cuda or t.dtype != tdt or t.dim() != 2 or t.shape[1] != self.nin or not t.is_contiguous():
                raise ValueError("inputs must be contiguous %s CUDA tensors [N, %d]" % (tdt, self.nin))
        if x1.shape[0] != x2.shape[0]:
            raise ValueError("x1 and x2 must hold the same number of pairs")
        N = x1.shape[0]
        need = istp_real_workspace_bytes(self._h, N)
        if need < 0:
            raise CgtpError(CGTP_EUNSUP, "forward_real (spin %d)" % self.spin)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x1.device)
        elif workspace.dtype != torch.uint8 or not workspace.is_cuda or workspace.numel() < need:
            raise ValueError("workspace must be a uint8 CUDA tensor of at least %d bytes" % need)
        if out is None:
            out = torch.empty((N, self.nout), dtype=tdt, device=x1.device)
        elif out.dtype != tdt or not out.is_contiguous() or tuple(out.shape) != (N, self.nout):
            raise ValueError("out must be a contiguous %s tensor [N, %d]" % (tdt, self.nout))
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        istp_forward_real(self._h, x1.data_ptr(), x2.data_ptr(), out.data_ptr(), N, workspace.data_ptr(),
                          workspace.numel(), s.cuda_stream)
        return out

    def backward_weighted(self, x1, x2, grad_out, w1=None, w2=None, wo=None, stream=None):
        """Gradients w.r.t. x1 [N, C, nin] and x2 [N, C, nin] of sum(grad_out * forward_weighted(x1, x2, w1, w2, wo))."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        if not x1.is_cuda or x1.dtype != tdt or x1.dim() != 3 or x1.shape[2] != self.nin or not x1.is_contiguous():
            raise ValueError("x1 must be a contiguous %s CUDA tensor [N, C, %d]" % (tdt, self.nin))
        N, C = x1.shape[0], x1.shape[1]
        for t, n, what in ((x2, self.nin, "x2"), (grad_out, self.nout, "grad_out")):
            if not t.is_cuda or t.dtype != tdt or tuple(t.shape) != (N, C, n):
                raise ValueError("%s must be a %s CUDA tensor [N, C, %d] (x2 per channel)" % (what, tdt, n))
        nl, nlo = istp_num_labels(self.L, self.spin), istp_num_labels(2 * self.L, self.spin)
        given = [w for w in (w1, w2, wo) if w is not None]
        per_pair = bool(given) and given[0].dim() == 3
        for w, n in ((w1, nl), (w2, nl), (wo, nlo)):
            if w is None:
                continue
            want = (N, C, n) if per_pair else (C, n)
            if w.dtype != tdt or not w.is_cuda or not w.is_contiguous() or tuple(w.shape) != want:
                raise ValueError("weights must be contiguous %s CUDA tensors %s (all per channel or all per pair)"
                                 % (tdt, want))
        x2 = x2.contiguous()
        g1, g2 = torch.empty_like(x1), torch.empty_like(x2)
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        ptr = lambda w: w.data_ptr() if w is not None else None
        istp_backward_weighted(self._h, x1.data_ptr(), x2.data_ptr(), ptr(w1), ptr(w2), ptr(wo),
                               grad_out.contiguous().data_ptr(), g1.data_ptr(), g2.data_ptr(), N, C, per_pair,
                               s.cuda_stream)
        return g1, g2

    def backward_real(self, x1, x2, grad_out, workspace=None, stream=None):
        """Gradients of sum(grad_out * forward_real(x1, x2)) w.r.t. x1 and x2 (real basis, spin 0 plans)."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        N = x1.shape[0]
        for t, n, what in ((x1, self.nin, "x1"), (x2, self.nin, "x2"), (grad_out, self.nout, "grad_out")):
            if not t.is_cuda or t.dtype != tdt or tuple(t.shape) != (N, n) or not t.is_contiguous():
                raise ValueError("%s must be a contiguous %s CUDA tensor [N, %d]" % (what, tdt, n))
        need = istp_real_backward_workspace_bytes(self._h, N)
        if need < 0:
            raise CgtpError(CGTP_EUNSUP, "backward_real (spin %d, L %d)" % (self.spin, self.L))
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x1.device)
        elif workspace.dtype != torch.uint8 or not workspace.is_cuda or workspace.numel() < need:
            raise ValueError("workspace must be a uint8 CUDA tensor of at least %d bytes" % need)
        g1, g2 = torch.empty_like(x1), torch.empty_like(x2)
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        istp_backward_real(self._h, x1.data_ptr(), x2.data_ptr(), grad_out.contiguous().data_ptr(), g1.data_ptr(),
                           g2.data_ptr(), N, workspace.data_ptr(), workspace.numel(), s.cuda_stream)
        return g1, g2

    def backward_query(self) -> dict:
        return istp_backward_query(self._h)

    def backward(self, x1, x2, grad_out, need_x1=True, need_x2=True, stream=None):
        """(grad_x1, grad_x2) for grad_out = dLoss/dout; a gradient not asked for is None."""
        import torch
        tdt = {"fp32": torch.float32, "fp64": torch.float64}[self.dtype]
        N = x1.shape[0]
        for t, n in ((x1, self.nin), (x2, self.nin), (grad_out, self.nout)):
            if (not t.is_cuda or t.dtype != tdt or t.dim() != 2 or t.shape[0] != N or t.shape[1] != n
                    or not t.is_contiguous()):
                raise ValueError("backward takes contiguous %s CUDA tensors x1, x2 [N, %d] and grad_out [N, %d]"
                                 % (tdt, self.nin, self.nout))
        g1 = torch.empty_like(x1) if need_x1 else None
        g2 = torch.empty_like(x2) if need_x2 else None
        s = stream if stream is not None else torch.cuda.current_stream(x1.device)
        istp_backward(self._h, x1.data_ptr(), x2.data_ptr(), grad_out.data_ptr(),
                      g1.data_ptr() if g1 is not None else None, g2.data_ptr() if g2 is not None else None, N,
                      s.cuda_stream)
        return g1, g2

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            istp_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

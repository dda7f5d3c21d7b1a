"""Seeded synthetic workloads for the full CGTP (shared by tests and the benchmark).

This module only draws inputs; it holds none of the tensor-product arithmetic,
so both the GPU path and the CPU oracle may use it.

Recipe (one per workload): a CPU ``torch.Generator`` seeded with the degree
L draws x1, then x2, each ``randn(N, (L+1)^2)`` in float64 (iid N(0, 1)
coefficients, dense, every path present).  The "scaled" workload multiplies
each degree-l block by 1/(l+1) before the cast.  The draw is then cast to the
workload's dtype; a checker consumes the cast values upcast to float64, so a
measured error is the GPU arithmetic error alone.  Large workloads are
checked on a seeded, sorted subsample of pairs (``randperm`` with seed L+1).
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    name: str
    L: int
    N: int
    dtype: str            # "fp32" | "fp64"
    scaled: bool = False  # degree-l block multiplied by 1/(l+1)
    check_pairs: int = 0  # 0: check every pair; else size of the seeded subsample

    @property
    def seed(self) -> int:
        return self.L

    @property
    def n_coeffs(self) -> int:
        return (self.L + 1) ** 2

    @property
    def n_outputs(self) -> int:
        return (self.L + 1) ** 4


WORKLOADS = [
    Workload("cgtp_L2_N64_fp64", 2, 64, "fp64"),
    Workload("cgtp_L4_N100000_fp32", 4, 100_000, "fp32"),
    Workload("cgtp_L8_N65536_fp32_scaled", 8, 65_536, "fp32", scaled=True),
    Workload("cgtp_L16_N8192_fp32", 16, 8_192, "fp32", check_pairs=64),
    Workload("cgtp_L32_N1024_fp32", 32, 1_024, "fp32", check_pairs=4),
]
BY_L = {w.L: w for w in WORKLOADS}


def block_slice(l: int) -> slice:
    """Columns of degree l in a [.., (L+1)^2] feature row (index l^2 + l + m)."""
    return slice(l * l, (l + 1) * (l + 1))


def torch_dtype(name: str):
    import torch
    return {"fp32": torch.float32, "fp64": torch.float64}[name]


def draw(L: int, N: int, dtype: str = "fp32", scaled: bool = False, seed: int | None = None):
    """Returns (x1, x2) as CPU torch tensors [N, (L+1)^2] of the given dtype."""
    import torch
    g = torch.Generator("cpu").manual_seed(L if seed is None else seed)
    n = (L + 1) ** 2
    x1 = torch.randn(N, n, dtype=torch.float64, generator=g)
    x2 = torch.randn(N, n, dtype=torch.float64, generator=g)
    if scaled:
        s = torch.empty(n, dtype=torch.float64)
        for l in range(L + 1):
            s[block_slice(l)] = 1.0 / (l + 1)
        x1 = x1 * s
        x2 = x2 * s
    return x1.to(torch_dtype(dtype)), x2.to(torch_dtype(dtype))


def draw_rows(ncols: int, N: int, dtype: str = "fp32", seed: int = 0):
    """Returns (x1, x2) as CPU torch tensors [N, ncols]: iid N(0, 1) in float64, then cast."""
    import torch
    g = torch.Generator("cpu").manual_seed(seed)
    x1 = torch.randn(N, ncols, dtype=torch.float64, generator=g)
    x2 = torch.randn(N, ncols, dtype=torch.float64, generator=g)
    return x1.to(torch_dtype(dtype)), x2.to(torch_dtype(dtype))


# Channel-wise CGTP with path weights: x1 [N, C, (L+1)^2]; x2 [N, (L+1)^2]
# when shared by the channels of a pair, else [N, C, (L+1)^2]; weights
# [C, P] (one row per channel) or [N, C, P] (per pair), P = number of paths.
# Same recipe (iid N(0, 1) in float64, then cast), seed L + 200; x1, then x2,
# then the weights are drawn from one generator.
def num_paths(L: int) -> int:
    """Paths (l1, l2, l3) of degree L: sum over l1, l2 of 2 min(l1, l2) + 1."""
    return (L + 1) * (2 * L * L + 4 * L + 3) // 3


@dataclass(frozen=True)
class ChannelWorkload:
    name: str
    L: int
    N: int                # pairs
    C: int                # channels
    x2_shared: bool
    weights: str          # "none" | "channel" | "pair"
    dtype: str
    check_rows: int       # 0: every (pair, channel) row; else a seeded subsample of rows

    @property
    def seed(self) -> int:
        return self.L + 200


def channel_inputs(L: int, N: int, C: int, x2_shared: bool, weights: str, dtype: str = "fp32", seed: int = 0):
    """(x1, x2, w) as CPU torch tensors; w is None for weights == "none"."""
    import torch
    g = torch.Generator("cpu").manual_seed(seed)
    nin = (L + 1) ** 2
    x1 = torch.randn(N, C, nin, dtype=torch.float64, generator=g)
    x2 = torch.randn(*((N, nin) if x2_shared else (N, C, nin)), dtype=torch.float64, generator=g)
    w = None
    if weights != "none":
        shape = (C, num_paths(L)) if weights == "channel" else (N, C, num_paths(L))
        w = torch.randn(*shape, dtype=torch.float64, generator=g).to(torch_dtype(dtype))
    return x1.to(torch_dtype(dtype)), x2.to(torch_dtype(dtype)), w


def channel_check_rows(wk: ChannelWorkload):
    """Sorted (pair, channel) row indices checked against the oracle."""
    import torch
    rows = wk.N * wk.C
    if not wk.check_rows or wk.check_rows >= rows:
        return list(range(rows))
    g = torch.Generator("cpu").manual_seed(wk.seed + 1)
    return sorted(torch.randperm(rows, generator=g)[: wk.check_rows].tolist())


# A message-passing layer at the headline degree: 512 pairs (edges) of 16
# channels, the second input (the edge's harmonics) shared by the channels,
# one weight per path and channel.  8192 rows, as many as the L = 16 workload.
CHANNEL_WORKLOADS = [
    ChannelWorkload("cgtp_L16_N512_C16_fp32_x2shared_weighted", 16, 512, 16, True, "channel", "fp32", 8),
]


# Multiple-input, multiple-output signal products: spin 0 (Gaunt) rows hold
# (L+1)^2 values, spin 1 (vector) rows 3 (L+1)^2; same recipe as above
# (seed L + 100 spin), checked on a seeded subsample of pairs.
@dataclass(frozen=True)
class IstpWorkload:
    name: str
    L: int
    spin: int
    N: int
    dtype: str
    check_pairs: int

    @property
    def seed(self) -> int:
        return self.L + 100 * self.spin

    @property
    def n_coeffs(self) -> int:
        return (2 * self.spin + 1) * (self.L + 1) ** 2

    @property
    def n_outputs(self) -> int:
        return (2 * self.spin + 1) * (2 * self.L + 1) ** 2


ISTP_WORKLOADS = [
    IstpWorkload("vstp_L32_N16384_fp32", 32, 1, 16_384, "fp32", 4),
    IstpWorkload("gtp_L32_N65536_fp32", 32, 0, 65_536, "fp32", 8),
    IstpWorkload("vstp_L16_N65536_fp32", 16, 1, 65_536, "fp32", 16),
    # the rank-2 tensor-harmonic product (spin 2) at L = 16
    IstpWorkload("tstp_L16_N16384_fp32", 16, 2, 16_384, "fp32", 4),
]


def istp_inputs(w: IstpWorkload):
    return draw_rows(w.n_coeffs, w.N, w.dtype, w.seed)


def istp_check_indices(w: IstpWorkload):
    import torch
    g = torch.Generator("cpu").manual_seed(w.seed + 1)
    return torch.sort(torch.randperm(w.N, generator=g)[: w.check_pairs]).values


def workload_inputs(w: Workload):
    return draw(w.L, w.N, w.dtype, w.scaled, w.seed)


def check_indices(w: Workload):
    """Sorted pair indices a checker compares (all pairs, or the seeded subsample)."""
    import torch
    if w.check_pairs == 0 or w.check_pairs >= w.N:
        return torch.arange(w.N)
    g = torch.Generator("cpu").manual_seed(w.seed + 1)
    return torch.sort(torch.randperm(w.N, generator=g)[: w.check_pairs]).values


# Channel-wise signal products with label weights: x1 [N, C, n_in]; x2
# [N, n_in] when shared by the channels, else [N, C, n_in]; weights w1, w2
# [C, n_lab(L)], wo [C, n_lab(2L)] (per channel) or [N, C, ...] (per pair),
# n_lab irrep labels per row (L + 1, 3 L + 1 or 5 L - 1 for spin 0, 1, 2).  Same
# recipe (iid N(0, 1) in float64, then cast), seed L + 300 + spin; x1, x2,
# w1, w2, wo drawn in that order from one generator.
def istp_num_labels(L: int, spin: int) -> int:
    """Irrep labels (j, l), l <= L, |l - spin| <= j <= l + spin, of a row."""
    return sum(2 * min(l, spin) + 1 for l in range(L + 1))


@dataclass(frozen=True)
class IstpChannelWorkload:
    name: str
    L: int
    spin: int
    N: int                # pairs
    C: int                # channels
    x2_shared: bool
    weights: str          # "none" | "channel" | "pair"
    dtype: str
    check_rows: int       # 0: every row; else a seeded subsample of (pair, channel) rows

    @property
    def seed(self) -> int:
        return self.L + 300 + self.spin


def istp_channel_inputs(spin: int, L: int, N: int, C: int, x2_shared: bool, weights: str, dtype: str = "fp32",
                        seed: int = 0):
    """(x1, x2, w1, w2, wo) as CPU torch tensors; the weights are None for weights == "none"."""
    import torch
    g = torch.Generator("cpu").manual_seed(seed)
    nin = (2 * spin + 1) * (L + 1) ** 2
    x1 = torch.randn(N, C, nin, dtype=torch.float64, generator=g)
    x2 = torch.randn(*((N, nin) if x2_shared else (N, C, nin)), dtype=torch.float64, generator=g)
    ws = [None, None, None]
    if weights != "none":
        lead = (C,) if weights == "channel" else (N, C)
        for k, Lx in enumerate((L, L, 2 * L)):
            ws[k] = torch.randn(*lead, istp_num_labels(Lx, spin), dtype=torch.float64, generator=g).to(torch_dtype(dtype))
    return (x1.to(torch_dtype(dtype)), x2.to(torch_dtype(dtype))) + tuple(ws)


def istp_channel_check_rows(wk: IstpChannelWorkload):
    import torch
    rows = wk.N * wk.C
    if not wk.check_rows or wk.check_rows >= rows:
        return list(range(rows))
    g = torch.Generator("cpu").manual_seed(wk.seed + 1)
    return sorted(torch.randperm(rows, generator=g)[: wk.check_rows].tolist())


# The vector product as a message-passing layer at L = 16: 4096 pairs (edges)
# x 16 channels = 65536 rows, as many as the L = 16 row workload; x2 (the
# edge's harmonics) shared by the channels, per-channel label weights.
ISTP_CHANNEL_WORKLOADS = [
    IstpChannelWorkload("vstp_L16_N4096_C16_fp32_x2shared_weighted", 16, 1, 4096, 16, True, "channel", "fp32", 16),
]


# The Gaunt product in the real spherical-harmonic basis: rows drawn as for
# the signal products (seed L + 400), real-basis coefficients.
REAL_WORKLOADS = [
    IstpWorkload("gtp_real_L16_N65536_fp32", 16, 0, 65_536, "fp32", 8),
    IstpWorkload("vstp_real_L16_N65536_fp32", 16, 1, 65_536, "fp32", 8),
]


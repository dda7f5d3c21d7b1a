"""The C ABI without a GPU: the library loads, exports every function that
include/*.h declares, and its host-side queries agree with the oracle's
layouts and with the kernels' resource limits."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

import oracle.istp as oi
import paper_2602_21466_amd as lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        for m in re.finditer(r"^[A-Za-z_][\w\s\*]*?\b(\w+)\s*\(", text, flags=re.M):
            if not m.group(0).lstrip().startswith(("typedef", "#", "enum", "return")):
                names.add(m.group(1))
    return names


def test_library_exports_every_declared_function():
    declared = _declared()
    assert {"cgtp_plan", "cgtp_forward", "istp_plan", "istp_forward"} <= declared
    so = ctypes.CDLL(lib._build.LIB)
    missing = [n for n in sorted(declared) if not hasattr(so, n)]
    assert not missing, missing
    assert declared == set(lib.exported_symbols())


def test_istp_row_layouts_match_the_oracle():
    for L in range(6):
        assert lib.istp_num_inputs(L, 0) == oi.gaunt_size(L)
        assert lib.istp_num_inputs(L, 1) == oi.vector_size(L)
        assert lib.istp_num_outputs(L, 0) == oi.gaunt_size(2 * L)
        assert lib.istp_num_outputs(L, 1) == oi.vector_size(2 * L)
        for j, l in oi.vector_labels(L):
            assert lib.istp_label_offset(1, j, l) == oi.vector_offset(j, l)
        for l in range(L + 1):
            assert lib.istp_label_offset(0, l, l) == l * l
    for L in range(6):
        assert lib.istp_num_inputs(L, 2) == oi.spin_size(2, L)
        assert lib.istp_num_outputs(L, 2) == oi.spin_size(2, 2 * L)
        assert lib.istp_num_labels(L, 2) == len(oi.spin_labels(2, L))
        for k, (j, l) in enumerate(oi.spin_labels(2, L)):
            assert lib.istp_label_offset(2, j, l) == oi.spin_offset(2, j, l)
            assert lib.istp_label_index(2, j, l) == k
    assert lib.istp_label_offset(1, 0, 0) == -1 and lib.istp_label_offset(1, 3, 1) == -1
    assert lib.istp_label_offset(0, 1, 2) == -1 and lib.istp_num_inputs(-1, 0) == -1
    assert lib.istp_label_offset(2, 1, 0) == -1 and lib.istp_label_offset(2, 0, 1) == -1
    assert lib.istp_num_inputs(3, 3) == -1


@pytest.mark.parametrize("dtype", ["fp32", "fp64"])
def test_istp_plan_geometry(dtype):
    """Every supported plan fits LDS and the accumulator budget; the grid is the exact one."""
    esz = 4 if dtype == "fp32" else 8
    for spin in (0, 1, 2):
        # accumulator tiles a wave may hold (spin 2 keeps its products' ten components in registers)
        mt = min(13 if dtype == "fp32" else 4, 7 if spin == 2 else 13)
        lmax = (lib.ISTP_TENSOR_MAX_L if spin == 2 else lib.ISTP_MAX_L)[dtype]
        for L in range(lmax + 1):
            d = lib.istp_plan_describe(L, spin, dtype)
            assert d["R"] == L + 1 and d["Phi"] >= 4 * L + 1 and d["A"] * d["B"] == d["Phi"]
            assert d["lds_bytes"] <= 160 * 1024
            assert d["n_proj"] <= 16 * mt
            assert 2 * d["C"] * d["pairs"] <= 16 and d["G"] in (4, 8, 12, 16)
            assert d["hc_len"] == d["C"] * (2 * L + 1) ** 2
            assert d["nin"] == lib.istp_num_inputs(L, spin) and d["nout"] == lib.istp_num_outputs(L, spin)
            assert d["pairs"] * d["hc_len"] * esz + 16 <= d["lds_bytes"] + 16
        with pytest.raises(lib.CgtpError):
            lib.istp_plan_describe(lmax + 1, spin, dtype)

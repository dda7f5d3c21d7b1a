"""Compiles the HIP library (libcgtp.so: full CGTP and the MIMO signal products) in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libcgtp.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in
           ("cgtp_plan.cpp", "cgtp_kernels.hip", "cgtp_kernels_channels.hip", "cgtp_backward.hip", "cgtp_kernels_real.hip", "istp_plan.cpp", "istp_kernels.hip", "istp_kernels_real.hip",
            "istp_kernels_channels.hip", "istp_kernels_tensor.hip", "istp_kernels_channels_tensor.hip",
            "istp_real.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed FP32 instructions are switched off for all device code.
FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-Wall", "-Wno-unused-result"]


def build(force: bool = True, extra=None) -> str:
    """Compiles every source to an object in parallel (one hipcc each), then links the library."""
    if not force and os.path.exists(LIB):
        return LIB
    tag = ".tmp%d" % os.getpid()
    objs = [os.path.join(HERE, "csrc", os.path.basename(src) + tag + ".o") for src in SOURCES]
    compile_flags = [f for f in FLAGS if f != "-shared"]
    procs = [subprocess.Popen([HIPCC] + compile_flags + list(extra or []) + ["-c", src, "-o", obj])
             for src, obj in zip(SOURCES, objs)]
    failed = [src for src, p in zip(SOURCES, procs) if p.wait() != 0]
    try:
        if failed:
            raise subprocess.CalledProcessError(1, "hipcc", "failed: %s" % ", ".join(failed))
        tmp = LIB + tag
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp], check=True)
        os.replace(tmp, LIB)
    finally:
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    return LIB


if __name__ == "__main__":
    print(build())

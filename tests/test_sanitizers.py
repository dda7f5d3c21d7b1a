"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The plan sources (cgtp_plan.cpp, istp_plan.cpp) are built host-only with g++
against a stand-in for the HIP runtime (tests/sanitize/: four runtime calls
and the kernel launchers stubbed, allocations failing), together with the
oracle (oracle/cgtp_oracle.c), and driven by tests/sanitize/driver.cpp: every
plan's host maths and table building up to L = 32, the exported host maths,
istp_plan_describe, argument validation and the oracle's products and
gradients.  Any sanitizer report (out-of-bounds access, leak, signed
overflow, invalid shift, ...) ends the run with a non-zero status.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2602_21466_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if shutil.which("g++") is None or shutil.which("gcc") is None:
        pytest.skip("no host compiler")
    out = tmp_path_factory.mktemp("san")
    flags = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    inc = ["-D__HIP_PLATFORM_AMD__", "-I", SAN, "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include")]
    objs = []
    jobs = []
    for src, cc in ((os.path.join(CSRC, "cgtp_plan.cpp"), "g++"), (os.path.join(CSRC, "istp_plan.cpp"), "g++"),
                    (os.path.join(SAN, "stubs.cpp"), "g++"), (os.path.join(SAN, "driver.cpp"), "g++"),
                    (os.path.join(ROOT, "oracle", "cgtp_oracle.c"), "gcc")):
        obj = str(out / (os.path.basename(src) + ".o"))
        std = ["-std=c++17"] if cc == "g++" else ["-std=c11", "-fopenmp"]
        jobs.append(subprocess.Popen([cc] + std + flags + inc + ["-c", src, "-o", obj],
                                     stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
        objs.append(obj)
    for j in jobs:
        log = j.communicate(timeout=600)[0].decode(errors="replace")
        assert j.returncode == 0, log[-3000:]
    exe = str(out / "driver")
    r = subprocess.run(["g++"] + flags + objs + ["-fopenmp", "-lm", "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


def test_host_code_is_clean_under_asan_and_ubsan(driver):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    r = subprocess.run([driver], capture_output=True, text=True, timeout=900, env=env)
    print(r.stdout[-2000:])
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "sanitized host code OK" in r.stdout
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr

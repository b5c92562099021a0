"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Two instrumented programs are built here (cached under _build/san by a hash
of their sources and flags) and run on the CPU:

- the CPU oracle (oracle/oracle.c) with a driver that runs every oracle
  function on small, ragged and empty shapes and checks it against plain
  loops or the oracle's second form (tests/sanitize/oracle_san.c);
- libqx's host side -- argument validation, every planner, and executor
  create / run / profile / destroy with injected allocation failures through
  the host double of the device runtime (tests/sanitize/qx_san.cpp).  The
  device code is compiled as usual and never runs; only host code carries
  the sanitizers.

Any sanitizer report aborts the program (-fno-sanitize-recover=all), and
leaks are reported at exit.
"""
import concurrent.futures as cf
import hashlib
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_DIR = os.path.join(ROOT, "_build", "san")
CSRC = os.path.join(ROOT, "paper_2606_09905_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

QX_SOURCES = [os.path.join(CSRC, f) for f in
              ("api.cpp", "k_gemm.hip", "k_gemm_nt.hip", "k_valu.hip", "k_attn.hip", "k_reduce.hip", "scratch.hip")]
# every -fsanitize= applies to the host pass only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
HIP_FLAGS = ["-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include")]
GCC_SAN = ["gcc", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-std=c11", "-Wall", "-Wextra"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1",
           OMP_NUM_THREADS="2")


def _digest(paths, flags):
    h = hashlib.sha256(" ".join(flags).encode())
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd[:3])} ... failed:\n{r.stderr[-4000:]}")


def _build_oracle():
    srcs = [os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "tests", "sanitize", "oracle_san.c")]
    exe = os.path.join(SAN_DIR, f"oracle_san_{_digest(srcs, GCC_SAN)}")
    if not os.path.exists(exe):
        os.makedirs(SAN_DIR, exist_ok=True)
        _run(GCC_SAN + srcs + ["-o", exe + ".tmp", "-lm"])
        os.replace(exe + ".tmp", exe)
    return exe


def _build_qx():
    driver = os.path.join(ROOT, "tests", "sanitize", "qx_san.cpp")
    headers = [os.path.join(ROOT, "include", h) for h in ("qx.h", "qx_testing.h")] + \
              [os.path.join(CSRC, "qx_internal.h")]
    srcs = QX_SOURCES + [driver]
    exe = os.path.join(SAN_DIR, f"qx_san_{_digest(srcs + headers, HIP_FLAGS + HOST_SAN)}")
    if os.path.exists(exe):
        return exe
    os.makedirs(SAN_DIR, exist_ok=True)

    def obj(src):
        o = os.path.join(SAN_DIR, os.path.basename(src) + ".san.o")
        _run([HIPCC, *HIP_FLAGS, *HOST_SAN, "-c", src, "-o", o])
        return o

    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(obj, srcs))
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, *objs, "-o", exe + ".tmp"])
    os.replace(exe + ".tmp", exe)
    return exe


def _check(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=600)
    report = r.stdout[-2000:] + r.stderr[-6000:]
    assert r.returncode == 0, report
    assert r.stdout.strip().endswith("ok"), report
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, report


def test_oracle_under_asan_ubsan():
    _check(_build_oracle())


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_planner_and_executor_under_asan_ubsan():
    _check(_build_qx())

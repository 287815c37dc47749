"""Build libhpd.so (gfx950 HIP kernels + the C ABI) in-tree.

    python -m paper_2607_18839_amd.build

Every HIP source is compiled with hipcc for gfx950 only; the host planner is
plain C++ built with g++.  Objects go to paper_2607_18839_amd/_build/ and the
library to paper_2607_18839_amd/libhpd.so.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhpd.so")
PEAKS = os.path.join(PKG, "peaks")   # microbenchmark of the box's own peaks (bench.py runs it for box_peaks)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_SOURCES = ["attn_kernels.hip", "gemm_kernels.hip", "decode.hip", "pmtp.hip", "timing.hip", "api.hip"]
CXX_SOURCES = ["plan.cpp", "kv_pool.cpp", "scheduler.cpp"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
# Packed fp32 VALU forms are disabled for all device code.  MFMA results
# are kept in architectural VGPRs (the accumulator-register form made the
# allocator shuttle accumulators through v_accvgpr moves inside the k loops).
HIP_FLAGS = COMMON + [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
                      "-packed-fp32-ops", "-mllvm", "-amdgpu-mfma-vgpr-form",
                      "-Wno-unused-command-line-argument"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    for s in HIP_SOURCES:
        src = os.path.join(CSRC, s)
        if os.path.exists(src):
            jobs.append([HIPCC] + HIP_FLAGS + ["-c", src, "-o", os.path.join(BUILD, s + ".o")])
    for s in CXX_SOURCES:
        jobs.append(["g++"] + COMMON + ["-Wall", "-c", os.path.join(CSRC, s), "-o", os.path.join(BUILD, s + ".o")])
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        for out in ex.map(_run, jobs):
            if verbose and out.strip():
                print(out)
    objs = [j[-1] for j in jobs]
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs)
    os.replace(tmp, LIB)
    _run([HIPCC] + HIP_FLAGS + ["-o", PEAKS + ".tmp", os.path.join(CSRC, "peaks.hip")])
    os.replace(PEAKS + ".tmp", PEAKS)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

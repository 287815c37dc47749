"""The host-side C++ (planner, paged K/V pool, Algorithm 1 scheduler) under
AddressSanitizer and UndefinedBehaviorSanitizer: tests/native/host_stress.cpp
is built with those three sources by g++ (host code only, no HIP) and run
over several seeds of random valid and invalid inputs.  Its invariants are
listed in its header; any sanitizer report aborts the run."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_18839_amd", "csrc")
FLAGS = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")


def _build(out_dir, sources, name):
    exe = os.path.join(out_dir, name)
    cmd = ["g++", *FLAGS, "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, *sources, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


@pytest.fixture(scope="module")
def stress_exe(tmp_path_factory):
    d = str(tmp_path_factory.mktemp("host_stress"))
    srcs = [os.path.join(ROOT, "tests", "native", "host_stress.cpp")] + \
           [os.path.join(CSRC, f) for f in ("plan.cpp", "kv_pool.cpp", "scheduler.cpp")]
    return _build(d, srcs, "host_stress")


def test_sanitizers_are_active(tmp_path):
    """Control: a heap overflow built with the same flags is reported, so a
    clean stress run means something."""
    src = tmp_path / "overflow.cpp"
    src.write_text("#include <vector>\nint main(int c, char **) { std::vector<int> v(4); return v.data()[3 + c]; }\n")
    exe = _build(str(tmp_path), [str(src)], "overflow")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr


@pytest.mark.parametrize("seed", range(6))
def test_host_stress_under_sanitizers(stress_exe, seed):
    r = subprocess.run([stress_exe, str(seed), "1500"], capture_output=True, text=True, timeout=600,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1"))
    print(r.stdout)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "iterations ok" in r.stdout

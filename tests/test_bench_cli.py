"""bench.py command-line contract that needs no GPU."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_algorithmic_work_of_c3():
    sys.path.insert(0, ROOT)
    import bench
    from workloads import make_attn_batch
    b = make_attn_batch("c3", 0)
    w = bench.attn_work(b.prefix_len, b.branch_page, b.num_new, b.past_len, 16, 2, 64, 2, 2)
    assert w["T"] == 129
    assert w["shared_flop"] == 4 * 16 * 64 * 129 * 4096 == 2164260864
    rows = int((b.past_len + b.num_new).sum())
    assert w["private_bytes"] == 2 * rows * 2 * 64 * 2 + 2 * 129 * 16 * 64 * 2


def test_traffic_summaries_parse_and_cover_the_reported_kernels():
    """The bench reads HBM bytes per launch from profiles/traffic_<workload>.md;
    every kind it may report is there as a positive byte count (the figure
    itself is used only while its kernel source is unchanged)."""
    import re
    sys.path.insert(0, ROOT)
    import bench
    kinds = {"c4": ("shared_prefix", "merge", "gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "norm_input",
                    "shared_phase", "private_phase", "lm_head", "verify", "draft_token"),
             "c5": ("shared_prefix", "merge", "shared_phase", "private_phase")}
    for workload, names in kinds.items():
        text = open(os.path.join(ROOT, "profiles", f"traffic_{workload}.md")).read()
        block = json.loads(re.search(r"```json\n(.*?)```", text, re.S).group(1))
        assert block["fetch_factor"] > 0 and block["write_factor"] > 0
        for n in names:
            k = block["kernels"][n]
            assert k["traffic_bytes"] > 0 and k["source"] in block["code_sha256"]
            got = bench._traffic(n, workload)
            assert got is None or got == k["traffic_bytes"]
    assert bench._traffic("shared_prefix", "c9") is None   # no summary: no figure


def test_code_digest_ignores_comments_only(tmp_path):
    sys.path.insert(0, ROOT)
    import bench
    a, b, c = tmp_path / "a.hip", tmp_path / "b.hip", tmp_path / "c.hip"
    a.write_text("int f(int x) {  // doubles\n  return 2 * x;\n}\n")
    b.write_text("/* header */\n// a note\nint f(int x) {\n\n  return 2 * x;   // the same code\n}\n")
    c.write_text("int f(int x) {\n  return 3 * x;\n}\n")
    assert bench.code_digest(str(a)) == bench.code_digest(str(b)) != bench.code_digest(str(c))


def test_box_peak_only_for_the_measured_units():
    """The box's own peaks cover bf16 MFMA and HBM reads: a bf16 or HBM
    roofline gets the second denominator, an fp32 one gets none."""
    sys.path.insert(0, ROOT)
    import bench
    pk = {"read_gbs": 6400.0, "mfma_bf16_tflops": 2340.0}
    r = bench.add_box_peak({"unit": "TFLOP/s", "peak": bench.BF16_PEAK_TFLOPS, "achieved": 234.0}, pk)
    assert r["box_peak"] == 2340.0 and abs(r["box_frac"] - 0.1) < 1e-12
    r = bench.add_box_peak({"unit": "GB/s", "peak": 8000.0, "achieved": 3200.0}, pk)
    assert r["box_peak"] == 6400.0 and abs(r["box_frac"] - 0.5) < 1e-12
    r = bench.add_box_peak({"unit": "TFLOP/s", "peak": bench.FP32_PEAK_TFLOPS, "achieved": 0.3}, pk)
    assert r["box_peak"] is None and r["box_frac"] is None
    assert bench.add_box_peak(None, pk) is None

"""Benchmark of the branch-parallel decode step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4|c3|c5|c2|c1]

A step is one pass of the whole hot path over one batch of seeded synthetic
input already resident in HBM.  The default workload is c4, the full decode
step of the 18-layer synthetic decoder (RMSNorm + QKV projection with the new
K/V appended, shared-prefix / private / merge attention kernels, O projection,
RMSNorm + SwiGLU MLP, per layer) over one dense page: 1 layout branch (k = 1,
512 past tokens) and 32 content branches (k = 4, lognormal past lengths) with
a 4096-token shared prefix.  The single-layer workloads c1, c2, c3 and c5 time
one hpd_branch_attn_step.

Prints one JSON line.  `value` is branch-tokens/s = (sum of k_b) / step time.
`roofline` describes the dominant kernel; its duration comes from HIP events
recorded by the library around each of its launches during a second timed
pass of the same K steps.  `cpu_baseline` times the fp64 oracle on the host.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--layers", type=int, default=None, help="c4 only: fewer layers (not for reporting)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--warm", action="store_true", help="attention workloads: reuse one input replica")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    return ap.parse_args()


# ----------------------------------------------------------------- algorithmic work

def attn_work(prefix_len, branch_page, num_new, past_len, Hq, Hkv, D, s_in, s_out):
    """Algorithmic FLOPs / bytes of the shared and private phases (method's
    definition: what must be read and computed, not implementation scratch)."""
    prefix_len = np.asarray(prefix_len, np.int64)
    num_new = np.asarray(num_new, np.int64)
    past_len = np.asarray(past_len, np.int64)
    T = int(num_new.sum())
    page_T = np.zeros(len(prefix_len), np.int64)
    np.add.at(page_T, np.asarray(branch_page), num_new)
    q_bytes = T * Hq * D * s_in
    o_bytes = T * Hq * D * s_out
    shared_flop = int(4 * Hq * D * np.sum(page_T * prefix_len))
    shared_bytes = int(2 * prefix_len.sum() * Hkv * D * s_in + q_bytes + o_bytes)
    priv_keys = past_len + num_new
    private_bytes = int(2 * priv_keys.sum() * Hkv * D * s_in + q_bytes + o_bytes)
    vis = sum(int(k * (L + 1) + k * (k - 1) // 2) for k, L in zip(num_new, past_len))
    private_flop = int(4 * Hq * D * vis)
    return dict(T=T, shared_flop=shared_flop, shared_bytes=shared_bytes,
                private_flop=private_flop, private_bytes=private_bytes)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "gpus_requested": args.gpus}))
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(3)
    from paper_2607_18839_amd import _lib
    _lib.load()
    if args.workload == "c4":
        res = bench_decode(args, torch, _lib)
    else:
        res = bench_attention(args, torch, _lib)
    print(json.dumps(res))


def _time_steps(torch, step, K, W, stream):
    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(K):
        step(W + i)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / K


def _kernel_pass(torch, _lib, step, K, W):
    """Second pass of K steps with library-side per-kernel event timing."""
    _lib.hpd_kernel_timing(1, 200000)
    _lib.hpd_kernel_times_read()
    for i in range(K):
        step(W + i)
    torch.cuda.synchronize()
    t = _lib.hpd_kernel_times_read()
    _lib.hpd_kernel_timing(0)
    return {k: dict(launches=c, avg_us=(1000.0 * ms / c if c else None)) for k, (c, ms) in t.items()
            if not k.startswith("_") and c}


def _cpu_info():
    try:
        model = [l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name")][0]
    except Exception:
        model = "unknown"
    return model, len(os.sched_getaffinity(0))


def bench_attention(args, torch, _lib):
    from paper_2607_18839_amd.torch_api import BranchAttention
    from workloads import make_attn_batch
    b = make_attn_batch(args.workload, args.seed)
    tdt = torch.bfloat16 if b.dtype == "bf16" else torch.float32
    s_in = 2 if b.dtype == "bf16" else 4
    layer = BranchAttention(b.num_q_heads, b.num_kv_heads, b.prefix_len, b.branch_page, b.num_new,
                            b.past_len, dtype=tdt)

    def dev(a):
        if b.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()
    base = [dev(getattr(b, f)) for f in ("q", "shared_k", "shared_v", "priv_k", "priv_v")]
    per = sum(t.numel() * t.element_size() for t in base)
    reps = 1 if args.warm else max(1, int(np.ceil((1 << 30) / per)))
    replicas = [base] + [[t.clone() for t in base] for _ in range(reps - 1)]
    out = torch.empty((layer.T, b.num_q_heads, 64), dtype=tdt, device="cuda")
    stream = torch.cuda.current_stream()

    def step(i):
        q, sk, sv, pk, pv = replicas[i % reps]
        layer(q, sk, sv, pk, pv, out=out)

    ms = _time_steps(torch, step, args.steps, args.warmup, stream)
    kern = _kernel_pass(torch, _lib, step, args.steps, args.warmup)
    w = attn_work(b.prefix_len, b.branch_page, b.num_new, b.past_len, b.num_q_heads, b.num_kv_heads, 64,
                  s_in, s_in)
    peak_mfma = BF16_PEAK_TFLOPS if b.dtype == "bf16" else FP32_PEAK_TFLOPS
    sh = kern.get("shared_prefix", {}).get("avg_us")
    pr = kern.get("private", {}).get("avg_us")
    if sh:
        kern["shared_prefix"].update(flop=w["shared_flop"], tflops=w["shared_flop"] / sh / 1e6,
                                     mfma_frac=w["shared_flop"] / sh / 1e6 / peak_mfma)
    if pr:
        kern["private"].update(bytes=w["private_bytes"], gbs=w["private_bytes"] / pr / 1e3,
                               hbm_frac=w["private_bytes"] / pr / 1e3 / HBM_PEAK_GBS)
    roof = None
    if sh:
        ach = w["shared_flop"] / sh / 1e6
        roof = {"bound": "mfma", "kernel": "shared_prefix_kernel", "achieved": ach, "peak": peak_mfma,
                "unit": "TFLOP/s", "frac": ach / peak_mfma, "traffic": None,
                "algorithmic_per_launch": w["shared_flop"]}
    res = {
        "metric": "branch-tokens/s per decode step", "value": w["T"] / (ms / 1e3), "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": b.dtype, "data": "synthetic",
        "config": {"workload": f"{args.workload}: single attention layer", "pages": b.num_pages,
                   "branches": b.num_branches, "branch_tokens": w["T"],
                   "prefix_len_total": int(b.prefix_len.sum()),
                   "private_rows": int((b.past_len + b.num_new).sum()), "heads": [b.num_q_heads, b.num_kv_heads, 64],
                   "cache": "warm" if args.warm else f"cold ({reps} input replicas rotated)"},
        "roofline": roof, "kernels": kern,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_attention(b, args.cpu_seconds, w["T"])
    return res


def cpu_attention(b, budget_s, T):
    from oracle.attention import attention_for_batch
    model, ncpu = _cpu_info()
    times = []
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        attention_for_batch(b)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_start > budget_s or len(times) >= 50:
            break
    t = float(np.median(times))
    return {"value": T / t, "unit": "branch-tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{len(times)} full single-layer steps of the same batch, median {t:.3f} s "
                      f"(numpy einsum, single thread)",
            "cpu": model, "cpus_available": ncpu}


def bench_decode(args, torch, _lib):
    raise SystemExit("decode-step benchmark not built yet")


if __name__ == "__main__":
    main()

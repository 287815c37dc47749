"""Benchmark of the branch-parallel decode step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4|c3|c3f|c5|c2|c1|engine]

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
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--layers", type=int, default=None, help="c4 only: fewer layers (not for reporting)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--warm", action="store_true", help="attention workloads: reuse one input replica")
    ap.add_argument("--weights", choices=("packed", "torch"), default="packed",
                    help="c4: projection weights packed once at load (HPD_WEIGHTS_PACKED) or in torch layout")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--pmtp", action="store_true",
                    help="c4: each step also runs P-MTP verification and drafting (LM head, 151,936-token vocab)")
    ap.add_argument("--paged", type=int, default=0, metavar="BLOCK_ROWS",
                    help="K/V through block tables of this many rows (hpd_kv_pool, fragmented pool); 0 = contiguous")
    ap.add_argument("--no-box-peaks", action="store_true",
                    help="skip the microbenchmark of this GPU's own peaks (the second roofline denominator)")
    return ap.parse_args()


def box_peaks():
    """This GPU's own peaks from the `peaks` microbenchmark (streaming read
    GB/s, dense bf16 MFMA TFLOP/s), run as a child process before this
    process touches the GPU; None if it is not built or fails."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2607_18839_amd", "peaks")
    if not os.path.exists(exe):
        return None
    try:
        r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=180)
        if r.returncode != 0:
            return None
        p = json.loads(r.stdout.strip().splitlines()[-1])
    except (OSError, ValueError, IndexError, subprocess.TimeoutExpired):
        return None
    return {"read_gbs": p.get("read_gbs"), "copy_gbs": p.get("copy_gbs"),
            "mfma_bf16_tflops": max(p.get("mfma_bf16_tflops") or 0.0, p.get("mfma32_bf16_tflops") or 0.0),
            "empty_kernel_graph_us": p.get("empty_kernel_graph_us"),
            "source": "paper_2607_18839_amd/peaks on this GPU (streaming read over 1 GiB; 16x16x32 and "
                      "32x32x16 bf16 MFMA loops), measured in this run"}


def add_box_peak(roof, peaks):
    """The roofline's second denominator: the same achieved rate over this
    GPU's own measured peak."""
    if roof is None:
        return roof
    bp = None
    if peaks:
        # the microbenchmark measures bf16 MFMA and HBM reads only: a kernel
        # priced against another peak (fp32) has no box denominator
        if roof["unit"] == "GB/s":
            bp = peaks.get("read_gbs")
        elif roof["unit"] == "TFLOP/s" and roof.get("peak") == BF16_PEAK_TFLOPS:
            bp = peaks.get("mfma_bf16_tflops")
    roof["box_peak"] = bp
    roof["box_frac"] = roof["achieved"] / bp if bp and roof.get("achieved") else None
    return roof


# ----------------------------------------------------------------- algorithmic work

def attn_work(prefix_len, branch_page, num_new, past_len, Hq, Hkv, D, s_in, s_out, fork_len=None):
    """Algorithmic FLOPs / bytes of the shared and private phases (method's
    definition: what must be read and computed, not implementation scratch).
    With fork offsets a branch's tokens meet only its F_b visible prefix keys."""
    prefix_len = np.asarray(prefix_len, np.int64)
    num_new = np.asarray(num_new, np.int64)
    past_len = np.asarray(past_len, np.int64)
    T = int(num_new.sum())
    q_bytes = T * Hq * D * s_in
    o_bytes = T * Hq * D * s_out
    F = prefix_len[np.asarray(branch_page)] if fork_len is None else np.asarray(fork_len, np.int64)
    shared_flop = int(4 * Hq * D * np.sum(num_new * F))
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
    peaks = None if args.no_box_peaks else box_peaks()   # before this process initialises the GPU
    import torch
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(3)
    from paper_2607_18839_amd import _lib
    _lib.load()
    if args.workload in ("c4", "c4q"):
        res = bench_decode(args, torch, _lib)
    elif args.workload == "engine":
        res = bench_engine(args, torch, _lib)
    else:
        res = bench_attention(args, torch, _lib)
    if isinstance(res, dict) and "roofline" in res:
        res["roofline"] = add_box_peak(res["roofline"], peaks)
        res["box_peaks"] = peaks
    print(json.dumps(res))


def _graph_time(torch, step, n_inputs, K, W, per_graph=1):
    """Captures HIP graphs (torch's CUDAGraph on ROCm) of per_graph
    consecutive steps each, step j running step(j % n_inputs), so that the
    graphs together cover every input (max(1, n_inputs // per_graph) graphs).
    Replays them round-robin for the W warm-up steps untimed, then times
    exactly K steps (K / per_graph replays; per_graph divides K) with an event
    after each replay.  Several steps per graph keep the GPU busy when one
    step is shorter than the host's cost of a replay.  Returns (mean ms per
    step, K, {p10, p50, p90} of the per-replay times / per_graph in ms)."""
    assert K % per_graph == 0
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):           # eager warm-up outside capture
        for i in range(n_inputs):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graphs = []
    for i in range(max(1, n_inputs // per_graph)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for j in range(per_graph):
                step((i * per_graph + j) % n_inputs)
        graphs.append(g)
    for w in range(max(1, -(-W // per_graph))):
        graphs[w % len(graphs)].replay()
    n = K // per_graph
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(n):
        graphs[i % len(graphs)].replay()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(n)]) / per_graph
    pct = {f"p{q}": float(np.percentile(per, q)) for q in (10, 50, 90)}
    return ev[0].elapsed_time(ev[n]) / K, K, pct


def _steps_per_graph(K):
    """Steps per graph for the single-layer workloads: the largest of 8, 5,
    4, 2, 1 that divides K."""
    return next(g for g in (8, 5, 4, 2, 1) if K % g == 0)


def _kernel_pass(torch, _lib, step, K, W, queue_cycles=20_000_000):
    """Per-kernel durations from the HIP events the library binds to each of
    its launches (start and end of the kernel's execution).  Every step is
    first queued behind a bounded spin kernel (torch.cuda._sleep), so its
    launches run back to back on the GPU as in the timed region."""
    _lib.hpd_kernel_timing(1, 200000)
    _lib.hpd_kernel_times_read()
    tot = {}
    for i in range(K):
        torch.cuda._sleep(queue_cycles)
        step(W + i)
        torch.cuda.synchronize()
        for k, (c, ms) in _lib.hpd_kernel_times_read().items():
            a = tot.setdefault(k, [0, 0.0])
            a[0] += c
            a[1] += ms
    _lib.hpd_kernel_timing(0)
    return {k: dict(launches=c, avg_us=(1000.0 * ms / c if c else None)) for k, (c, ms) in tot.items()
            if not k.startswith("_") and c}


def _phase_pass(torch, _lib, step, K, W, work, queue_cycles=2_000_000, measured=False, workload="c4"):
    """Per-kernel durations with the attention phases in launches of their own
    (hpd_attn_phase_isolation): the shared-prefix items alone (MFMA-bound) and
    the private items alone (HBM-bound), next to the co-scheduled launch.
    measured: also the rocprofv3-measured HBM bytes of each phase launch
    (profiles/traffic_<workload>.md) and the rate they give."""
    _lib.hpd_attn_phase_isolation(True)
    try:
        kern = _kernel_pass(torch, _lib, step, K, W, queue_cycles)
    finally:
        _lib.hpd_attn_phase_isolation(False)
    out = {}
    sh, pr = kern.get("shared_prefix", {}).get("avg_us"), kern.get("private", {}).get("avg_us")
    if sh:
        out["shared_only_us"] = sh
        out["shared_mfma_frac"] = work["shared_flop"] / sh / 1e6 / BF16_PEAK_TFLOPS
    if pr:
        out["private_us"] = pr
        out["private_algorithmic_bytes"] = work["private_bytes"]
        out["private_gbs"] = work["private_bytes"] / pr / 1e3
        out["private_hbm_frac"] = work["private_bytes"] / pr / 1e3 / HBM_PEAK_GBS
    if measured:
        for phase, us in (("shared_phase", sh), ("private_phase", pr)):
            tb = _traffic(phase, workload)
            if us and tb:
                out[phase + "_measured_bytes"] = tb
                out[phase + "_measured_gbs"] = tb / us / 1e3
    return out


def _paged_layout(_lib, st, block_rows, seed):
    """Block tables for a batch from an hpd_kv_pool whose free list was first
    fragmented (short sequences reserved, then released in random order), and
    the pool row of every packed shared / private row."""
    rng = np.random.default_rng(seed + 1000)
    B = block_rows
    nblk = lambda n: -(-int(n) // B)
    need = sum(nblk(P) for P in st["prefix_len"]) + sum(nblk(L + k) for L, k in zip(st["past_len"], st["num_new"]))
    pool = _lib.KvPool(need + 64, B)
    junk = []
    for _ in range(32):
        j = pool.new()
        pool.reserve(j, int(rng.integers(1, 3)) * B)
        junk.append(j)
    for j in rng.permutation(len(junk)):
        pool.release(junk[int(j)])
    roots = []
    for P in st["prefix_len"]:
        r = pool.new()
        pool.reserve(r, int(P))
        roots.append(r)
    kids = []
    fork = st.get("fork_len")
    for i, p in enumerate(st["branch_page"]):
        k = pool.new(roots[int(p)], int(st["prefix_len"][int(p)]) if fork is None else int(fork[i]))
        pool.reserve(k, int(st["past_len"][i] + st["num_new"][i]))
        kids.append(k)
    pg = pool.batch_tables(roots, kids)
    blocks = np.asarray(pg["blocks"], np.int64)

    def rows(first, n):
        i = np.arange(int(n))
        return blocks[int(first) + i // B] * B + i % B
    sh = np.concatenate([rows(pg["page_block0"][p], P) for p, P in enumerate(st["prefix_len"])])
    pr = np.concatenate([rows(pg["branch_block0"][b], L + k)
                         for b, (L, k) in enumerate(zip(st["past_len"], st["num_new"]))])
    return pg, sh, pr, pg["num_blocks"] * B


def _to_pool(torch, t, rows, n_rows):
    """Device pool tensor holding packed row i of t at pool row rows[i]."""
    out = torch.zeros((n_rows,) + tuple(t.shape[1:]), dtype=t.dtype, device=t.device)
    out[torch.from_numpy(rows).to(t.device)] = t
    return out


def code_digest(path):
    """sha256 of a C++/HIP source with its comments, trailing blanks and empty
    lines removed: an edit of the comments alone leaves it unchanged."""
    import hashlib
    import re
    text = re.sub(r"/\*.*?\*/", "", open(path, encoding="utf-8").read(), flags=re.S)
    lines = [re.sub(r"//.*$", "", l).rstrip() for l in text.splitlines()]
    return hashlib.sha256("\n".join(l for l in lines if l).encode()).hexdigest()


def _traffic(kind, workload="c4"):
    """HBM bytes per launch of kernel kind from profiles/traffic_<workload>.md
    (rocprofv3 FETCH_SIZE / WRITE_SIZE runs scaled by a plain copy kernel's
    readings), or None when there is no such summary or the kernel's source
    code (comments aside) has changed since the counters were taken."""
    import re
    root = os.path.dirname(os.path.abspath(__file__))
    try:
        text = open(os.path.join(root, "profiles", f"traffic_{workload}.md")).read()
        block = json.loads(re.search(r"```json\n(.*?)```", text, re.S).group(1))
        k = block["kernels"][kind]
        src = os.path.join(root, "paper_2607_18839_amd", "csrc", k["source"])
        if code_digest(src) != block["code_sha256"][k["source"]]:
            return None
        return k["traffic_bytes"]
    except (OSError, KeyError, AttributeError, ValueError):
        return None


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
    st = dict(prefix_len=b.prefix_len, branch_page=b.branch_page, num_new=b.num_new, past_len=b.past_len,
              fork_len=b.fork_len)
    pg = _paged_layout(_lib, st, args.paged, args.seed) if args.paged else None
    layer = BranchAttention(b.num_q_heads, b.num_kv_heads, b.prefix_len, b.branch_page, b.num_new,
                            b.past_len, dtype=tdt, fork_len=b.fork_len, paged=pg and pg[0])

    def dev(a):
        if b.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()
    base = [dev(getattr(b, f)) for f in ("q", "shared_k", "shared_v", "priv_k", "priv_v")]
    if pg:
        _, sh_rows, pr_rows, n_pool = pg
        base = base[:1] + [_to_pool(torch, t, r, n_pool) for t, r in
                           zip(base[1:], (sh_rows, sh_rows, pr_rows, pr_rows))]
    per = sum(t.numel() * t.element_size() for t in base)
    reps = 1 if args.warm else max(1, int(np.ceil((1 << 30) / per)))
    replicas = [base] + [[t.clone() for t in base] for _ in range(reps - 1)]
    out = torch.empty((layer.T, b.num_q_heads, 64), dtype=tdt, device="cuda")
    stream = torch.cuda.current_stream()

    def step(i):
        q, sk, sv, pk, pv = replicas[i % reps]
        layer(q, sk, sv, pk, pv, out=out)

    per_graph = _steps_per_graph(args.steps)
    ms, timed, pct = _graph_time(torch, step, reps, args.steps, args.warmup, per_graph)
    kern = _kernel_pass(torch, _lib, step, min(args.steps, 20), args.warmup, queue_cycles=2_000_000)
    w = attn_work(b.prefix_len, b.branch_page, b.num_new, b.past_len, b.num_q_heads, b.num_kv_heads, 64,
                  s_in, s_in, b.fork_len)
    peak_mfma = BF16_PEAK_TFLOPS if b.dtype == "bf16" else FP32_PEAK_TFLOPS
    sh = kern.get("shared_prefix", {}).get("avg_us")
    pr = kern.get("private", {}).get("avg_us")
    # bf16: one launch runs the shared-prefix and the private work items
    sh_flop = w["shared_flop"] + (0 if pr else w["private_flop"])
    if sh:
        kern["shared_prefix"].update(flop=sh_flop, tflops=sh_flop / sh / 1e6,
                                     mfma_frac=sh_flop / sh / 1e6 / peak_mfma,
                                     includes_private=not pr)
    if pr:
        kern["private"].update(bytes=w["private_bytes"], gbs=w["private_bytes"] / pr / 1e3,
                               hbm_frac=w["private_bytes"] / pr / 1e3 / HBM_PEAK_GBS)
    if b.dtype == "bf16":
        kern["phases_isolated"] = _phase_pass(torch, _lib, step, min(args.steps, 20), args.warmup, w,
                                              measured=not args.paged, workload=args.workload)
    roof = None
    if sh:
        ach = sh_flop / sh / 1e6
        roof = {"bound": "mfma", "kernel": "shared_prefix", "achieved": ach, "peak": peak_mfma,
                "unit": "TFLOP/s", "frac": ach / peak_mfma,
                "traffic": None if args.paged else _traffic("shared_prefix", args.workload),
                "algorithmic_per_launch": sh_flop}
    res = {
        "metric": "branch-tokens/s per decode step", "value": w["T"] / (ms / 1e3), "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": timed, "warmup": args.warmup, "ms_per_step": ms, "latency_ms": pct,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": b.dtype, "data": "synthetic", "timing": f"HIP graph replay ({per_graph} steps per graph, each on its own input replica)",
        "config": {"workload": f"{args.workload}: single attention layer", "pages": b.num_pages,
                   "branches": b.num_branches, "branch_tokens": w["T"],
                   "prefix_len_total": int(b.prefix_len.sum()),
                   "private_rows": int((b.past_len + b.num_new).sum()), "heads": [b.num_q_heads, b.num_kv_heads, 64],
                   "fork_offsets": None if b.fork_len is None else
                   {"visible_prefix_keys": int(np.asarray(b.fork_len, np.int64).sum()),
                    "rule": "layout branch whole prefix; content branches uniform in [1024, P]"},
                   "cache": "warm" if args.warm else f"cold ({reps} input replicas rotated)",
                   "kv": f"paged ({args.paged}-row blocks, fragmented pool)" if args.paged else "contiguous"},
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
        # median of at least 3 runs, or 1 run when a run exceeds 10 s
        if times[-1] > 10.0 or len(times) >= 50 or (len(times) >= 3 and time.perf_counter() - t_start > budget_s):
            break
    t = float(np.median(times))
    return {"value": T / t, "unit": "branch-tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{len(times)} full single-layer steps of the same batch, median {t:.3f} s "
                      f"(numpy einsum, single thread; median of >= 3 runs, or 1 run when a run exceeds 10 s)",
            "cpu": model, "cpus_available": ncpu}


def gemm_work(T, Hq, Hkv, D, H, I):
    """Algorithmic bytes of one launch of each projection kernel: weights once,
    activations in and outputs out for the T real token rows."""
    nq, nkv = Hq * D, Hkv * D
    return {
        "gemm_qkv": (nq + 2 * nkv) * H * 2 + T * H * 2 + T * (nq + 2 * nkv) * 2,
        "gemm_o": H * nq * 2 + T * nq * 2 + 2 * T * H * 4,
        "gemm_gate_up": 2 * I * H * 2 + 2 * T * H * 2 + 2 * T * I * 2,
        "gemm_down": H * I * 2 + 2 * T * I * 2 + 2 * T * H * 4,
        "norm": T * H * 4 + 2 * T * H * 2,
    }


def bench_decode(args, torch, _lib):
    from paper_2607_18839_amd.torch_api import DecodeStep
    from workloads import make_decode_inputs
    inp = make_decode_inputs(args.workload, args.seed, num_layers=args.layers)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    w = {k: [dev(a) for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    for k in ("q_norm", "k_norm"):   # c4q: Qwen3-style head gains
        if getattr(inp, k, None) is not None:
            w[k] = [dev(a) for a in getattr(inp, k)]
    sk = [dev(a) for a in inp.shared_k]
    sv = [dev(a) for a in inp.shared_v]
    pk = [dev(a) for a in inp.priv_k]
    pv = [dev(a) for a in inp.priv_v]
    st = dict(prefix_len=inp.prefix_len, branch_page=inp.branch_page, num_new=inp.num_new, past_len=inp.past_len)
    pg = _paged_layout(_lib, st, args.paged, args.seed) if args.paged else None
    if pg:
        _, sh_rows, pr_rows, n_pool = pg
        sk, sv = [_to_pool(torch, t, sh_rows, n_pool) for t in sk], [_to_pool(torch, t, sh_rows, n_pool) for t in sv]
        pk, pv = [_to_pool(torch, t, pr_rows, n_pool) for t in pk], [_to_pool(torch, t, pr_rows, n_pool) for t in pv]
    step_obj = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                          inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps,
                          packed=args.weights == "packed", paged=pg and pg[0], rope_theta=inp.rope_theta)
    del w   # the packed copies are held by step_obj; the torch-layout tensors are not read again
    h_in = torch.from_numpy(inp.hidden_in).cuda()
    h_out = torch.empty_like(h_in)
    stream = torch.cuda.current_stream()
    vd = None
    if args.pmtp:
        from paper_2607_18839_amd.torch_api import VerifyDraft
        from workloads import get_config, make_pmtp_inputs
        c = get_config("c4")["pmtp"]
        pm = make_pmtp_inputs(inp.hidden, c["vocab"], c["draft_inner"], c["weight_std"], args.seed)
        vd = VerifyDraft(step_obj, {k: dev(getattr(pm, k)) for k in ("lm_head", "embed", "w_draft_gate",
                                                                     "w_draft_up", "w_draft_down")})
        pm_host = pm if not args.no_cpu_baseline else None   # the oracle's copy for the CPU leg
        del pm
        tokens_in = torch.from_numpy(np.random.default_rng(args.seed).integers(0, c["vocab"], size=step_obj.T)
                                     .astype(np.int32)).cuda()
        nbr = len(inp.num_new)
        ver = torch.empty(step_obj.T, dtype=torch.int32, device="cuda")
        nacc = torch.empty(nbr, dtype=torch.int32, device="cuda")
        drafts = torch.empty((nbr, _lib.HPD_MAX_K), dtype=torch.int32, device="cuda")

    def step(i):
        step_obj(h_in, sk, sv, pk, pv, hidden_out=h_out)
        if vd is not None:
            vd(h_out, tokens_in, ver, nacc, drafts)

    ms, timed, pct = _graph_time(torch, step, 1, args.steps, args.warmup)
    kern = _kernel_pass(torch, _lib, step, min(args.steps, 10), args.warmup)
    T, Hq, Hkv, D, H, I = step_obj.T, inp.num_q_heads, inp.num_kv_heads, 64, inp.hidden, inp.intermediate
    aw = attn_work(inp.prefix_len, inp.branch_page, inp.num_new, inp.past_len, Hq, Hkv, D, 2, 2)
    gw = gemm_work(T, Hq, Hkv, D, H, I)
    for name, k in kern.items():
        us = k["avg_us"]
        if name == "shared_prefix":   # bf16: also runs the private work items
            fl = aw["shared_flop"] + (0 if "private" in kern else aw["private_flop"])
            k.update(bound="mfma", flop=fl, tflops=fl / us / 1e6, frac=fl / us / 1e6 / BF16_PEAK_TFLOPS,
                     includes_private="private" not in kern)
        elif name == "private":
            k.update(bound="hbm", bytes=aw["private_bytes"], gbs=aw["private_bytes"] / us / 1e3,
                     frac=aw["private_bytes"] / us / 1e3 / HBM_PEAK_GBS)
        elif name in gw:
            k.update(bound="hbm", bytes=gw[name], gbs=gw[name] / us / 1e3, frac=gw[name] / us / 1e3 / HBM_PEAK_GBS)
        elif name == "lm_head" and vd is not None:   # the LM head's weights once per launch
            lb = vd.vocab * H * 2
            k.update(bound="hbm", bytes=lb, gbs=lb / us / 1e3, frac=lb / us / 1e3 / HBM_PEAK_GBS)
        k["total_us_per_step"] = us * k["launches"] / min(args.steps, 10)
    dom = max(kern, key=lambda n: kern[n]["total_us_per_step"])
    kern["phases_isolated"] = _phase_pass(torch, _lib, step, min(args.steps, 10), args.warmup, aw,
                                          measured=args.workload == "c4" and not args.paged)
    d = kern[dom]
    # the measured bytes belong to the c4 step with packed weights and contiguous K/V
    tr = _traffic(dom) if args.workload == "c4" and not args.paged and args.weights == "packed" else None
    if d.get("bound") == "mfma":
        roof = {"bound": "mfma", "kernel": dom, "achieved": d["tflops"], "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": d["frac"], "traffic": tr, "algorithmic_per_launch": d["flop"]}
    else:
        roof = {"bound": "hbm", "kernel": dom, "achieved": d.get("gbs"), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": d.get("frac"), "traffic": tr, "algorithmic_per_launch": d.get("bytes")}
    res = {
        "metric": "branch-tokens/s per decode step", "value": T / (ms / 1e3), "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": timed, "warmup": args.warmup, "ms_per_step": ms, "latency_ms": pct,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "timing": "HIP graph replay (one step per graph)",
        "data": "synthetic (seeded N(0,1) KV and hidden, N(0,0.02) bf16 weights)",
        "config": {"workload": f"{args.workload}: full decode step, 18-layer synthetic decoder, 1 page, "
                               "1 layout (k=1) + 32 content (k=4) branches, 4096-token shared prefix"
                               + (", Qwen3-style per-head QK norm and rotary embedding (base 1e6)"
                                  if args.workload == "c4q" else ""),
                   "layers": inp.num_layers, "hidden": H, "intermediate": I, "heads": [Hq, Hkv, D],
                   "branch_tokens": T, "branches": int(len(inp.num_new)), "prefix_len": int(inp.prefix_len[0]),
                   "private_rows": int((inp.past_len + inp.num_new).sum()),
                   "weights": args.weights + (" (packed once before timing)" if args.weights == "packed" else ""),
                   "kv": f"paged ({args.paged}-row blocks, fragmented pool)" if args.paged else "contiguous",
                   "pmtp": None if vd is None else
                   {"vocab": vd.vocab, "draft_inner": vd.draft_inner,
                    "per_step": "verification of all T positions + drafting of each branch's next window"}},
        "roofline": roof, "kernels": kern,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_decode(inp, args.cpu_seconds, T)
        if vd is not None:
            cpu_pmtp(res["cpu_baseline"], inp, pm_host, tokens_in.cpu().numpy(), T)
    return res


def cpu_decode(inp, budget_s, T):
    """The fp64 oracle on the first n layers of the same step (n sized to the
    time budget), scaled to a whole step."""
    from oracle.decode import decode_step
    model, ncpu = _cpu_info()
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = ncpu
    t0 = time.perf_counter()
    decode_step(inp, num_layers=1)
    t1 = time.perf_counter() - t0
    n = int(max(1, min(inp.num_layers, budget_s // max(t1, 1e-3))))
    runs = []
    for _ in range(3):   # median of 3 runs, or 1 run when a run takes more than 10 s
        t0 = time.perf_counter()
        decode_step(inp, num_layers=n)
        runs.append(time.perf_counter() - t0)
        if runs[-1] > 10.0:
            break
    t = float(np.median(runs)) * inp.num_layers / n
    return {"value": T / t, "unit": "branch-tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"first {n} of {inp.num_layers} layers of the same step (fp64 numpy, BLAS matmuls), "
                      f"scaled to the full step: {t:.2f} s/step ({len(runs)} run(s), median; "
                      "median of 3, or 1 run when a run exceeds 10 s)",
            "cpu": model, "cpus_available": ncpu, "single_thread_c3": cpu_c3_single_thread()}


def cpu_c3_single_thread():
    """The attention oracle on the c3 layer (seed 0) once with one BLAS
    thread: the single-core reference of the oracle timing."""
    from oracle.attention import attention_for_batch
    from workloads import make_attn_batch
    b = make_attn_batch("c3", 0)
    try:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(1)
    except Exception:
        limit = None
    try:
        t0 = time.perf_counter()
        attention_for_batch(b)
        t = time.perf_counter() - t0
    finally:
        if limit is not None:
            limit.restore_original_limits()
    T = int(b.num_new.sum())
    return {"seconds": t, "value": T / t, "unit": "branch-tokens/s", "threads": 1,
            "sample": "one full c3 attention layer (seed 0), fp64 numpy"}


def bench_engine(args, torch, _lib):
    """The continuous-batching loop (host scheduler -> embedding lookup ->
    paged decode step -> P-MTP verification and drafting -> commit) on the
    c4 decoder with the 151,936-token LM head, over a closed-loop stream of
    16 pages in flight (a finished page is replaced by a new one; prompt
    U[1024, 4096] rows) whose layout branches fork U{4..32} content
    branches each (fork tokens planted at the bonus token, each step with
    probability 1/2, until the page has its count); every request records
    at most 64 tokens.  Prefill rows are a synthetic fill.  Timed: K
    iterations after W, each ending with the host reading the verified
    tokens (the scheduler needs them)."""
    from paper_2607_18839_amd.engine import Engine
    from workloads import get_config, make_decode_inputs, make_pmtp_inputs
    inp = make_decode_inputs("c4", args.seed, num_layers=args.layers)
    c = get_config("c4")["pmtp"]
    pm = make_pmtp_inputs(inp.hidden, c["vocab"], c["draft_inner"], c["weight_std"], args.seed)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    w = {k: [dev(a) for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    pw = {k: dev(getattr(pm, k)) for k in ("lm_head", "embed", "w_draft_gate", "w_draft_up", "w_draft_down")}
    FORK, CHILD, EOS = c["vocab"] - 3, c["vocab"] - 2, c["vocab"] - 1
    cfg = dict(num_blocks=4096, block_rows=64, kv_threshold=0.9, window=4, max_active=64, fork_token=FORK,
               child_token=CHILD, eos_token=EOS)
    eng = Engine(w, pw, inp.hidden, inp.intermediate, inp.num_q_heads, inp.num_kv_heads, cfg, rms_eps=inp.rms_eps)
    del w, pw
    rng = np.random.default_rng([args.seed, 11])
    want_children, spawned = {}, {}

    def new_page():
        pid = eng.submit(int(rng.integers(1024, 4097)), int(rng.integers(0, c["vocab"] - 3)), 64)
        want_children[pid], spawned[pid] = int(rng.integers(4, 33)), 0

    for _ in range(16):
        new_page()

    def plant(batch):
        q = 0
        for b, k in enumerate(batch["num_new"]):
            r = int(batch["request"][b])
            if batch["fork_len"][b] == 0 and spawned.get(r, 0) < want_children.get(r, 0) and rng.random() < 0.5:
                batch["verified"][q + batch["n_acc"][b]] = FORK
                batch["draft_out"][b, 0] = FORK
                spawned[r] += 1
            q += k

    eng.on_results = plant

    def step():   # one iteration; a finished page is replaced by a new one (16 pages in flight)
        b = eng.step()
        for _ in eng.outputs():
            new_page()
        return b

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    eng.host_s = {k: 0.0 for k in eng.host_s}
    tokens = branches = emitted = idle = pages_done = 0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        n0 = len(want_children)
        b = step()
        pages_done += len(want_children) - n0
        if b["num_branches"] == 0:
            idle += 1
            continue
        tokens += b["num_tokens"]
        branches += b["num_branches"]
        emitted += int(np.sum(b["n_acc"]) + b["num_branches"])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    K = args.steps
    cnt = eng.sched.counts()
    return {
        "metric": "branch-tokens/s per decode step", "value": tokens / wall, "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": wall / K * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "timing": "wall clock of K engine iterations (host scheduling, plan, upload, GPU step, result read-back)",
        "data": "synthetic (seeded N(0,0.02) bf16 weights; prefill rows a seeded N(0,1) fill; planted fork tokens)",
        "config": {"workload": "engine: Algorithm 1 continuous batching, c4 decoder (18 layers) + P-MTP "
                               "(151,936-token vocab, window 4), 16 pages in flight, prompt U[1024, 4096], "
                               "U{4..32} forks per page, <= 64 tokens per request",
                   "sched": {k: v for k, v in cfg.items() if not k.endswith("token")}},
        "engine": {"mean_tokens_per_step": tokens / max(K - idle, 1),
                   "mean_branches_per_step": branches / max(K - idle, 1), "idle_steps": idle,
                   "emitted_tokens_per_s": emitted / wall,
                   "host_ms_per_step": {k: v / K * 1e3 for k, v in eng.host_s.items()},
                   "after": cnt, "children_spawned": int(sum(spawned.values())), "pages_finished": pages_done},
    }


def cpu_pmtp(cpu, inp, pm, tokens_in, T):
    """Adds the oracle's verification and drafting of one step (fp64 LM head
    over every position, then k - 1 draft advances per branch) to the
    decode-step baseline.  The step's input hidden state stands in for its
    output (same shape; the oracle's cost does not depend on the values)."""
    from oracle.pmtp import draft, verify
    f = lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    W_lm, E = f(pm.lm_head), f(pm.embed)
    Wg, Wu, Wd = f(pm.w_draft_gate), f(pm.w_draft_up), f(pm.w_draft_down)
    t0 = time.perf_counter()
    ver, n_acc, bonus, seed_row, _ = verify(inp.hidden_in, tokens_in, inp.num_new, None, W_lm)
    draft(np.asarray(inp.hidden_in, np.float64)[seed_row], bonus, int(max(inp.num_new)) - 1, E, Wg, Wu, Wd,
          None, W_lm, inp.rms_eps)
    tp = time.perf_counter() - t0
    t_step = T / cpu["value"] + tp
    cpu["value"] = T / t_step
    cpu["sample"] += f"; plus the oracle's P-MTP verification and drafting of the whole step ({tp:.2f} s)"
    return cpu


if __name__ == "__main__":
    main()

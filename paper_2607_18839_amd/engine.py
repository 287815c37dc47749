"""Continuous batching over the library's entry points (section "Inference
Workflow", Algorithm 1): the host scheduler (hpd_sched_*) picks each step's
batch of pages and branches, the embedding lookup, the decode step and the
P-MTP verification / drafting run on it with the batch's paged block tables,
and the verified tokens go back to the scheduler.

Argument marshalling only: torch allocates the device buffers (K/V pools,
workspace, token and hidden-state buffers); every step runs in the library.
The rows a batch asks to prefill (a new page's prompt, a preempted request's
dropped rows) are the caller's: the prefill is not part of the decode step,
and `prefill` is called with the engine and the batch before the step.
"""
import time

import numpy as np
import torch

from . import _lib
from .torch_api import _stream, pack_gate_up, pack_weight


def pool_rows(batch, b, lo, hi):
    """Pool rows of rows lo..hi-1 of branch b's own sequence (a parent: its
    page's rows)."""
    pg = batch["paged"]
    B = pg["block_rows"]
    r = np.arange(lo, hi, dtype=np.int64)
    return pg["blocks"][pg["branch_block0"][b] + r // B].astype(np.int64) * B + r % B


def synthetic_prefill(seed=0):
    """A prefill stand-in: writes seeded N(0, 1) bf16 K/V into the rows the
    batch asks for (a new page's prompt rows, a resumed request's dropped
    rows).  The values stand in for what a prefill would compute; they do
    not reproduce the rows a request had before it was preempted."""
    def fill(engine, batch):
        for b in range(batch["num_branches"]):
            lo, hi = int(batch["prefill_from"][b]), int(batch["prefill_to"][b])
            if hi <= lo:
                continue
            rows = torch.from_numpy(pool_rows(batch, b, lo, hi)).to(engine.device)
            g = torch.Generator(device=engine.device).manual_seed(seed * 1_000_003 + int(batch["request"][b]) * 65_537
                                                                  + lo)
            shape = (2, engine.num_layers, hi - lo, engine.num_kv_heads, _lib.HPD_HEAD_DIM)
            vals = torch.randn(shape, generator=g, device=engine.device).to(torch.bfloat16)
            for l in range(engine.num_layers):
                engine.k_pool[l].index_copy_(0, rows, vals[0, l])
                engine.v_pool[l].index_copy_(0, rows, vals[1, l])
    return fill


class Engine:
    """One GPU's continuous-batching loop.

    ``weights``: per-layer lists of bf16 device tensors in torch Linear layout
    ('w_qkv', 'w_o', 'w_gate', 'w_up', 'w_down'); ``pmtp``: 'lm_head',
    'embed', 'w_draft_gate', 'w_draft_up', 'w_draft_down' (bf16 device).
    ``sched``: hpd_sched_config fields as keywords (num_blocks, block_rows,
    kv_threshold, window, max_active, fork_token, child_token, eos_token).
    """

    def __init__(self, weights, pmtp, hidden, intermediate, num_q_heads, num_kv_heads, sched, rms_eps=1e-6,
                 prefill=None, device="cuda", stream=None):
        self.device = torch.device(device)
        self.hidden, self.num_q_heads, self.num_kv_heads = hidden, num_q_heads, num_kv_heads
        self.num_layers = len(weights["w_qkv"])
        self.window = int(sched["window"])
        self.prefill = prefill or synthetic_prefill()
        self._w = dict(w_qkv=[pack_weight(w, stream) for w in weights["w_qkv"]],
                       w_o=[pack_weight(w, stream) for w in weights["w_o"]],
                       w_gate=[pack_gate_up(g, u, stream) for g, u in zip(weights["w_gate"], weights["w_up"])],
                       w_down=[pack_weight(w, stream, f16=True) for w in weights["w_down"]])
        ptr = {k: [t.data_ptr() for t in v] for k, v in self._w.items()}
        self.model = _lib.model_desc(self.num_layers, hidden, intermediate, rms_eps, ptr["w_qkv"], ptr["w_o"],
                                     ptr["w_gate"], ptr["w_gate"], ptr["w_down"],
                                     weight_format=_lib.HPD_WEIGHTS_PACKED)
        self.vocab = pmtp["lm_head"].shape[0]
        self._p = dict(lm_head=pack_weight(pmtp["lm_head"], stream),
                       gate_up=pack_gate_up(pmtp["w_draft_gate"], pmtp["w_draft_up"], stream),
                       down=pack_weight(pmtp["w_draft_down"], stream, f16=True),
                       embed=pmtp["embed"].contiguous())
        self.pmtp = _lib.hpd_pmtp_desc(self.vocab, pmtp["w_draft_gate"].shape[0], self._p["lm_head"].data_ptr(),
                                       None, self._p["embed"].data_ptr(), self._p["gate_up"].data_ptr(),
                                       self._p["down"].data_ptr(), self.window)
        self.sched = _lib.Sched(sched["num_blocks"], sched["block_rows"], sched["kv_threshold"], self.window,
                                sched["max_active"], sched["fork_token"], sched["child_token"], sched["eos_token"])
        rows = sched["num_blocks"] * sched["block_rows"]
        shape = (rows, num_kv_heads, _lib.HPD_HEAD_DIM)
        self.k_pool = [torch.zeros(shape, dtype=torch.bfloat16, device=self.device) for _ in range(self.num_layers)]
        self.v_pool = [torch.zeros(shape, dtype=torch.bfloat16, device=self.device) for _ in range(self.num_layers)]
        self._kp = [t.data_ptr() for t in self.k_pool]
        self._vp = [t.data_ptr() for t in self.v_pool]
        self.workspace = torch.empty(0, dtype=torch.uint8, device=self.device)
        self._buf = {}
        # host seconds per phase: the scheduler, planning and upload, enqueueing
        # the step's launches (embedding, decode step, verification), the commit
        self.host_s = dict(schedule=0.0, plan=0.0, enqueue=0.0, commit=0.0)
        self.steps = 0
        self.on_results = None   # optional hook(batch, verified, n_acc, draft_out) before the commit

    def submit(self, prompt_len, first_token, max_new):
        return self.sched.submit(prompt_len, first_token, max_new)

    def _buffer(self, name, n, dtype):
        t = self._buf.get(name)
        if t is None or t.numel() < n:
            t = torch.empty(max(n, 1) * 2, dtype=dtype, device=self.device)
            self._buf[name] = t
        return t[:n]

    def step(self):
        """One iteration on torch's current stream (the prefill, the library
        launches and the read-back of the results share it); returns the
        batch with the step's results (host arrays under 'verified', 'n_acc',
        'draft_out', 'hidden_out'), or the empty batch when nothing was
        active."""
        t0 = time.perf_counter()
        batch = self.sched.schedule()
        t1 = time.perf_counter()
        self.host_s["schedule"] += t1 - t0
        nb, T = batch["num_branches"], batch["num_tokens"]
        if nb == 0:
            self.sched.commit(None, None, None)
            return batch
        self.prefill(self, batch)
        t2 = time.perf_counter()
        plan = _lib.hpd_plan_create(self.num_q_heads, self.num_kv_heads, batch["prefix_len"], batch["branch_page"],
                                    batch["num_new"], batch["past_len"], fork_len=batch["fork_len"],
                                    paged=batch["paged"])
        need = (plan.workspace_bytes + _lib.hpd_decode_workspace_bytes(self.model, plan) +
                _lib.hpd_pmtp_workspace_bytes(self.model, self.pmtp, plan))
        if self.workspace.numel() < need:
            self.workspace = torch.empty(need * 3 // 2 + 4096, dtype=torch.uint8, device=self.device)
        ws, ws_bytes = self.workspace.data_ptr(), self.workspace.numel()
        s = _stream(None)
        _lib.hpd_plan_upload(plan, ws, ws_bytes, s)
        t_enq = time.perf_counter()
        self.host_s["plan"] += t_enq - t2
        tok = self._buffer("tokens", T, torch.int32)
        tok.copy_(torch.from_numpy(batch["tokens_in"].astype(np.int32)))
        h_in = self._buffer("h_in", T * self.hidden, torch.float32)
        h_out = self._buffer("h_out", T * self.hidden, torch.float32)
        # the three results share one buffer, read back with one copy
        res = self._buffer("results", T + nb + nb * _lib.HPD_MAX_K, torch.int32)
        ver, nacc, drafts = res[:T], res[T:T + nb], res[T + nb:]
        _lib.hpd_embed_tokens(self._p["embed"].data_ptr(), self.vocab, self.hidden, tok.data_ptr(), T,
                              h_in.data_ptr(), s)
        _lib.hpd_decode_step(self.model, plan, h_in.data_ptr(), h_out.data_ptr(), self._kp, self._vp, self._kp,
                             self._vp, ws, ws_bytes, s)
        _lib.hpd_verify_draft_step(self.model, self.pmtp, plan, h_out.data_ptr(), tok.data_ptr(), ver.data_ptr(),
                                   nacc.data_ptr(), drafts.data_ptr(), ws, ws_bytes, s)
        self.host_s["enqueue"] += time.perf_counter() - t_enq
        host = res.cpu().numpy()
        batch["verified"] = host[:T]
        batch["n_acc"] = host[T:T + nb]
        batch["draft_out"] = host[T + nb:].reshape(nb, _lib.HPD_MAX_K)
        batch["hidden_out"] = h_out
        batch["plan"] = plan
        if self.on_results is not None:
            self.on_results(batch)
        t3 = time.perf_counter()
        self.sched.commit(batch["verified"], batch["n_acc"], batch["draft_out"])
        self.host_s["commit"] += time.perf_counter() - t3
        self.steps += 1
        return batch

    def outputs(self):
        """Finished pages since the last call: [(page id, tokens)]."""
        out = []
        while (o := self.sched.next_output()) is not None:
            out.append(o)
        return out

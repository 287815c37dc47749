"""torch-facing wrappers: allocate device memory with torch, call the C ABI.

Nothing here computes any part of the step; it only sizes and allocates
buffers and passes pointers and the current HIP stream.
"""
import torch

from . import _lib

DT = {torch.bfloat16: _lib.HPD_BF16, torch.float32: _lib.HPD_F32}


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _p(t):
    return None if t is None else t.data_ptr()


class BranchAttention:
    """One attention layer of the branch-parallel step for a fixed batch shape.

    The plan (bookkeeping + work lists) is built once on the host and copied
    into a torch-allocated device workspace; each call launches the kernels.
    """

    def __init__(self, num_q_heads, num_kv_heads, prefix_len, branch_page, num_new, past_len,
                 dtype=torch.bfloat16, out_dtype=None, fork_len=None, prefix_row=None,
                 priv_row=None, softmax_scale=0.0, device="cuda", stream=None, paged=None):
        self.dtype = dtype
        self.out_dtype = dtype if out_dtype is None else out_dtype
        self.num_q_heads = num_q_heads
        self.plan = _lib.hpd_plan_create(num_q_heads, num_kv_heads, prefix_len, branch_page, num_new,
                                         past_len, softmax_scale=softmax_scale, dtype=DT[dtype],
                                         out_dtype=DT[self.out_dtype], prefix_row=prefix_row,
                                         priv_row=priv_row, fork_len=fork_len, paged=paged)
        self.info = _lib.hpd_plan_query(self.plan)
        self.T = self.info["T"]
        self.ws_bytes = self.plan.workspace_bytes
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)
        _lib.hpd_plan_upload(self.plan, self.workspace.data_ptr(), self.ws_bytes, _stream(stream))

    def __call__(self, q, shared_k, shared_v, priv_k, priv_v, out=None, lse=None, stream=None):
        if out is None:
            out = torch.empty((self.T, self.num_q_heads, _lib.HPD_HEAD_DIM), dtype=self.out_dtype,
                              device=q.device)
        for name, t in (("q", q), ("shared_k", shared_k), ("shared_v", shared_v), ("priv_k", priv_k),
                        ("priv_v", priv_v)):
            if t is not None and (t.dtype != self.dtype or not t.is_contiguous()):
                raise ValueError(f"{name} must be a contiguous {self.dtype} tensor")
        _lib.hpd_branch_attn_step(self.plan, _p(q), _p(shared_k), _p(shared_v), _p(priv_k), _p(priv_v),
                                  _p(out), _p(lse), self.workspace.data_ptr(), self.ws_bytes,
                                  _stream(stream))
        return out


def pack_weight(w, stream=None, f16=False):
    """Packed copy of a bf16 [rows][cols] device tensor: bf16
    (hpd_pack_weight) or converted to fp16 (hpd_pack_weight_f16)."""
    rows, cols = w.shape
    out = torch.empty(w.shape, dtype=torch.float16 if f16 else w.dtype, device=w.device)
    fn = _lib.hpd_pack_weight_f16 if f16 else _lib.hpd_pack_weight
    fn(w.data_ptr(), rows, cols, out.data_ptr(), _stream(stream))
    return out


def pack_gate_up(w_gate, w_up, stream=None):
    """Packed fp16 gate/up pair (hpd_pack_gate_up) of two bf16 [I][hidden] tensors."""
    inter, hidden = w_gate.shape
    out = torch.empty((2 * inter, hidden), dtype=torch.float16, device=w_gate.device)
    _lib.hpd_pack_gate_up(w_gate.data_ptr(), w_up.data_ptr(), inter, hidden, out.data_ptr(), _stream(stream))
    return out


class DecodeStep:
    """One decode step of the decoder stack for a fixed batch shape.

    ``weights`` maps 'w_qkv', 'w_o', 'w_gate', 'w_up', 'w_down' (and
    optionally 'g_attn_norm', 'g_mlp_norm', and the Qwen3-style 'q_norm',
    'k_norm' head gains) to lists of per-layer bf16 device tensors in torch
    Linear layout; ``rope_theta`` > 0 turns on the rotary embedding.  The tensors must stay alive while the
    step is used.  packed=True packs the projection weights once here
    (HPD_WEIGHTS_PACKED, a device copy of the weights) and the step reads
    the packed copies.
    """

    def __init__(self, num_q_heads, num_kv_heads, prefix_len, branch_page, num_new, past_len,
                 weights, hidden, intermediate, rms_eps=1e-6, prefix_row=None, priv_row=None,
                 device="cuda", stream=None, packed=False, fork_len=None, paged=None, rope_theta=0.0):
        self.attn = BranchAttention(num_q_heads, num_kv_heads, prefix_len, branch_page, num_new, past_len,
                                    dtype=torch.bfloat16, prefix_row=prefix_row, priv_row=priv_row,
                                    device=device, stream=stream, fork_len=fork_len, paged=paged)
        self.T = self.attn.T
        self.hidden = hidden
        self.num_layers = len(weights["w_qkv"])
        fmt = _lib.HPD_WEIGHTS_TORCH
        if packed:
            weights = dict(weights)
            weights["w_gate"] = [pack_gate_up(g, u, stream) for g, u in zip(weights["w_gate"], weights["w_up"])]
            weights["w_up"] = weights["w_gate"]   # ignored by the packed format
            for k in ("w_qkv", "w_o"):
                weights[k] = [pack_weight(w, stream) for w in weights[k]]
            weights["w_down"] = [pack_weight(w, stream, f16=True) for w in weights["w_down"]]
            fmt = _lib.HPD_WEIGHTS_PACKED
        self._weights = weights   # keeps packed copies alive
        ptrs = {k: [t.data_ptr() for t in v] for k, v in weights.items()}
        self.model = _lib.model_desc(self.num_layers, hidden, intermediate, rms_eps, ptrs["w_qkv"], ptrs["w_o"],
                                     ptrs["w_gate"], ptrs["w_up"], ptrs["w_down"], ptrs.get("g_attn_norm"),
                                     ptrs.get("g_mlp_norm"), weight_format=fmt, q_norm=ptrs.get("q_norm"),
                                     k_norm=ptrs.get("k_norm"), rope_theta=rope_theta)
        self.plan_bytes = self.attn.ws_bytes
        self.ws_bytes = self.plan_bytes + _lib.hpd_decode_workspace_bytes(self.model, self.attn.plan)
        # one workspace holding the plan tables (uploaded) and the step's scratch
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        _lib.hpd_plan_upload(self.attn.plan, self.workspace.data_ptr(), self.ws_bytes, _stream(stream))

    def __call__(self, hidden_in, shared_k, shared_v, priv_k, priv_v, hidden_out=None, stream=None):
        if hidden_out is None:
            hidden_out = torch.empty_like(hidden_in)
        if hidden_in.dtype != torch.float32 or hidden_in.shape != (self.T, self.hidden):
            raise ValueError("hidden_in must be float32 [T, hidden]")
        _lib.hpd_decode_step(self.model, self.attn.plan, hidden_in.data_ptr(), hidden_out.data_ptr(),
                             [t.data_ptr() for t in shared_k], [t.data_ptr() for t in shared_v],
                             [t.data_ptr() for t in priv_k], [t.data_ptr() for t in priv_v],
                             self.workspace.data_ptr(), self.ws_bytes, _stream(stream))
        return hidden_out


class VerifyDraft:
    """P-MTP verification and drafting after a decode step (hpd_verify_draft_step).

    ``pmtp`` maps 'lm_head' [V][hidden], 'embed' [V][hidden], 'w_draft_gate',
    'w_draft_up' [I_d][2 hidden], 'w_draft_down' [hidden][I_d] (bf16 device
    tensors, torch Linear layout) and optionally 'g_final' [hidden]; the
    projections are packed once here.  ``step`` is the DecodeStep whose plan
    and workspace it shares (the workspace is enlarged if needed).  ``window``
    is the next window's length per branch (hpd_pmtp_desc.window; 0 = the
    largest k_b of the step).
    """

    def __init__(self, step, pmtp, stream=None, window=0):
        self.step = step
        self.vocab, self.hidden = pmtp["lm_head"].shape
        self.draft_inner = pmtp["w_draft_gate"].shape[0]
        self._w = dict(lm_head=pack_weight(pmtp["lm_head"], stream),
                       gate_up=pack_gate_up(pmtp["w_draft_gate"], pmtp["w_draft_up"], stream),
                       down=pack_weight(pmtp["w_draft_down"], stream, f16=True),
                       embed=pmtp["embed"].contiguous(), g_final=pmtp.get("g_final"))
        g = self._w["g_final"]
        self.desc = _lib.hpd_pmtp_desc(self.vocab, self.draft_inner, self._w["lm_head"].data_ptr(),
                                       None if g is None else g.data_ptr(), self._w["embed"].data_ptr(),
                                       self._w["gate_up"].data_ptr(), self._w["down"].data_ptr(), window)
        plan = step.attn.plan
        self.ws_bytes = step.plan_bytes + _lib.hpd_pmtp_workspace_bytes(step.model, self.desc, plan)
        if self.ws_bytes > step.ws_bytes:   # one workspace for both steps
            step.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=step.workspace.device)
            step.ws_bytes = self.ws_bytes
            _lib.hpd_plan_upload(plan, step.workspace.data_ptr(), step.ws_bytes, _stream(stream))
        self.T = step.T

    def __call__(self, hidden, tokens_in, verified=None, n_acc=None, draft_out=None, stream=None):
        dev = hidden.device
        nb = len(self.step.attn.info["q_row"])
        verified = torch.empty(self.T, dtype=torch.int32, device=dev) if verified is None else verified
        n_acc = torch.empty(nb, dtype=torch.int32, device=dev) if n_acc is None else n_acc
        draft_out = torch.empty((nb, _lib.HPD_MAX_K), dtype=torch.int32, device=dev) if draft_out is None else draft_out
        _lib.hpd_verify_draft_step(self.step.model, self.desc, self.step.attn.plan, hidden.data_ptr(),
                                   tokens_in.data_ptr(), verified.data_ptr(), n_acc.data_ptr(), draft_out.data_ptr(),
                                   self.step.workspace.data_ptr(), self.step.ws_bytes, _stream(stream))
        return verified, n_acc, draft_out

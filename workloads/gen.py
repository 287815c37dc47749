"""Seeded generator of branch-parallel decode-step inputs.

Everything is drawn from ``numpy.random.default_rng(seed)`` (PCG64) in a
fixed order, so a (workload, seed) pair always yields the same bits:

1. structure: for every page its prefix length P_p, then its number of
   content branches, then the past private length of each of its branches in
   branch order (layout branch first, when the page has one);
2. values, all ``standard_normal`` in fp64: for every page its shared K then
   its shared V; then for every branch its Q, its private K and its private V.
   The decoder-stack workload instead draws, for every layer, each page's
   shared K then V and each branch's past private K then V; then the hidden
   input; then per layer the weights W_qkv, W_o, W_gate, W_up, W_down
   (N(0, std^2)).

Storage types: fp32 workloads keep float32 arrays; bf16 workloads keep the
bf16 bit patterns as uint16, rounded fp64 -> fp32 -> bf16 with
round-to-nearest-even at each step.  Both the oracle and the GPU path read
these stored values, so the rounding itself never enters a parity comparison.

Layout of the packed arrays (row-major, contiguous):
  q         [T][Hq][D]       tokens in branch order, each branch's k_b tokens
  shared_k  [sum P_p][Hkv][D]  pages in order
  shared_v  like shared_k
  priv_k    [sum (L_b + k_b)][Hkv][D]  branches in order; branch b's rows are
            its L_b past tokens followed by its k_b new tokens
  priv_v    like priv_k
Only concatenation produces these arrays; no offset table is computed here.
"""

from dataclasses import dataclass, field

import numpy as np

from .configs import get_config


# ----------------------------------------------------------------- bf16 bits

def f64_to_bf16_bits(x):
    """fp64 -> fp32 (RNE) -> bf16 (RNE) bit patterns as uint16."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f64(bits):
    """Exact value of bf16 bit patterns, as fp64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def _store(x, dtype):
    if dtype == "bf16":
        return f64_to_bf16_bits(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def stored_to_f64(a, dtype):
    """Exact fp64 value of a stored array (bf16 bits or float32)."""
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------- structure

def _draw_len(spec, rng, index=None):
    kind = spec[0]
    if kind == "fixed":
        return int(spec[1])
    if kind == "list":
        return int(spec[1][index])
    if kind == "uniform":
        return int(rng.integers(spec[1], spec[2] + 1))
    if kind == "lognormal":
        median, sigma, lo, hi = spec[1:]
        z = rng.standard_normal()
        v = np.rint(np.exp(np.log(median) + sigma * z))
        return int(min(max(v, lo), hi))
    raise ValueError(f"unknown length spec {spec!r}")


def make_structure(cfg, rng):
    """Draw the ragged page/branch structure of one batch.

    Returns a dict of int32 arrays: prefix_len[num_pages], branch_page[nb],
    num_new[nb], past_len[nb], and a bool array is_layout[nb].
    """
    prefix_len, branch_page, num_new, past_len, is_layout = [], [], [], [], []
    for p in range(cfg["num_pages"]):
        prefix_len.append(_draw_len(cfg["prefix"], rng))
        n_content = _draw_len(cfg["content_count"], rng)
        if cfg.get("layout") is not None:
            branch_page.append(p)
            num_new.append(int(cfg["layout"]["k"]))
            past_len.append(_draw_len(cfg["layout"]["past"], rng))
            is_layout.append(True)
        for i in range(n_content):
            branch_page.append(p)
            num_new.append(int(cfg["content_k"]))
            past_len.append(_draw_len(cfg["content_past"], rng, i))
            is_layout.append(False)
    return dict(
        prefix_len=np.asarray(prefix_len, dtype=np.int32),
        branch_page=np.asarray(branch_page, dtype=np.int32),
        num_new=np.asarray(num_new, dtype=np.int32),
        past_len=np.asarray(past_len, dtype=np.int32),
        is_layout=np.asarray(is_layout, dtype=bool),
    )


# ----------------------------------------------------------------- batches

@dataclass
class AttnBatch:
    """One attention layer's inputs for a ragged branch batch."""
    name: str
    seed: int
    dtype: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prefix_len: np.ndarray
    branch_page: np.ndarray
    num_new: np.ndarray
    past_len: np.ndarray
    is_layout: np.ndarray
    q: np.ndarray
    shared_k: np.ndarray
    shared_v: np.ndarray
    priv_k: np.ndarray
    priv_v: np.ndarray
    fork_len: np.ndarray = None   # optional per-branch visible prefix; None = whole prefix

    @property
    def num_pages(self):
        return int(self.prefix_len.shape[0])

    @property
    def num_branches(self):
        return int(self.num_new.shape[0])

    @property
    def num_tokens(self):
        return int(self.q.shape[0])

    def f64(self, name):
        """Exact fp64 value of one stored tensor ('q', 'shared_k', ...)."""
        return stored_to_f64(getattr(self, name), self.dtype)


def _values_for(structure, Hq, Hkv, D, dtype, rng):
    shared_k, shared_v, q, priv_k, priv_v = [], [], [], [], []
    for P in structure["prefix_len"]:
        shared_k.append(rng.standard_normal((int(P), Hkv, D)))
        shared_v.append(rng.standard_normal((int(P), Hkv, D)))
    for k, L in zip(structure["num_new"], structure["past_len"]):
        q.append(rng.standard_normal((int(k), Hq, D)))
        priv_k.append(rng.standard_normal((int(L + k), Hkv, D)))
        priv_v.append(rng.standard_normal((int(L + k), Hkv, D)))

    def cat(parts, tail):
        if not parts:
            return _store(np.zeros((0,) + tail), dtype)
        return _store(np.concatenate(parts, axis=0), dtype)
    return dict(q=cat(q, (Hq, D)), shared_k=cat(shared_k, (Hkv, D)),
                shared_v=cat(shared_v, (Hkv, D)), priv_k=cat(priv_k, (Hkv, D)),
                priv_v=cat(priv_v, (Hkv, D)))


def attn_batch_from_structure(structure, num_q_heads, num_kv_heads, head_dim,
                              dtype, seed, name="custom"):
    """Values for a given structure, drawn from their own seeded stream."""
    rng = np.random.default_rng(seed)
    vals = _values_for(structure, num_q_heads, num_kv_heads, head_dim, dtype, rng)
    return AttnBatch(name=name, seed=seed, dtype=dtype, num_q_heads=num_q_heads,
                     num_kv_heads=num_kv_heads, head_dim=head_dim,
                     prefix_len=structure["prefix_len"], branch_page=structure["branch_page"],
                     num_new=structure["num_new"], past_len=structure["past_len"],
                     is_layout=structure.get("is_layout",
                                             np.zeros(len(structure["num_new"]), bool)),
                     fork_len=structure.get("fork_len"), **vals)


def draw_fork_len(structure, visual, rng):
    """Per-branch visible prefix F_b: the layout branch sees its page's whole
    prefix, a content branch a uniform integer in [min(visual, P), P]."""
    out = []
    for b, p in enumerate(structure["branch_page"]):
        P = int(structure["prefix_len"][p])
        if structure["is_layout"][b]:
            out.append(P)
        else:
            out.append(int(rng.integers(min(visual, P), P + 1)))
    return np.asarray(out, dtype=np.int32)


def make_attn_batch(cfg_or_name, seed):
    """Structure then values (then fork offsets, if the workload has them) of
    one single-layer workload, from one stream."""
    cfg = get_config(cfg_or_name) if isinstance(cfg_or_name, str) else cfg_or_name
    rng = np.random.default_rng(seed)
    st = make_structure(cfg, rng)
    vals = _values_for(st, cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"],
                       cfg["dtype"], rng)
    fork = draw_fork_len(st, cfg["fork"]["visual"], rng) if cfg.get("fork") else None
    return AttnBatch(name=cfg["name"], seed=seed, dtype=cfg["dtype"],
                     num_q_heads=cfg["num_q_heads"], num_kv_heads=cfg["num_kv_heads"],
                     head_dim=cfg["head_dim"], fork_len=fork, **st, **vals)


@dataclass
class DecodeInputs:
    """Inputs of one decode step of the synthetic decoder stack.

    Per layer l: shared_k[l], shared_v[l] [sum P][Hkv][D] bf16 bits;
    priv_k[l], priv_v[l] [sum (L_b + k_b)][Hkv][D] bf16 bits whose k_b new
    rows per branch are zero (the step writes them).  hidden_in [T][hidden]
    float32 holding bf16-representable values.  Weights are bf16 bits in
    torch Linear layout W[out][in]: w_qkv [(Hq + 2 Hkv) D][hidden] (q rows,
    then k rows, then v rows), w_o [hidden][Hq D], w_gate and w_up
    [intermediate][hidden], w_down [hidden][intermediate].
    """
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_layers: int
    hidden: int
    intermediate: int
    rms_eps: float
    prefix_len: np.ndarray
    branch_page: np.ndarray
    num_new: np.ndarray
    past_len: np.ndarray
    is_layout: np.ndarray
    hidden_in: np.ndarray
    shared_k: list = field(default_factory=list)
    shared_v: list = field(default_factory=list)
    priv_k: list = field(default_factory=list)
    priv_v: list = field(default_factory=list)
    w_qkv: list = field(default_factory=list)
    w_o: list = field(default_factory=list)
    w_gate: list = field(default_factory=list)
    w_up: list = field(default_factory=list)
    w_down: list = field(default_factory=list)
    # Qwen3-style attention (model "qwen3" in the config): per-layer [64] bf16
    # gains of the per-head q / k RMSNorm and the rotary base; None / 0 = off
    q_norm: list = None
    k_norm: list = None
    rope_theta: float = 0.0

    @property
    def num_tokens(self):
        return int(self.hidden_in.shape[0])


def make_decode_inputs(cfg_or_name, seed, num_layers=None):
    """Structure, per-layer KV, hidden input and weights of the decoder step.

    ``num_layers`` may shorten the stack (tests use fewer layers); the draw
    order stays the same, so layer l of a short stack equals layer l of the
    full one only for the KV part.
    """
    cfg = get_config(cfg_or_name) if isinstance(cfg_or_name, str) else cfg_or_name
    m = cfg["model"]
    Lyr = int(num_layers if num_layers is not None else m["num_layers"])
    Hq, Hkv, D = cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"]
    H, I, std = m["hidden"], m["intermediate"], m["weight_std"]
    rng = np.random.default_rng(seed)
    st = make_structure(cfg, rng)
    out = DecodeInputs(name=cfg["name"], seed=seed, num_q_heads=Hq, num_kv_heads=Hkv,
                       head_dim=D, num_layers=Lyr, hidden=H, intermediate=I,
                       rms_eps=float(m["rms_eps"]), hidden_in=None, **st)
    for _ in range(Lyr):
        sk, sv = [], []
        for P in st["prefix_len"]:
            sk.append(rng.standard_normal((int(P), Hkv, D)))
            sv.append(rng.standard_normal((int(P), Hkv, D)))
        pk, pv = [], []
        for k, L in zip(st["num_new"], st["past_len"]):
            pk.append(np.concatenate([rng.standard_normal((int(L), Hkv, D)),
                                      np.zeros((int(k), Hkv, D))]))
            pv.append(np.concatenate([rng.standard_normal((int(L), Hkv, D)),
                                      np.zeros((int(k), Hkv, D))]))
        out.shared_k.append(f64_to_bf16_bits(np.concatenate(sk)))
        out.shared_v.append(f64_to_bf16_bits(np.concatenate(sv)))
        out.priv_k.append(f64_to_bf16_bits(np.concatenate(pk)))
        out.priv_v.append(f64_to_bf16_bits(np.concatenate(pv)))
    T = int(st["num_new"].sum())
    out.hidden_in = bf16_bits_to_f64(f64_to_bf16_bits(rng.standard_normal((T, H)))).astype(np.float32)
    for _ in range(Lyr):
        out.w_qkv.append(f64_to_bf16_bits(std * rng.standard_normal(((Hq + 2 * Hkv) * D, H))))
        out.w_o.append(f64_to_bf16_bits(std * rng.standard_normal((H, Hq * D))))
        out.w_gate.append(f64_to_bf16_bits(std * rng.standard_normal((I, H))))
        out.w_up.append(f64_to_bf16_bits(std * rng.standard_normal((I, H))))
        out.w_down.append(f64_to_bf16_bits(std * rng.standard_normal((H, I))))
    qw = m.get("qwen3")
    if qw:   # own stream (seed, 13): every draw above is unchanged
        out.rope_theta = float(qw["rope_theta"])
        if qw.get("qk_norm"):
            r2 = np.random.default_rng([seed, 13])
            gain = lambda: f64_to_bf16_bits(1.0 + 0.1 * r2.standard_normal(D))
            out.q_norm = [gain() for _ in range(Lyr)]
            out.k_norm = [gain() for _ in range(Lyr)]
    return out


@dataclass
class PmtpInputs:
    """Weights of P-MTP verification and drafting (bf16 bits, torch Linear
    layout): lm_head and embed [V][hidden], w_draft_gate and w_draft_up
    [I_d][2 hidden], w_draft_down [hidden][I_d]; g_final None (ones)."""
    vocab: int
    draft_inner: int
    lm_head: np.ndarray
    embed: np.ndarray
    w_draft_gate: np.ndarray
    w_draft_up: np.ndarray
    w_draft_down: np.ndarray
    g_final: np.ndarray = None


def make_pmtp_inputs(hidden, vocab, draft_inner, weight_std, seed):
    """P-MTP weights drawn N(0, std^2) from their own stream (seed, 7), in the
    order lm_head, embed, gate, up, down; they leave every other draw of the
    workload unchanged."""
    rng = np.random.default_rng([seed, 7])
    w = lambda r, c: f64_to_bf16_bits(rng.standard_normal((r, c)) * weight_std)
    return PmtpInputs(vocab=vocab, draft_inner=draft_inner, lm_head=w(vocab, hidden), embed=w(vocab, hidden),
                      w_draft_gate=w(draft_inner, 2 * hidden), w_draft_up=w(draft_inner, 2 * hidden),
                      w_draft_down=w(hidden, draft_inner))

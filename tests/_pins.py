"""Pins of the fp64 oracle: checks against things other than the oracle itself.

Each pin takes the oracle modules as arguments (so the mutation tests can run
the same pins against deliberately broken copies of the oracle) and returns a
non-negative error; the pin holds when the error is <= its tolerance.

Kinds of pin used (none retypes the oracle's own formula):
  hand        closed forms derived by hand (tests/golden/hand_cases.json)
  brute       pure-Python enumeration of each token's visible key list
  library     torch's scaled_dot_product_attention / rms_norm / silu in fp64
  identity    split + LSE merge equals attention over the concatenated keys
  invariant   softmax rows sum to 1, isolation, causal prefix consistency,
              branch-permutation equivariance, visible-count recovery
"""

import json
import math
import os

import numpy as np
import torch

from workloads import get_config
from workloads.gen import attn_batch_from_structure, make_decode_inputs

from ._brute import brute_attention

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TOL = 1e-12


def _worse(err, *vals):
    """The largest of the errors; NaN counts as an infinite error (Python's
    max would silently drop it)."""
    for v in vals:
        v = float(v)
        err = float("inf") if math.isnan(v) else max(err, v)
    return err


def _st(batch):
    return dict(prefix_len=batch.prefix_len, branch_page=batch.branch_page,
                num_new=batch.num_new, past_len=batch.past_len, fork_len=batch.fork_len)


def _run(att, batch, keys="all", return_weights=False):
    return att.attention(batch.f64("q"), batch.f64("shared_k"), batch.f64("shared_v"),
                         batch.f64("priv_k"), batch.f64("priv_v"), _st(batch),
                         batch.num_q_heads, batch.num_kv_heads, keys=keys,
                         return_weights=return_weights)


def tiny_structures():
    """Small ragged structures covering: several pages, L = 0, k = 1 and k > 1,
    a page whose only branch has an empty prefix, and unequal group sizes."""
    S = []
    S.append(dict(prefix_len=np.array([5], np.int32), branch_page=np.array([0, 0, 0], np.int32),
                  num_new=np.array([1, 3, 2], np.int32), past_len=np.array([4, 0, 2], np.int32)))
    S.append(dict(prefix_len=np.array([3, 0, 6], np.int32), branch_page=np.array([0, 1, 2, 2], np.int32),
                  num_new=np.array([2, 1, 1, 3], np.int32), past_len=np.array([1, 2, 0, 5], np.int32)))
    S.append(dict(prefix_len=np.array([7], np.int32), branch_page=np.array([0], np.int32),
                  num_new=np.array([4], np.int32), past_len=np.array([3], np.int32)))
    return S


def fork_structures():
    """Tiny structures with per-branch fork points F_b < P_p (a branch sees its
    page's prefix only up to its fork position, section "Layout-Coordinated
    Parallel Decoding", paragraph "Dynamic Branch Forking and Efficient Context
    Isolation"): F_b in {0, 1, a middle value, P_p} on one page, the same mix
    over three pages (one of them empty), and one branch whose fork cuts the
    prefix while k > 1."""
    S = []
    S.append(dict(prefix_len=np.array([7], np.int32), branch_page=np.array([0, 0, 0, 0], np.int32),
                  num_new=np.array([1, 3, 2, 2], np.int32), past_len=np.array([2, 0, 3, 1], np.int32),
                  fork_len=np.array([7, 0, 1, 4], np.int32)))
    S.append(dict(prefix_len=np.array([5, 0, 9], np.int32), branch_page=np.array([0, 0, 1, 2, 2, 2], np.int32),
                  num_new=np.array([2, 1, 1, 3, 1, 2], np.int32), past_len=np.array([0, 3, 2, 1, 4, 0], np.int32),
                  fork_len=np.array([5, 2, 0, 0, 9, 3], np.int32)))
    S.append(dict(prefix_len=np.array([6], np.int32), branch_page=np.array([0], np.int32),
                  num_new=np.array([4], np.int32), past_len=np.array([2], np.int32),
                  fork_len=np.array([3], np.int32)))
    return S


def tiny_batches(dtype="f32"):
    out = []
    for i, st in enumerate(tiny_structures() + fork_structures()):
        for Hq, Hkv, D in [(4, 2, 8), (2, 1, 3), (6, 3, 4)]:
            out.append(attn_batch_from_structure(st, Hq, Hkv, D, dtype, seed=100 + i))
    return out


def _fork_list(b):
    return None if b.fork_len is None else [int(f) for f in b.fork_len]


# ------------------------------------------------------------------ pins

def pin_hand_cases(att, plan=None, dec=None):
    with open(os.path.join(GOLDEN, "hand_cases.json")) as f:
        cases = json.load(f)["cases"]
    ns = {"e": math.e, "log": math.log, "exp": math.exp, "__builtins__": {}}
    err = 0.0
    for c in cases:
        st = dict(prefix_len=np.array(c["prefix_len"]), branch_page=np.array(c["branch_page"]),
                  num_new=np.array(c["num_new"]), past_len=np.array(c["past_len"]))
        arr = {k: np.array(c[k], dtype=np.float64) for k in ("q", "shared_k", "shared_v", "priv_k", "priv_v")}
        O, lse = att.attention(arr["q"], arr["shared_k"], arr["shared_v"], arr["priv_k"], arr["priv_v"],
                               st, c["Hq"], c["Hkv"])
        eO = np.vectorize(lambda s: eval(s, ns))(np.array(c["expected_O"], dtype=object)).astype(np.float64)
        eL = np.vectorize(lambda s: eval(s, ns))(np.array(c["expected_lse"], dtype=object)).astype(np.float64)
        err = _worse(err, float(np.abs(O - eO).max()), float(np.abs(lse - eL).max()))
    return err


def pin_brute_force(att, plan=None, dec=None):
    err = 0.0
    for b in tiny_batches():
        O, lse = _run(att, b)
        D = b.head_dim
        bO, bL = brute_attention(b.f64("q").tolist(), b.f64("shared_k").tolist(), b.f64("shared_v").tolist(),
                                 b.f64("priv_k").tolist(), b.f64("priv_v").tolist(), b.prefix_len.tolist(),
                                 b.branch_page.tolist(), b.num_new.tolist(), b.past_len.tolist(),
                                 b.num_q_heads, b.num_kv_heads, 1.0 / math.sqrt(D),
                                 fork_len=_fork_list(b))
        err = _worse(err, float(np.abs(O - np.array(bO)).max()), float(np.abs(lse - np.array(bL)).max()))
    return err


def pin_split_merge(att, plan=None, dec=None):
    """merge(shared-only partial, private-only partial) == attention over all keys."""
    err = 0.0
    for b in tiny_batches():
        O, lse = _run(att, b)
        s = _run(att, b, keys="shared")
        p = _run(att, b, keys="private")
        Om, lm = att.lse_merge([s, p])
        err = _worse(err, float(np.abs(O - Om).max()), float(np.abs(lse - lm).max()))
        # merging with an empty partial (lse = -inf) is the identity
        empty = (np.full_like(O, 7.0), np.full_like(lse, -np.inf))
        Oe, le = att.lse_merge([(O, lse), empty])
        err = _worse(err, float(np.abs(O - Oe).max()), float(np.abs(lse - le).max()))
    return err


def _sdpa_single_branch(b, mask_bottom_right):
    """torch fp64 SDPA over [prefix up to the fork ; private] for a one-branch batch."""
    P = int(b.prefix_len[0]) if b.fork_len is None else int(b.fork_len[0])
    L, k = int(b.past_len[0]), int(b.num_new[0])
    G = b.num_q_heads // b.num_kv_heads
    q = torch.from_numpy(b.f64("q")).permute(1, 0, 2)[None]            # [1, Hq, k, D]
    K = torch.from_numpy(np.concatenate([b.f64("shared_k")[:P], b.f64("priv_k")[:L + k]]))
    V = torch.from_numpy(np.concatenate([b.f64("shared_v")[:P], b.f64("priv_v")[:L + k]]))
    K = K.permute(1, 0, 2).repeat_interleave(G, dim=0)[None]            # [1, Hq, N, D]
    V = V.permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    mask = None
    if mask_bottom_right:
        N = P + L + k
        mask = torch.zeros(k, N, dtype=torch.bool)
        for j in range(k):
            mask[j, :P + L + j + 1] = True
    out = torch.nn.functional.scaled_dot_product_attention(q, K, V, attn_mask=mask)
    return out[0].permute(1, 0, 2).numpy()


def pin_sdpa_k1(att, plan=None, dec=None):
    """1 branch, k = 1: plain decode attention over [prefix ; private], no mask."""
    err = 0.0
    for (P, L, Hq, Hkv, D, seed) in [(9, 4, 4, 2, 8, 1), (0, 6, 2, 2, 5, 2), (17, 0, 8, 2, 16, 3)]:
        st = dict(prefix_len=np.array([P]), branch_page=np.array([0]), num_new=np.array([1]),
                  past_len=np.array([L]))
        b = attn_batch_from_structure(st, Hq, Hkv, D, "f32", seed)
        O, _ = _run(att, b)
        err = _worse(err, float(np.abs(O - _sdpa_single_branch(b, False)).max()))
    return err


def pin_sdpa_bottom_right(att, plan=None, dec=None):
    """1 branch, k > 1: SDPA with an explicit bottom-right causal mask."""
    err = 0.0
    for (P, L, k, Hq, Hkv, D, seed) in [(9, 4, 3, 4, 2, 8, 4), (0, 0, 5, 4, 1, 4, 5), (12, 7, 4, 6, 3, 8, 6)]:
        st = dict(prefix_len=np.array([P]), branch_page=np.array([0]), num_new=np.array([k]),
                  past_len=np.array([L]))
        b = attn_batch_from_structure(st, Hq, Hkv, D, "f32", seed)
        O, _ = _run(att, b)
        err = _worse(err, float(np.abs(O - _sdpa_single_branch(b, True)).max()))
    return err


def pin_sdpa_fork(att, plan=None, dec=None):
    """1 branch whose fork point cuts its page's prefix (F < P): SDPA over the
    first F prefix rows and the private rows, bottom-right mask.  The prefix
    rows past the fork get large keys, so seeing any of them moves O."""
    err = 0.0
    for (P, F, L, k, Hq, Hkv, D, seed) in [(12, 5, 3, 3, 4, 2, 8, 8), (9, 0, 2, 2, 2, 1, 4, 9),
                                           (10, 1, 0, 4, 6, 3, 8, 10), (7, 7, 1, 2, 4, 2, 8, 11)]:
        st = dict(prefix_len=np.array([P]), branch_page=np.array([0]), num_new=np.array([k]),
                  past_len=np.array([L]), fork_len=np.array([F]))
        b = attn_batch_from_structure(st, Hq, Hkv, D, "f32", seed)
        b.shared_k = b.shared_k.copy()
        b.shared_k[F:] *= 4.0
        O, _ = _run(att, b)
        err = _worse(err, float(np.abs(O - _sdpa_single_branch(b, True)).max()))
    return err


def pin_rows_sum_to_one(att, plan=None, dec=None):
    err = 0.0
    for b in tiny_batches():
        _, _, ws = _run(att, b, return_weights=True)
        for w in ws:
            err = _worse(err, float(np.abs(w.sum(axis=2) - 1.0).max()))
            if (w < 0).any():
                return float("inf")
    return err


def pin_visible_count(att, plan=None, dec=None):
    """Q = 0 makes O the mean of the visible V rows.  With V of key i set to
    (1, i) in shared/private position codes, O recovers the exact visible
    count F_b + L_b + j + 1 (1 / O[0] = count) and which rows were seen."""
    err = 0.0
    for st in tiny_structures() + fork_structures():
        Hq, Hkv, D = 4, 2, 3
        b = attn_batch_from_structure(st, Hq, Hkv, D, "f32", seed=7)
        q = np.zeros_like(b.f64("q"))
        sk = np.zeros_like(b.f64("shared_k"))
        pk = np.zeros_like(b.f64("priv_k"))
        sv = np.zeros_like(b.f64("shared_v"))
        pv = np.zeros_like(b.f64("priv_v"))
        sv[:, :, 0] = 1.0
        pv[:, :, 0] = 1.0
        sv[:, :, 1] = np.arange(sv.shape[0])[:, None] + 1.0            # shared row id + 1
        pv[:, :, 2] = np.arange(pv.shape[0])[:, None] + 1.0            # private row id + 1
        O, lse = att.attention(q, sk, sv, pk, pv, _st(b), Hq, Hkv)
        # expected, by walking the structure with running counters
        t, prow, pstart = 0, 0, np.concatenate([[0], np.cumsum(st["prefix_len"])])
        for bi in range(len(st["num_new"])):
            p, k, L = int(st["branch_page"][bi]), int(st["num_new"][bi]), int(st["past_len"][bi])
            F = int(st["prefix_len"][p]) if "fork_len" not in st else int(st["fork_len"][bi])
            for j in range(k):
                n = F + L + j + 1
                srow_sum = sum(range(int(pstart[p]) + 1, int(pstart[p]) + F + 1))
                prow_sum = sum(range(prow + 1, prow + L + j + 2))
                exp_row = np.array([1.0, srow_sum / n, prow_sum / n])
                err = _worse(err, float(np.abs(O[t] - exp_row[None]).max()),
                          float(np.abs(lse[t] - math.log(n)).max()))
                t += 1
            prow += L + k
    return err


def pin_isolation(att, plan=None, dec=None):
    """Changing one branch's private K/V changes no other branch's output."""
    err = 0.0
    for b in tiny_batches():
        O, _ = _run(att, b)
        nb = b.num_branches
        for victim in range(nb):
            pk, pv = b.f64("priv_k").copy(), b.f64("priv_v").copy()
            r0 = int(np.sum(b.past_len[:victim] + b.num_new[:victim]))
            r1 = r0 + int(b.past_len[victim] + b.num_new[victim])
            pk[r0:r1] += 3.0
            pv[r0:r1] -= 5.0
            O2, _ = att.attention(b.f64("q"), b.f64("shared_k"), b.f64("shared_v"), pk, pv, _st(b),
                                  b.num_q_heads, b.num_kv_heads)
            t0 = int(np.sum(b.num_new[:victim]))
            t1 = t0 + int(b.num_new[victim])
            keep = np.ones(O.shape[0], bool)
            keep[t0:t1] = False
            err = _worse(err, float(np.abs(O[keep] - O2[keep]).max()) if keep.any() else 0.0)
            if not np.abs(O[t0:t1] - O2[t0:t1]).max() > 1e-6:   # the victim itself must change
                return float("inf")
    return err


def pin_causal_prefix(att, plan=None, dec=None):
    """Token j of a branch equals the last token of the same branch run with
    k = j + 1 (trailing drafts removed)."""
    err = 0.0
    for b in tiny_batches():
        O, lse = _run(att, b)
        q, pk, pv = b.f64("q"), b.f64("priv_k"), b.f64("priv_v")
        t0 = 0
        r0 = 0
        for bi in range(b.num_branches):
            k, L = int(b.num_new[bi]), int(b.past_len[bi])
            for j in range(k):
                st = dict(prefix_len=b.prefix_len, branch_page=np.array([b.branch_page[bi]]),
                          num_new=np.array([j + 1]), past_len=np.array([L]),
                          fork_len=None if b.fork_len is None else np.array([b.fork_len[bi]]))
                O1, l1 = att.attention(q[t0:t0 + j + 1], b.f64("shared_k"), b.f64("shared_v"),
                                       pk[r0:r0 + L + j + 1], pv[r0:r0 + L + j + 1], st,
                                       b.num_q_heads, b.num_kv_heads)
                err = _worse(err, float(np.abs(O1[j] - O[t0 + j]).max()),
                          float(np.abs(l1[j] - lse[t0 + j]).max()))
            t0 += k
            r0 += L + k
    return err


def pin_equivariance(att, plan=None, dec=None):
    """Reversing the branch order within each page permutes the outputs."""
    err = 0.0
    for b in tiny_batches():
        O, _ = _run(att, b)
        nb = b.num_branches
        order = sorted(range(nb), key=lambda i: (int(b.branch_page[i]), -i))
        q, pk, pv = b.f64("q"), b.f64("priv_k"), b.f64("priv_v")
        qs, pks, pvs, Os = [], [], [], []
        t_start = np.concatenate([[0], np.cumsum(b.num_new)])
        r_start = np.concatenate([[0], np.cumsum(b.past_len + b.num_new)])
        for i in order:
            qs.append(q[t_start[i]:t_start[i + 1]])
            pks.append(pk[r_start[i]:r_start[i + 1]])
            pvs.append(pv[r_start[i]:r_start[i + 1]])
            Os.append(O[t_start[i]:t_start[i + 1]])
        st = dict(prefix_len=b.prefix_len, branch_page=b.branch_page[order],
                  num_new=b.num_new[order], past_len=b.past_len[order],
                  fork_len=None if b.fork_len is None else b.fork_len[order])
        O2, _ = att.attention(np.concatenate(qs), b.f64("shared_k"), b.f64("shared_v"),
                              np.concatenate(pks), np.concatenate(pvs), st,
                              b.num_q_heads, b.num_kv_heads)
        err = _worse(err, float(np.abs(O2 - np.concatenate(Os)).max()))
    return err


def pin_plan_walk(att=None, plan=None, dec=None):
    """canonical_plan vs a running-counter walk over the branches."""
    err = 0
    for st in tiny_structures() + fork_structures() + [
            dict(prefix_len=np.array([4, 4]), branch_page=np.array([1, 1]),
                 num_new=np.array([2, 3]), past_len=np.array([0, 9]))]:
        fork = st.get("fork_len")
        pl = plan.canonical_plan(st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"], fork)
        q_row, priv_row, vis, forks = [], [], [], []
        tq, tr = 0, 0
        page_T = [0] * len(st["prefix_len"])
        for bi in range(len(st["num_new"])):
            q_row.append(tq)
            priv_row.append(tr)
            p = int(st["branch_page"][bi])
            page_T[p] += int(st["num_new"][bi])
            F = int(st["prefix_len"][p]) if fork is None else int(fork[bi])
            forks.append(F)
            for j in range(int(st["num_new"][bi])):
                vis.append(F + int(st["past_len"][bi]) + j + 1)
            tq += int(st["num_new"][bi])
            tr += int(st["past_len"][bi]) + int(st["num_new"][bi])
        page_q, acc = [], 0
        for v in page_T:
            page_q.append(acc)
            acc += v
        pre, acc = [], 0
        for v in st["prefix_len"]:
            pre.append(acc)
            acc += int(v)
        for got, want in [(pl["q_row"], q_row), (pl["priv_row"], priv_row), (pl["visible"], vis),
                          (pl["page_T"], page_T), (pl["page_q_row"], page_q), (pl["prefix_row"], pre),
                          (pl["fork"], forks)]:
            if list(map(int, got)) != list(want):
                err += 1
    return float(err)


# --------------------------------------------------------------- decode pins

def _textbook_decoder(inp, branch_sel=None):
    """Pre-norm GQA decoder step written with torch fp64 library routines.

    Each selected branch is processed on its own: its k tokens attend to
    [page prefix ; its past rows ; its new rows] with an explicit bottom-right
    causal mask.  Returns the branch outputs concatenated in branch order.
    """
    Hq, Hkv, D, H = inp.num_q_heads, inp.num_kv_heads, inp.head_dim, inp.hidden
    G = Hq // Hkv

    def val(bits):
        u = torch.from_numpy(np.asarray(bits).astype(np.int32) << 16)
        return u.view(torch.float32).to(torch.float64)

    nb = len(inp.num_new)
    sel = range(nb) if branch_sel is None else branch_sel
    outs = []
    pstart = np.concatenate([[0], np.cumsum(inp.prefix_len)])
    tstart = np.concatenate([[0], np.cumsum(inp.num_new)])
    rstart = np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)])
    for bi in sel:
        p, k, L = int(inp.branch_page[bi]), int(inp.num_new[bi]), int(inp.past_len[bi])
        # the branch sees its page's prefix up to its fork point, and its
        # tokens sit at positions F + L + j of its own sequence
        fork = getattr(inp, "fork_len", None)
        P = int(inp.prefix_len[p]) if fork is None else int(fork[bi])
        h = torch.from_numpy(inp.hidden_in[tstart[bi]:tstart[bi] + k].astype(np.float64))
        for l in range(inp.num_layers):
            x = torch.nn.functional.rms_norm(h, (H,), eps=inp.rms_eps)
            qkv = x @ val(inp.w_qkv[l]).T
            q = qkv[:, :Hq * D].reshape(k, Hq, D)
            kr = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(k, Hkv, D)
            if getattr(inp, "rope_theta", 0.0) or getattr(inp, "q_norm", None) is not None:
                q, kr = _qwen3_library(inp, l, q, kr, [P + L + j for j in range(k)])
            kn = kr.to(torch.float32).to(torch.bfloat16).to(torch.float64)
            vn = qkv[:, (Hq + Hkv) * D:].reshape(k, Hkv, D).to(torch.float32).to(torch.bfloat16).to(torch.float64)
            sk = val(inp.shared_k[l])[pstart[p]:pstart[p] + P]
            sv = val(inp.shared_v[l])[pstart[p]:pstart[p] + P]
            pk = val(inp.priv_k[l])[rstart[bi]:rstart[bi] + L]
            pv = val(inp.priv_v[l])[rstart[bi]:rstart[bi] + L]
            K = torch.cat([sk, pk, kn]).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
            V = torch.cat([sv, pv, vn]).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
            N = P + L + k
            mask = torch.zeros(k, N, dtype=torch.bool)
            for j in range(k):
                mask[j, :P + L + j + 1] = True
            a = torch.nn.functional.scaled_dot_product_attention(q.permute(1, 0, 2)[None], K, V, attn_mask=mask)
            a = a[0].permute(1, 0, 2).reshape(k, Hq * D)
            h = h + a @ val(inp.w_o[l]).T
            x = torch.nn.functional.rms_norm(h, (H,), eps=inp.rms_eps)
            m = torch.nn.functional.silu(x @ val(inp.w_gate[l]).T) * (x @ val(inp.w_up[l]).T)
            h = h + m @ val(inp.w_down[l]).T
        outs.append(h.numpy())
    return np.concatenate(outs)


def _qwen3_library(inp, l, q, k, pos):
    """Qwen3-style q / k of one branch with library routines: torch's rms_norm
    over each head with the gain, then transformers' Qwen3RotaryEmbedding and
    apply_rotary_pos_emb at positions pos (fp32 angles there)."""
    from transformers import Qwen3Config
    from transformers.models.qwen3.modeling_qwen3 import Qwen3RotaryEmbedding, apply_rotary_pos_emb
    D = q.shape[-1]
    val = lambda b: torch.from_numpy(np.asarray(b, np.int32) << 16).view(torch.float32).to(torch.float64)
    if getattr(inp, "q_norm", None) is not None:
        q = torch.nn.functional.rms_norm(q, (D,), weight=val(inp.q_norm[l]), eps=inp.rms_eps)
    if getattr(inp, "k_norm", None) is not None:
        k = torch.nn.functional.rms_norm(k, (D,), weight=val(inp.k_norm[l]), eps=inp.rms_eps)
    if getattr(inp, "rope_theta", 0.0):
        cfg = Qwen3Config(head_dim=D, hidden_size=inp.hidden, num_attention_heads=q.shape[1],
                          num_key_value_heads=k.shape[1], max_position_embeddings=4096, rope_theta=inp.rope_theta)
        cos, sin = Qwen3RotaryEmbedding(cfg)(torch.zeros(1, len(pos), D), torch.tensor(pos)[None])
        qo, ko = apply_rotary_pos_emb(q.permute(1, 0, 2)[None], k.permute(1, 0, 2)[None], cos.double(), sin.double())
        q, k = qo[0].permute(1, 0, 2), ko[0].permute(1, 0, 2)
    return q, k


def small_decode_inputs(seed=3, layers=2, qwen3=None, fork=None):
    model = dict(num_layers=layers, hidden=32, intermediate=48, weight_std=0.2, rms_eps=1e-6)
    if qwen3:
        model["qwen3"] = qwen3
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, head_dim=8, num_pages=1,
                     prefix=("fixed", 11), layout=dict(k=1, past=("fixed", 5)),
                     content_count=("fixed", 2), content_k=3,
                     content_past=("list", [0, 4]), model=model)
    inp = make_decode_inputs(cfg, seed)
    if fork is not None:
        inp.fork_len = np.asarray(fork, np.int64)
    return inp


def pin_decode_textbook(att=None, plan=None, dec=None):
    inp = small_decode_inputs()
    h, _, _ = dec.decode_step(inp)
    ref = _textbook_decoder(inp)
    return float(np.abs(h - ref).max())


def pin_decode_kv_written(att=None, plan=None, dec=None):
    """The K/V rows the step writes equal the bf16 rounding (torch) of the
    projections of the normed residual stream entering each layer, which the
    textbook decoder recomputes branch by branch; checked for layer 0 where
    the residual stream is the input."""
    inp = small_decode_inputs()
    _, nk, nv = dec.decode_step(inp)
    Hq, Hkv, D, H = inp.num_q_heads, inp.num_kv_heads, inp.head_dim, inp.hidden
    x = torch.nn.functional.rms_norm(torch.from_numpy(inp.hidden_in.astype(np.float64)), (H,), eps=inp.rms_eps)
    w = torch.from_numpy(inp.w_qkv[0].astype(np.int32) << 16).view(torch.float32).to(torch.float64)
    qkv = x @ w.T
    T = x.shape[0]
    kb = qkv[:, Hq * D:(Hq + Hkv) * D].to(torch.float32).to(torch.bfloat16).reshape(T, Hkv, D)
    vb = qkv[:, (Hq + Hkv) * D:].to(torch.float32).to(torch.bfloat16).reshape(T, Hkv, D)
    kbits = kb.view(torch.int16).numpy().astype(np.uint16)
    vbits = vb.view(torch.int16).numpy().astype(np.uint16)
    return float(np.count_nonzero(kbits != nk[0]) + np.count_nonzero(vbits != nv[0]))


def pin_decode_qwen3_library(att=None, plan=None, dec=None):
    """The step with per-head QK norm and rotary embedding against the
    branch-by-branch decoder built from torch's rms_norm / SDPA and
    transformers' Qwen3 rotary routines (base 10^2, so positions 11..20 turn
    every frequency by a visible angle)."""
    inp = small_decode_inputs(qwen3=dict(rope_theta=100.0, qk_norm=True))
    h, _, _ = dec.decode_step(inp)
    return float(np.abs(h - _textbook_decoder(inp)).max())


def pin_decode_textbook_fork(att=None, plan=None, dec=None):
    """Fork points 11 (the whole 11-row prefix), 0 and 6 for the layout branch
    and the two content branches: each branch's textbook decode reads only its
    first F_b prefix rows."""
    inp = small_decode_inputs(fork=[11, 0, 6])
    h, _, _ = dec.decode_step(inp)
    return float(np.abs(h - _textbook_decoder(inp)).max())


def pin_decode_qwen3_fork(att=None, plan=None, dec=None):
    """The Qwen3-style step with fork points: the rotary position of token j of
    branch b is F_b + L_b + j (its place in its own sequence), checked against
    transformers' rotary routines at those positions."""
    inp = small_decode_inputs(qwen3=dict(rope_theta=100.0, qk_norm=True), fork=[11, 1, 6])
    h, _, _ = dec.decode_step(inp)
    return float(np.abs(h - _textbook_decoder(inp)).max())


ATTN_PINS = [pin_hand_cases, pin_brute_force, pin_split_merge, pin_sdpa_k1, pin_sdpa_bottom_right,
             pin_sdpa_fork, pin_rows_sum_to_one, pin_visible_count, pin_isolation, pin_causal_prefix,
             pin_equivariance]
PLAN_PINS = [pin_plan_walk]
DECODE_PINS = [pin_decode_textbook, pin_decode_kv_written, pin_decode_qwen3_library,
               pin_decode_textbook_fork, pin_decode_qwen3_fork]
# the Qwen3 pins: transformers takes the rotary angles in fp32 (about 1e-7 relative)
TOLERANCE = {pin_decode_textbook: 1e-10, pin_plan_walk: 0.0, pin_decode_kv_written: 0.0,
             pin_decode_qwen3_library: 1e-5, pin_decode_textbook_fork: 1e-10,
             pin_decode_qwen3_fork: 1e-5}

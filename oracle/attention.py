"""Branch-parallel attention of one layer, in fp64 (oracle side).

Test infrastructure: see the package docstring.

Definition followed (section "Layout-Coordinated Parallel Decoding",
paragraph "Dynamic Branch Forking and Efficient Context Isolation"; section
"Integration with P-MTP", parallel verification of drafts; section
"Overview", GQA): for page p, branch b on p, new token j < k_b and query head
h, with kv head g = h // (Hq / Hkv) (contiguous query-head groups):

  keys(b, j) = shared prefix rows 0 .. F_b - 1 of page p
             + private rows 0 .. L_b + j of branch b
               (its L_b past tokens and its new tokens 0..j; the private
               buffer of b holds L_b + k_b rows, the new tokens last)
  z_i   = scale * <Q[b, j, h], K_i[g]>,   scale = 1 / sqrt(D) by default
  lse   = log sum_i exp(z_i)            (natural log)
  O     = sum_i exp(z_i - lse) * V_i[g]

F_b is the page's whole prefix P_p unless a fork length is given.  No other
branch's private rows are ever visible (context isolation).

The split form computes the same quantity from two partial softmaxes, one over
the shared keys and one over the private keys, and merges them with the
log-sum-exp identity; the empty set has lse = -inf and weight 0.
"""

import numpy as np

from .plan import canonical_plan


def _structure(st):
    fork = st.get("fork_len")
    return (np.asarray(st["prefix_len"]), np.asarray(st["branch_page"]),
            np.asarray(st["num_new"]), np.asarray(st["past_len"]),
            None if fork is None else np.asarray(fork))


def _softmax_attend(z, visible, values):
    """Softmax attention over the visible keys of each row.

    z [k, Hq, N] scores, visible [k, N] bool, values [N, Hq, D].
    Returns O [k, Hq, D], lse [k, Hq] and the weights [k, Hq, N]
    (zero where not visible).  A row with no visible key gets lse = -inf,
    O = 0 and all-zero weights.
    """
    zm = np.where(visible[:, None, :], z, -np.inf)
    m = zm.max(axis=2) if zm.shape[2] else np.full(zm.shape[:2], -np.inf)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    e = np.where(visible[:, None, :], np.exp(zm - m_safe[:, :, None]), 0.0)
    s = e.sum(axis=2)
    lse = np.where(finite, m_safe + np.log(np.where(finite, s, 1.0)), -np.inf)
    w = np.where(finite[:, :, None], e / np.where(finite, s, 1.0)[:, :, None], 0.0)
    O = np.einsum("jhn,nhd->jhd", w, values)
    return O, lse, w


def attention(q, shared_k, shared_v, priv_k, priv_v, structure, num_q_heads,
              num_kv_heads, scale=None, keys="all", return_weights=False):
    """Attention of every new token of every branch.

    q [T][Hq][D], shared_k/v [sum P][Hkv][D], priv_k/v [sum (L+k)][Hkv][D],
    all fp64.  ``keys`` selects the key set: "all" (the definition),
    "shared" (prefix keys only) or "private" (the branch's own keys only);
    the latter two are the partials of the split form.
    Returns (O [T][Hq][D], lse [T][Hq]) and optionally a list of per-branch
    weight arrays [k_b][Hq][N_b] over the branch's concatenated key list
    (shared rows first, then private rows).
    """
    prefix_len, branch_page, num_new, past_len, fork_len = _structure(structure)
    plan = canonical_plan(prefix_len, branch_page, num_new, past_len, fork_len)
    q = np.asarray(q, dtype=np.float64)
    T, Hq, D = q.shape
    assert Hq == num_q_heads and Hq % num_kv_heads == 0
    G = Hq // num_kv_heads
    head_to_kv = np.arange(Hq) // G
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    O = np.zeros((T, Hq, D))
    lse = np.full((T, Hq), -np.inf)
    weights = []
    for b in range(num_new.shape[0]):
        p = int(branch_page[b])
        k, L = int(num_new[b]), int(past_len[b])
        F = int(plan["fork"][b])
        s0 = int(plan["prefix_row"][p])
        r0 = int(plan["priv_row"][b])
        t0 = int(plan["q_row"][b])
        use_shared = keys in ("all", "shared")
        use_priv = keys in ("all", "private")
        Ks = np.asarray(shared_k[s0:s0 + F], np.float64) if use_shared else np.zeros((0,) + shared_k.shape[1:])
        Vs = np.asarray(shared_v[s0:s0 + F], np.float64) if use_shared else np.zeros((0,) + shared_v.shape[1:])
        Kp = np.asarray(priv_k[r0:r0 + L + k], np.float64) if use_priv else np.zeros((0,) + priv_k.shape[1:])
        Vp = np.asarray(priv_v[r0:r0 + L + k], np.float64) if use_priv else np.zeros((0,) + priv_v.shape[1:])
        Kcat = np.concatenate([Ks, Kp], axis=0)[:, head_to_kv, :]   # [N, Hq, D]
        Vcat = np.concatenate([Vs, Vp], axis=0)[:, head_to_kv, :]
        ns, npv = Ks.shape[0], Kp.shape[0]
        # token j sees every shared key and private keys 0 .. L + j
        vis = np.zeros((k, ns + npv), dtype=bool)
        vis[:, :ns] = True
        for j in range(k):
            vis[j, ns:ns + min(npv, L + j + 1)] = True
        z = scale * np.einsum("jhd,nhd->jhn", q[t0:t0 + k], Kcat)
        Ob, lb, wb = _softmax_attend(z, vis, Vcat)
        O[t0:t0 + k] = Ob
        lse[t0:t0 + k] = lb
        if return_weights:
            weights.append(wb)
    if return_weights:
        return O, lse, weights
    return O, lse


def lse_merge(parts):
    """Merge partial softmax results (O_i, lse_i) with the log-sum-exp identity.

    lse = log sum_i exp(lse_i);  O = sum_i exp(lse_i - lse) * O_i.
    Partials with lse_i = -inf carry weight 0.
    """
    lses = np.stack([np.asarray(l, np.float64) for _, l in parts])      # [n, T, Hq]
    Os = np.stack([np.asarray(o, np.float64) for o, _ in parts])         # [n, T, Hq, D]
    m = lses.max(axis=0)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    w = np.where(np.isfinite(lses), np.exp(lses - m_safe[None]), 0.0)
    s = w.sum(axis=0)
    lse = np.where(finite, m_safe + np.log(np.where(finite, s, 1.0)), -np.inf)
    coef = np.where(finite[None], w / np.where(finite, s, 1.0)[None], 0.0)
    O = np.einsum("ith,ithd->thd", coef, Os)
    return O, lse


def split_attention(q, shared_k, shared_v, priv_k, priv_v, structure, num_q_heads,
                    num_kv_heads, scale=None):
    """The method's split form: shared partial, private partial, LSE merge.

    Returns (O, lse, (O_shared, lse_shared), (O_private, lse_private)).
    """
    shared = attention(q, shared_k, shared_v, priv_k, priv_v, structure,
                       num_q_heads, num_kv_heads, scale, keys="shared")
    private = attention(q, shared_k, shared_v, priv_k, priv_v, structure,
                        num_q_heads, num_kv_heads, scale, keys="private")
    O, lse = lse_merge([shared, private])
    return O, lse, shared, private


def attention_for_batch(batch, keys="all", scale=None, return_weights=False):
    """``attention`` on a workload batch, reading its stored values exactly."""
    st = dict(prefix_len=batch.prefix_len, branch_page=batch.branch_page,
              num_new=batch.num_new, past_len=batch.past_len, fork_len=batch.fork_len)
    return attention(batch.f64("q"), batch.f64("shared_k"), batch.f64("shared_v"),
                     batch.f64("priv_k"), batch.f64("priv_v"), st,
                     batch.num_q_heads, batch.num_kv_heads, scale=scale, keys=keys,
                     return_weights=return_weights)

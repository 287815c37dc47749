"""Canonical ragged bookkeeping of one branch-parallel step (oracle side).

Test infrastructure: see the package docstring.

The method runs every active branch of every page in one batched forward
(Algorithm 1, the parallel draft over the active pool).  Packing that batch
needs, per branch b with k_b new tokens and L_b past tokens on page p:

  q_row[b]       first query token of b      = sum over b' < b of k_b'
  priv_row[b]    first private K/V row of b  = sum over b' < b of (L_b' + k_b')
  prefix_row[p]  first shared K/V row of p   = sum over p' < p of P_p'
  page_q_row[p]  first query token of page p = sum of k_b over branches of
                 earlier pages
  page_T[p]      query tokens of page p      = sum of k_b over b on page p
  visible[t]     keys seen by token t = (j-th new token of b):
                 F_b + L_b + j + 1, where F_b is the visible prefix of b
                 (the whole prefix P_p unless a fork length is given).  The
                 branch sees its shared prefix, its own L_b past tokens and its
                 new tokens 0..j (section "Layout-Coordinated Parallel
                 Decoding", paragraph on context isolation; section
                 "Integration with P-MTP", parallel verification).

All values are int64 here.  The product's planner keeps its own copies (int32
for token indices, int64 for row offsets) and must agree bit-exactly.
"""

import numpy as np


def canonical_plan(prefix_len, branch_page, num_new, past_len, fork_len=None):
    prefix_len = np.asarray(prefix_len, dtype=np.int64)
    branch_page = np.asarray(branch_page, dtype=np.int64)
    num_new = np.asarray(num_new, dtype=np.int64)
    past_len = np.asarray(past_len, dtype=np.int64)
    nb, npg = num_new.shape[0], prefix_len.shape[0]

    def exclusive_cumsum(x):
        out = np.zeros(x.shape[0], dtype=np.int64)
        if x.shape[0] > 1:
            out[1:] = np.cumsum(x[:-1])
        return out

    q_row = exclusive_cumsum(num_new)
    priv_row = exclusive_cumsum(past_len + num_new)
    prefix_row = exclusive_cumsum(prefix_len)
    page_T = np.zeros(npg, dtype=np.int64)
    np.add.at(page_T, branch_page, num_new)
    page_q_row = exclusive_cumsum(page_T)
    if fork_len is None:
        fork = prefix_len[branch_page] if nb else np.zeros(0, np.int64)
    else:
        fork = np.asarray(fork_len, dtype=np.int64)
    T = int(num_new.sum())
    visible = np.zeros(T, dtype=np.int64)
    token_branch = np.repeat(np.arange(nb, dtype=np.int64), num_new)
    token_j = np.arange(T, dtype=np.int64) - q_row[token_branch]
    visible[:] = fork[token_branch] + past_len[token_branch] + token_j + 1
    return dict(T=T, q_row=q_row, priv_row=priv_row, prefix_row=prefix_row,
                page_T=page_T, page_q_row=page_q_row, visible=visible,
                fork=fork, token_branch=token_branch, token_j=token_j,
                priv_rows_total=int((past_len + num_new).sum()),
                shared_rows_total=int(prefix_len.sum()))

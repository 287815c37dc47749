"""Pure-Python brute force of branch-parallel attention, for tiny inputs.

It enumerates, for every (branch, new token, query head), the explicit list of
(key, value) rows the token may see -- the page's shared prefix up to the
branch's fork point, then the branch's own private rows up to and including
itself -- and evaluates softmax attention with Python floats.  It uses its own
offset walk (running counters) and no numpy arithmetic, so it shares neither
code nor vectorisation with the oracle.
"""

import math


def brute_attention(q, shared_k, shared_v, priv_k, priv_v, prefix_len, branch_page,
                    num_new, past_len, Hq, Hkv, scale, fork_len=None):
    """Nested lists in, nested lists out: O[t][h][d], lse[t][h]."""
    G = Hq // Hkv
    D = len(q[0][0]) if q else 0
    # running offsets
    page_start = []
    acc = 0
    for P in prefix_len:
        page_start.append(acc)
        acc += int(P)
    O, LSE = [], []
    t = 0
    prow = 0
    for b in range(len(num_new)):
        p = int(branch_page[b])
        k = int(num_new[b])
        L = int(past_len[b])
        F = int(prefix_len[p]) if fork_len is None else int(fork_len[b])
        for j in range(k):
            rows_o, rows_l = [], []
            for h in range(Hq):
                g = h // G
                keys = []
                for i in range(F):
                    keys.append((shared_k[page_start[p] + i][g], shared_v[page_start[p] + i][g]))
                for i in range(L + j + 1):
                    keys.append((priv_k[prow + i][g], priv_v[prow + i][g]))
                z = []
                for kk, _ in keys:
                    s = 0.0
                    for d in range(D):
                        s += float(q[t][h][d]) * float(kk[d])
                    z.append(scale * s)
                m = max(z)
                tot = 0.0
                for zi in z:
                    tot += math.exp(zi - m)
                lse = m + math.log(tot)
                o = [0.0] * D
                for zi, (_, vv) in zip(z, keys):
                    w = math.exp(zi - lse)
                    for d in range(D):
                        o[d] += w * float(vv[d])
                rows_o.append(o)
                rows_l.append(lse)
            O.append(rows_o)
            LSE.append(rows_l)
            t += 1
        prow += L + k
    return O, LSE

"""P-MTP verification and drafting after a decode step, fp64 (oracle side).

Test infrastructure: see the package docstring.

Follows section "Integration with P-MTP" and Algorithm 1 (speculative
decoding and verification), with the readings recorded in the design notes:

* Verification.  Branch b fed tokens s_0 .. s_{k-1} at its k positions (s_0
  its last accepted token, s_1.. its drafts).  The LM head on the final-norm
  output at position j gives y*_j = argmax_v logit_v (ties: smallest id).
  Draft s_i is verified when y*_{i-1} = s_i; n_acc is the length of the
  longest verified prefix s_1 .. s_n, and y*_n (the model's own token at the
  first unverified position) is the bonus token that opens the next window.
* Drafting.  From the hidden state f at position n and token t = y*_n, the
  small residual MLP advances f <- f + SwiGLU(RMSNorm([f ; embed(t)]))
  W_down^T and the next drafted token is the LM head argmax on RMSNorm(f);
  repeated until the window (k tokens: the bonus token and k - 1 drafts) is
  full.
* Decision precision.  The LM head's input is the bf16 rounding of
  x = h * g_final, as in the kernels (the argmax takes its decision on that
  rounded input; the per-token RMSNorm factor is positive and does not move
  the argmax, so logits here are computed without it).  Everything else is
  fp64.
"""

import numpy as np

from .decode import _bf16_value, rms_norm, silu


def lm_logits(h, g_final, w_lm):
    """Logits (up to the positive per-token norm factor) of the LM head on the
    bf16 rounding of h * g_final."""
    x = _bf16_value(np.asarray(h, np.float64) * (1.0 if g_final is None else g_final))
    return x @ np.asarray(w_lm, np.float64).T


def argmax_first(logits):
    """Index of the largest logit of each row; ties to the smallest index."""
    return np.argmax(logits, axis=-1)


def accepted(verified_tokens, fed_tokens):
    """Longest prefix of drafts fed_tokens[1:] verified by verified_tokens[:-1]."""
    n = 0
    while n < len(fed_tokens) - 1 and verified_tokens[n] == fed_tokens[n + 1]:
        n += 1
    return n


def verify(hidden, tokens_in, num_new, g_final, w_lm):
    """(verified [T], n_acc [nb], bonus [nb], seed_row [nb], logits [T][V])."""
    logits = lm_logits(hidden, g_final, w_lm)
    ver = argmax_first(logits)
    q0 = np.concatenate([[0], np.cumsum(num_new)[:-1]]).astype(np.int64)
    n_acc = np.array([accepted(ver[q:q + k], tokens_in[q:q + k]) for q, k in zip(q0, num_new)], np.int64)
    seed = q0 + n_acc
    return ver, n_acc, ver[seed], seed, logits


def draft_mlp(f, tok, embed, w_gate, w_up, w_down, eps):
    """One residual MLP advance of the draft state f [n][H] with tokens tok [n]."""
    d = np.concatenate([f, np.asarray(embed, np.float64)[tok]], axis=-1)
    x = rms_norm(d, eps)
    m = silu(x @ np.asarray(w_gate, np.float64).T) * (x @ np.asarray(w_up, np.float64).T)
    return f + m @ np.asarray(w_down, np.float64).T


def draft(f0, tok0, steps, embed, w_gate, w_up, w_down, g_final, w_lm, eps, forced=None):
    """Drafted tokens [n][steps] after the bonus tokens tok0 and the logits of
    each step ([steps][n][V]).  forced [n][steps] (optional) replaces each
    step's drafted token before the next advance (teacher forcing, so a test
    can follow a run that took another valid argmax)."""
    f = np.asarray(f0, np.float64)
    tok = np.asarray(tok0, np.int64)
    toks, all_logits = [], []
    for s in range(steps):
        f = draft_mlp(f, tok, embed, w_gate, w_up, w_down, eps)
        logits = lm_logits(f, g_final, w_lm)
        tok = argmax_first(logits)
        toks.append(tok)
        all_logits.append(logits)
        if forced is not None:
            tok = np.asarray(forced[:, s], np.int64)
    return (np.stack(toks, axis=1) if toks else np.zeros((len(tok0), 0), np.int64)), all_logits

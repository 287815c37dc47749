"""The five synthetic workloads of the branch-parallel decode step.

Shapes follow the method's setting: a page's layout branch and its content
branches each bring k new (draft-verify) query tokens, attend over the page's
shared prefix (visual + structural context) and over their own history
(section "Layout-Coordinated Parallel Decoding", "Dynamic Branch Forking and
Efficient Context Isolation"; section "Integration with P-MTP").  The decoder
shape (hidden 1024, FFN 3072, 16 query heads, GQA, SwiGLU, RMSNorm) is the
one the "Overview" section states for the LLM decoder, with 2 KV heads and 18
layers as the synthetic stack uses.

Distributions not fixed by the workload statements are resolved as follows
(each one is listed with its reason in the design notes):
  * lognormal private lengths: mu = ln(128), sigma = 1.0 (natural log),
    length = clip(rint(exp(mu + sigma * z)), lo, hi), rint = half-to-even
  * "uniform in [a, b]" is over the integers a..b inclusive
  * the layout branch of the multi-page workload draws its length from the
    same clipped lognormal as the content branches
"""

import copy

# Each length spec is one of
#   ("fixed", n)                      the same value for every draw
#   ("list", [n0, n1, ...])           one value per branch, in branch order
#   ("uniform", lo, hi)               integers lo..hi inclusive
#   ("lognormal", median, sigma, lo, hi)

CONFIGS = {
    # Single attention layer, fp32, 1 page, 4 content branches, k = 2.
    "c1": dict(
        name="c1", dtype="f32", num_q_heads=8, num_kv_heads=2, head_dim=64,
        num_pages=1, prefix=("fixed", 256),
        layout=None,
        content_count=("fixed", 4), content_k=2,
        content_past=("list", [8, 16, 32, 32]),
    ),
    # Single attention layer, bf16, 1 page, 1 layout (k=1, L=256) + 8 content (k=4).
    "c2": dict(
        name="c2", dtype="bf16", num_q_heads=16, num_kv_heads=2, head_dim=64,
        num_pages=1, prefix=("fixed", 1024),
        layout=dict(k=1, past=("fixed", 256)),
        content_count=("fixed", 8), content_k=4,
        content_past=("uniform", 16, 256),
    ),
    # Single attention layer, bf16, dense page: 1 layout (k=1, L=512) + 32 content.
    "c3": dict(
        name="c3", dtype="bf16", num_q_heads=16, num_kv_heads=2, head_dim=64,
        num_pages=1, prefix=("fixed", 4096),
        layout=dict(k=1, past=("fixed", 512)),
        content_count=("fixed", 32), content_k=4,
        content_past=("lognormal", 128.0, 1.0, 8, 1024),
    ),
    # Full decode step of an 18-layer synthetic decoder; attention as in c3.
    "c4": dict(
        name="c4", dtype="bf16", num_q_heads=16, num_kv_heads=2, head_dim=64,
        num_pages=1, prefix=("fixed", 4096),
        layout=dict(k=1, past=("fixed", 512)),
        content_count=("fixed", 32), content_k=4,
        content_past=("lognormal", 128.0, 1.0, 8, 1024),
        model=dict(num_layers=18, hidden=1024, intermediate=3072,
                   weight_std=0.02, rms_eps=1e-6),
        # P-MTP verification and drafting: the Qwen3 vocabulary size and a
        # draft MLP as wide as the hidden state (neither is stated for the
        # parser; readings in the design notes)
        pmtp=dict(vocab=151936, draft_inner=1024, weight_std=0.02),
    ),
    # c4 with Qwen3-style attention: per-head q / k RMSNorm (gains 1 + 0.1 N(0, 1))
    # and rotary position embedding, base 10^6 (the Qwen3 family's)
    "c4q": dict(
        name="c4q", dtype="bf16", num_q_heads=16, num_kv_heads=2, head_dim=64,
        num_pages=1, prefix=("fixed", 4096),
        layout=dict(k=1, past=("fixed", 512)),
        content_count=("fixed", 32), content_k=4,
        content_past=("lognormal", 128.0, 1.0, 8, 1024),
        model=dict(num_layers=18, hidden=1024, intermediate=3072,
                   weight_std=0.02, rms_eps=1e-6, qwen3=dict(rope_theta=1e6, qk_norm=True)),
    ),
    # c3 with per-branch fork offsets (tree-shaped prefix): a content branch
    # sees the page's prefix only up to its fork point F_b, drawn uniform in
    # [1024, P] (1024 = the visual-token part every branch sees); the layout
    # branch sees the whole prefix.  Drawn after all of c3's values, so the
    # structure and values equal c3's for the same seed.
    "c3f": dict(
        name="c3f", dtype="bf16", num_q_heads=16, num_kv_heads=2, head_dim=64,
        num_pages=1, prefix=("fixed", 4096),
        layout=dict(k=1, past=("fixed", 512)),
        content_count=("fixed", 32), content_k=4,
        content_past=("lognormal", 128.0, 1.0, 8, 1024),
        fork=dict(visual=1024),
    ),
    # Ragged multi-page batch: 16 pages, prefix U[1024, 4096], 4..32 content branches.
    "c5": dict(
        name="c5", dtype="bf16", num_q_heads=16, num_kv_heads=2, head_dim=64,
        num_pages=16, prefix=("uniform", 1024, 4096),
        layout=dict(k=1, past=("lognormal", 128.0, 1.0, 8, 1024)),
        content_count=("uniform", 4, 32), content_k=4,
        content_past=("lognormal", 128.0, 1.0, 8, 1024),
    ),
}


def get_config(name, **overrides):
    """A deep copy of a named workload with top-level fields overridden."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    return cfg

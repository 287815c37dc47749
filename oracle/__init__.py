"""fp64 CPU oracle of the branch-parallel decode step -- TEST INFRASTRUCTURE.

This package is the plain, slow, obviously-correct definition that the GPU
path is checked against.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product library never does, and shares no
code with it (the only common dependency is the seeded input generator in
``workloads``, which holds none of the method's arithmetic).

Paper: "HPD-Parsing: Hierarchical Parallel Document Parsing" (arXiv
2607.18839).  What is computed:

* every branch (the layout branch and each forked content branch) attends to
  the page's shared visual + structural prefix and to its own generation
  history only, never to other branches' text (section "Layout-Coordinated
  Parallel Decoding", paragraph "Dynamic Branch Forking and Efficient Context
  Isolation");
* each branch verifies k drafted tokens in one forward, so its k new tokens
  are causal among themselves (section "Integration with P-MTP", last
  paragraph; Algorithm 1, the parallel draft f_d over the active pool);
* the decoder is a GQA / RMSNorm / SwiGLU stack (section "Overview",
  paragraph "LLM Decoder").

Modules:
  plan       canonical ragged bookkeeping (row offsets, visible-key counts)
  attention  full attention, its shared/private partials and their LSE merge
  decode     one decode step of the synthetic decoder stack
  paged      the rows a paged K/V batch describes (block-table gather)
  pmtp       P-MTP verification (LM head argmax, acceptance) and drafting

Every function is pinned by the CPU tests against something other than
itself: brute force, library routines (torch SDPA in fp64), closed forms and
invariants.  No function here is "parity unpinned".
"""
from . import attention, decode, paged, plan, pmtp  # noqa: F401

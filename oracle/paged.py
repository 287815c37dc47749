"""Paged K/V rows (oracle side).

Test infrastructure: see the package docstring.

Definition followed (section "Inference Workflow", Algorithm 1: K/V held in
fixed-size blocks, a forked branch reading its page's prefix blocks by
reference): with blocks of B rows, row i of a sequence whose block list
starts at entry `first` of the block table is pool row
blocks[first + i // B] * B + i % B.  The paged step computes exactly the
attention of the rows this mapping gathers, so the oracle gathers them into
the packed layout and evaluates the plain attention definition.
"""

import numpy as np


def sequence_rows(blocks, first, n_rows, block_rows):
    """Pool row index of rows 0..n_rows-1 of one paged sequence (int64)."""
    i = np.arange(int(n_rows), dtype=np.int64)
    b = np.asarray(blocks, dtype=np.int64)[int(first) + i // int(block_rows)]
    return b * int(block_rows) + i % int(block_rows)


def gather_packed(pool_shared_k, pool_shared_v, pool_priv_k, pool_priv_v, structure, paged):
    """The packed arrays (pages' prefixes concatenated, then each branch's
    L_b + k_b private rows) that a paged batch describes."""
    B = int(paged["block_rows"])
    sh = [sequence_rows(paged["blocks"], paged["page_block0"][p], P, B)
          for p, P in enumerate(structure["prefix_len"])]
    pr = [sequence_rows(paged["blocks"], paged["branch_block0"][b], int(L) + int(k), B)
          for b, (L, k) in enumerate(zip(structure["past_len"], structure["num_new"]))]
    sh = np.concatenate(sh) if sh else np.zeros(0, np.int64)
    pr = np.concatenate(pr) if pr else np.zeros(0, np.int64)
    return (np.asarray(pool_shared_k)[sh], np.asarray(pool_shared_v)[sh],
            np.asarray(pool_priv_k)[pr], np.asarray(pool_priv_v)[pr])

"""Mask selection from a compute budget (Section 3.3, step 2) -- test
infrastructure only.

Steps in the paper's order, for one layer with a budget given as a fraction
of the dense layer's cost:
  1. the low-rank part gets a share of the budget (rule of thumb: one
     quarter to one third); its rank is a multiple of the block size, the
     largest that fits the share;
  2. the block size of the butterfly is the hardware block size b; the
     maximum stride of the flat block butterfly is raised to fill up the rest
     of the budget.
Cost unit: weight entries (kept b x b blocks, plus r (n_out + n_in) for the
low-rank factors) against budget * n_out * n_in.  Reading: "fill up" = the
largest power-of-two stride whose total stays within the budget, at least 1
(block diagonal), and strides past the next power of two of the square side
are not considered (they keep the same blocks).
"""
from __future__ import annotations

from . import mask as om


def select(n_out: int, n_in: int, b: int, budget: float, lowrank_share: float = 0.25):
    """Returns (r, max_stride, entries)."""
    assert n_out % b == 0 and n_in % b == 0 and 0 < budget <= 1 and 0 <= lowrank_share <= 1
    dense = n_out * n_in
    total = budget * dense
    per_rank = n_out + n_in
    # step 1: rank
    r = 0
    cand = b
    while cand <= min(n_out, n_in) and cand * per_rank <= lowrank_share * total:
        r = cand
        cand += b
    # step 2: maximum stride
    s = min(n_out, n_in) // b
    top = om.next_pow2(s)
    best, best_entries = None, None
    ms = 1
    while ms <= top:
        M = om.stretch_block_mask(n_out // b, n_in // b, ms)
        entries = int(M.sum()) * b * b + r * per_rank
        if best is None or entries <= total:
            best, best_entries = ms, entries
        if entries > total:
            break
        ms *= 2
    return r, best, best_entries

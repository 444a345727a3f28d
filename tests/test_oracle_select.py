"""Pins for the oracle's budget -> (rank, maximum stride) selection (CPU only).

Hand-worked case (Section 3.3, step 2): 1024 x 1024, b = 32, budget 1/4 of
the dense entries (262144), low-rank share 1/4 (65536 entries):
r (1024 + 1024) <= 65536 gives r = 32 (a multiple of 32) using exactly 65536;
the remaining 196608 entries hold 192 blocks of 32 x 32, i.e. 6 per block row
of the 32 x 32 grid = 1 + log2(max_stride) -> max_stride = 32.  Invariants:
the chosen configuration fits the budget (unless even the block diagonal
does not), the next stride up would not, and the rank grows with the budget
(the stride need not: when a larger budget admits the next multiple of b in
rank, that rank takes budget from the butterfly).
"""
import pytest

from oracle import mask as om
from oracle import select as osel


def test_hand_worked_1024():
    r, ms, entries = osel.select(1024, 1024, 32, 0.25, 0.25)
    assert (r, ms) == (32, 32)
    assert entries == 32 * 2048 + 192 * 1024 == 262144


def test_block_diagonal_floor_and_zero_share():
    # a budget below the block diagonal still returns max_stride 1
    r, ms, entries = osel.select(1024, 1024, 32, 0.01, 0.0)
    assert (r, ms) == (0, 1) and entries == 32 * 1024
    # all budget to the butterfly: density 6/32 at stride 32
    r, ms, _ = osel.select(1024, 1024, 32, 6 / 32, 0.0)
    assert (r, ms) == (0, 32)


@pytest.mark.parametrize("n_out,n_in,b", [(3072, 768, 32), (4096, 1024, 64), (16384, 4096, 128),
                                          (1024, 1024, 32), (768, 768, 32)])
def test_budget_invariants(n_out, n_in, b):
    prev_r = 0
    for k in range(1, 41):
        budget = k / 40
        r, ms, entries = osel.select(n_out, n_in, b, budget, 0.3)
        assert r % b == 0 and r * (n_out + n_in) <= 0.3 * budget * n_out * n_in + 1e-9
        if ms > 1:
            assert entries <= budget * n_out * n_in
        top = om.next_pow2(min(n_out, n_in) // b)
        if ms < top and entries <= budget * n_out * n_in:
            M = om.stretch_block_mask(n_out // b, n_in // b, 2 * ms)
            assert int(M.sum()) * b * b + r * (n_out + n_in) > budget * n_out * n_in
        assert r >= prev_r
        prev_r = r

"""Pins for the oracle's block cover and random block patterns (CPU only).

Block cover (appendix on the cost model): pinned by its defining properties,
checked by brute force on tiny masks (it is block-aligned, contains the mask,
and no block-aligned superset has fewer nonzeros), by idempotence on
block-aligned masks (the flat block butterfly at its own block size), and by
the closed form of its expected density for an element-wise random mask of
density d: 1 - (1 - d)^(b1 b2) per block.
"""
import itertools

import numpy as np
import pytest

import synth
from oracle import mask as om


def _aligned(M, b1, b2):
    m, n = M.shape
    for i in range(0, m, b1):
        for j in range(0, n, b2):
            blk = M[i:i + b1, j:j + b2]
            if blk.any() and not blk.all():
                return False
    return True


def test_minimal_block_aligned_superset_brute_force():
    rng = np.random.default_rng(0)
    for _ in range(20):
        M = rng.random((4, 4)) < 0.3
        C = om.block_cover(M, 2, 2)
        assert _aligned(C, 2, 2) and (C >= M).all()
        best = None
        for bits in itertools.product([0, 1], repeat=4):  # every 2x2-aligned 4x4 mask
            A = np.kron(np.array(bits).reshape(2, 2), np.ones((2, 2))).astype(bool)
            if (A >= M).all():
                best = A.sum() if best is None else min(best, A.sum())
        assert C.sum() == best


@pytest.mark.parametrize("nb,b,ms", [(8, 4, 4), (24, 2, 16), (16, 8, 2)])
def test_block_aligned_mask_is_its_own_cover(nb, b, ms):
    E = om.element_mask(om.square_block_mask(nb, ms), b)
    assert np.array_equal(om.block_cover(E, b, b), E)
    assert np.array_equal(om.block_cover(E, 1, b), E)


@pytest.mark.parametrize("p,d,b", [(1, 0.0125, 32), (2, 0.025, 32), (4, 0.05, 16), (8, 0.2, 32)])
def test_expected_cover_density(p, d, b):
    """Random p x p blocks of density d under a b x b cover: a cover block
    holds (b / p)^2 independent draws, so it is kept with probability
    1 - (1 - d)^((b / p)^2)."""
    n = 1024
    M = synth.random_block_mask(n, n, p, d, seed=3)
    assert abs(M.mean() - d) < 4 * np.sqrt(d * (1 - d) / (n // p) ** 2) + 1e-12
    C = om.block_cover(M, b, b)
    expect = 1 - (1 - d) ** ((b // p) ** 2)
    nblk = (n // b) ** 2
    assert abs(C.mean() - expect) < 4 * np.sqrt(expect * (1 - expect) / nblk) + 1e-9


def test_paper_actual_densities():
    """The paper's printed actual densities for random 8x8, 16x16 and 32x32
    blocks (tests/golden/microbench_actual_density.txt) against the closed
    form at 10% expected density, and against the oracle's cover of one
    seeded 4096 x 4096 draw."""
    import os
    rows = []
    for line in open(os.path.join(os.path.dirname(__file__), "golden", "microbench_actual_density.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            p, pct = line.split()
            rows.append((int(p), float(pct) / 100))
    for p, printed in rows:
        closed = 1 - 0.9 ** ((32 // p) ** 2)
        assert abs(closed - printed) < 0.005, (p, closed, printed)
        C = om.block_cover(synth.random_block_mask(4096, 4096, p, 0.10, seed=0), 32, 32)
        assert abs(C.mean() - printed) < 0.01, (p, C.mean(), printed)

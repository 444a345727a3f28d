"""Pins for the oracle's attention mask with the global component (CPU only).

The appendix on method details adds to the flat block butterfly attention
mask a block-aligned "global" component: horizontal and vertical stripes of
width w, whose support carries matrices of rank at most 2w.  Pinned against a
hand-derived fixture, the rank bound (numerically, on random values), the
reduction to the plain butterfly mask at zero width, symmetry and row counts,
and attention semantics: a global query row is exactly dense softmax
attention (scipy) over all keys.
"""
import os

import numpy as np
import pytest
from scipy.special import softmax

from oracle import attention as oa
from oracle import mask as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_n4_ms2_g1():
    rows = {}
    for line in open(os.path.join(GOLDEN, "attention_global_n4_ms2_g1.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        i, cols = line.split(":")
        rows[int(i)] = [int(c) for c in cols.split()]
    M = om.attention_block_mask(4, 2, 1)
    for i in range(4):
        assert list(np.nonzero(M[i])[0]) == rows[i]


@pytest.mark.parametrize("nb,b,g", [(8, 4, 1), (8, 4, 2), (16, 2, 3), (6, 3, 1)])
def test_global_component_rank_at_most_2w(nb, b, g):
    """Random values on the element support of the stripes: rank 2w exactly
    (generic values reach the bound when 2w <= n)."""
    rng = np.random.default_rng(nb * 100 + g)
    G = om.element_mask(om.global_block_mask(nb, g), b)
    A = np.where(G, rng.standard_normal(G.shape), 0.0)
    w = g * b
    r = np.linalg.matrix_rank(A)
    assert r <= 2 * w
    assert r == min(2 * w, nb * b)


@pytest.mark.parametrize("nb,ms", [(8, 8), (16, 4), (24, 16), (64, 64)])
def test_zero_width_is_butterfly(nb, ms):
    assert np.array_equal(om.attention_block_mask(nb, ms, 0), om.square_block_mask(nb, ms))


@pytest.mark.parametrize("nb,ms,g", [(16, 16, 1), (64, 64, 1), (64, 64, 2), (24, 8, 3)])
def test_symmetry_and_row_counts(nb, ms, g):
    M = om.attention_block_mask(nb, ms, g)
    F = om.square_block_mask(nb, ms)
    assert np.array_equal(M, M.T)
    for i in range(nb):
        if i < g:
            assert M[i].sum() == nb
        else:
            assert M[i].sum() == F[i].sum() + sum(1 for j in range(g) if not F[i, j])


def test_global_query_is_dense_attention():
    """A query in the horizontal stripe sees every key: its output row is the
    dense softmax attention row; every query gives the vertical stripe's keys
    nonzero weight."""
    rng = np.random.default_rng(7)
    nb, b, d, g = 8, 4, 4, 1
    S = nb * b
    Q, K, V = (rng.standard_normal((S, d)) for _ in range(3))
    Mel = om.element_mask(om.attention_block_mask(nb, 4, g), b)
    O, _, P = oa.forward_head(Q, K, V, Mel, 0.5)
    dense = softmax(Q @ K.T * 0.5, axis=1) @ V
    assert np.allclose(O[: g * b], dense[: g * b])
    assert (P[:, : g * b] > 0).all()
    assert not np.allclose(O[g * b:], dense[g * b:])

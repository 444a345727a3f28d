"""Pins for the oracle's mask construction (CPU only).

The oracle builds the flat block butterfly mask literally from the factor
definitions; these tests pin it against a hand-derived fixture, the XOR rule
stated by the workloads, the factor nonzero count and the per-row count of the
flat pattern.
"""
import math
import os

import numpy as np
import pytest

from oracle import mask as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def xor_rule(s, ms):
    """Kept iff i == j or i XOR j is a power of two smaller than ms."""
    F = np.zeros((s, s), bool)
    for i in range(s):
        for j in range(s):
            x = i ^ j
            F[i, j] = (x == 0) or (x & (x - 1) == 0 and x < ms)
    return F


def test_golden_n8_ms8():
    rows = {}
    for line in open(os.path.join(GOLDEN, "flat_butterfly_n8_ms8.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        i, cols = line.split(":")
        rows[int(i)] = [int(c) for c in cols.split()]
    F = om.flat_butterfly_support(8, 8)
    for i in range(8):
        assert list(np.nonzero(F[i])[0]) == rows[i]


@pytest.mark.parametrize("s", [1, 2, 3, 5, 8, 16, 24, 31, 32, 33, 64, 100, 128])
def test_factor_union_equals_xor_rule(s):
    ms = 1
    while ms <= 256:
        assert np.array_equal(om.square_block_mask(s, ms), xor_rule(s, ms)), (s, ms)
        ms *= 2


@pytest.mark.parametrize("n", [2, 4, 8, 16, 64])
def test_factor_has_two_nonzeros_per_row(n):
    k = 2
    while k <= n:
        S = om.factor_matrix_support(n, k)
        assert (S.sum(axis=1) == 2).all() and S.sum() == 2 * n
        k *= 2


@pytest.mark.parametrize("s", [2, 4, 16, 32, 64, 128])
def test_power_of_two_row_and_column_counts(s):
    ms = 1
    while ms <= s:
        F = om.square_block_mask(s, ms)
        c = 1 + int(math.log2(ms))
        assert (F.sum(axis=1) == c).all() and (F.sum(axis=0) == c).all()
        assert np.array_equal(F, F.T)
        ms *= 2


def test_special_cases():
    assert np.array_equal(om.square_block_mask(16, 1), np.eye(16, dtype=bool))
    assert om.square_block_mask(1, 8).all()
    assert om.square_block_mask(2, 2).all() and om.square_block_mask(2, 64).all()
    # strides beyond the square are clamped: same as max stride = side
    assert np.array_equal(om.square_block_mask(16, 1024), om.square_block_mask(16, 16))


@pytest.mark.parametrize("n_out,n_in,b,ms,nnzb,per_row", [
    (1024, 1024, 32, 32, 192, {6}),          # 32 x 32 block grid
    (3072, 768, 32, 16, 448, {4, 5}),        # 24-side square tiled 4x
    (4096, 1024, 64, 16, 320, {5}),
    (1024, 4096, 64, 16, 320, {20}),         # tiled along the input dim
    (4096, 4096, 64, 64, 448, {7}),          # attention score mask
    (16384, 4096, 128, 32, 768, {6}),
    (16384, 4096, 64, 32, 1536, {6}),
    (16384, 4096, 32, 32, 3072, {6}),
])
def test_workload_masks(n_out, n_in, b, ms, nnzb, per_row):
    M, (row_ptr, col_idx, col_ptr, row_idx, tperm) = om.layout(n_out, n_in, b, ms)
    assert M.sum() == nnzb and row_ptr[-1] == nnzb
    assert set(np.diff(row_ptr).tolist()) == per_row
    # tiled copies along the longer dim share their column (row) sets
    s = min(M.shape)
    for i in range(M.shape[0]):
        assert np.array_equal(M[i], M[i % s]) or M.shape[0] == s
    # the 24-side square: rows 0-15 keep 5 blocks, rows 16-23 keep 4
    if n_out == 3072:
        assert (M[:16].sum(1) == 5).all() and (M[16:24].sum(1) == 4).all()


def test_block_csr_roundtrip():
    rng = np.random.default_rng(3)
    for _ in range(20):
        M = rng.random((rng.integers(1, 12), rng.integers(1, 12))) < 0.4
        row_ptr, col_idx, col_ptr, row_idx, tperm = om.block_csr(M)
        R = np.zeros_like(M)
        for i in range(M.shape[0]):
            for p in range(row_ptr[i], row_ptr[i + 1]):
                R[i, col_idx[p]] = True
        assert np.array_equal(R, M)
        for j in range(M.shape[1]):
            for p in range(col_ptr[j], col_ptr[j + 1]):
                i = row_idx[p]
                q = tperm[p]
                assert col_idx[q] == j and row_ptr[i] <= q < row_ptr[i + 1]
        assert sorted(tperm.tolist()) == list(range(int(M.sum())))


def test_element_mask():
    F = om.square_block_mask(4, 2)
    E = om.element_mask(F, 3)
    assert E.shape == (12, 12)
    for e in range(12):
        for f in range(12):
            assert E[e, f] == F[e // 3, f // 3]

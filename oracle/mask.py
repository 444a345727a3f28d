"""Flat block butterfly mask, built literally from the factor definitions.

Test infrastructure only (see package docstring).

Notation follows Section 3 of the paper.  Everything here works in *block
units*: a block butterfly factor of size k*b with block size b has, in block
units, the support of a k x k butterfly factor, so the element mask is the
block mask with every entry expanded to a dense b x b block (the diagonal
blocks of the identity term are dense b x b blocks, like the blocks D_{i,j} of
the factors).
"""
from __future__ import annotations

import numpy as np


def next_pow2(n: int) -> int:
    p = 1
    while p < n:
        p *= 2
    return p


def factor_support(k: int) -> np.ndarray:
    """Support of one butterfly factor B_k (block units, k x k).

    Definition of the block butterfly factor: B_k = [[D1, D2], [D3, D4]],
    each D_i a (k/2) x (k/2) block-diagonal matrix.  So block (p, q) is
    nonzero iff p and q fall in quadrants (a, c) and share the same diagonal
    position t inside them: p = a*k/2 + t, q = c*k/2 + t.
    """
    assert k >= 2 and (k & (k - 1)) == 0
    h = k // 2
    S = np.zeros((k, k), dtype=bool)
    for a in range(2):
        for c in range(2):
            for t in range(h):
                S[a * h + t, c * h + t] = True
    return S


def factor_matrix_support(n: int, k: int) -> np.ndarray:
    """Support of the butterfly factor matrix B_k^{(n)} (block units, n x n).

    Definition of the block butterfly factor matrix: block-diagonal with n/k
    copies of a size-k factor.
    """
    assert n % k == 0
    S = np.zeros((n, n), dtype=bool)
    f = factor_support(k)
    for g in range(n // k):
        S[g * k:(g + 1) * k, g * k:(g + 1) * k] = f
    return S


def flat_butterfly_support(n: int, max_stride: int) -> np.ndarray:
    """Support of I + sum_{k=2,4,...,max_stride} B_k^{(n)} (definition of flat
    butterfly of maximum stride k), n a power of two.  Strides larger than n
    have no factor matrix and are skipped (the product form stops at B_n)."""
    assert n >= 1 and (n & (n - 1)) == 0
    assert max_stride >= 1 and (max_stride & (max_stride - 1)) == 0
    S = np.eye(n, dtype=bool)
    k = 2
    while k <= min(max_stride, n):
        S |= factor_matrix_support(n, k)
        k *= 2
    return S


def square_block_mask(s: int, max_stride: int) -> np.ndarray:
    """s x s flat block butterfly block mask.

    For s not a power of two (the paper's factors need a power-of-two size),
    the pattern of the next power of two is cropped to s x s: a partner that
    falls outside the square is dropped.
    """
    P = next_pow2(s)
    return flat_butterfly_support(P, max_stride)[:s, :s].copy()


def stretch_block_mask(nb_out: int, nb_in: int, max_stride: int) -> np.ndarray:
    """Rectangular block mask (Appendix on method details, rectangular matrices:
    the square mask is "stretched").  Reading used here: the square side is
    s = min(nb_out, nb_in) and the square pattern is repeated (tiled) along the
    longer dimension, i.e. kept(i, j) = F[i mod s, j mod s]."""
    s = min(nb_out, nb_in)
    F = square_block_mask(s, max_stride)
    M = np.zeros((nb_out, nb_in), dtype=bool)
    for i in range(nb_out):
        for j in range(nb_in):
            M[i, j] = F[i % s, j % s]
    return M


def element_mask(block_mask: np.ndarray, b: int) -> np.ndarray:
    """Expand a block mask to the element mask (each kept block dense b x b)."""
    return np.kron(block_mask.astype(np.int8), np.ones((b, b), np.int8)).astype(bool)


def block_csr(block_mask: np.ndarray):
    """Block-CSR of a block mask: kept blocks in row-major order (block row
    ascending, then block column ascending), plus its transpose (CSC).

    Returns int32 arrays (row_ptr, col_idx, col_ptr, row_idx, tperm), where
    tperm[p] is the CSR position of the p-th block in CSC order.
    """
    nbr, nbc = block_mask.shape
    row_ptr = [0]
    col_idx = []
    pos = {}
    for i in range(nbr):
        for j in range(nbc):
            if block_mask[i, j]:
                pos[(i, j)] = len(col_idx)
                col_idx.append(j)
        row_ptr.append(len(col_idx))
    col_ptr = [0]
    row_idx = []
    tperm = []
    for j in range(nbc):
        for i in range(nbr):
            if block_mask[i, j]:
                row_idx.append(i)
                tperm.append(pos[(i, j)])
        col_ptr.append(len(row_idx))
    as32 = lambda v: np.asarray(v, dtype=np.int32)
    return as32(row_ptr), as32(col_idx), as32(col_ptr), as32(row_idx), as32(tperm)


def layout(n_out: int, n_in: int, b: int, max_stride: int):
    """Block mask and block-CSR for an n_out x n_in weight with block size b."""
    assert n_out % b == 0 and n_in % b == 0
    M = stretch_block_mask(n_out // b, n_in // b, max_stride)
    return M, block_csr(M)


def global_block_mask(nb: int, global_blocks: int) -> np.ndarray:
    """The "global" component of the attention mask (appendix on method
    details, low-rank in attention), in block units: a horizontal stripe (the
    first `global_blocks` block rows: those queries attend to every key) and
    a vertical stripe (the first `global_blocks` block columns: every query
    attends to those keys).  With stripe width w = global_blocks * b, any
    matrix supported on it is the sum of one supported on w rows and one on
    w columns, so its rank is at most 2w: the restricted low-rank term.
    Reading: the stripes sit at the start of the sequence."""
    assert 0 <= global_blocks <= nb
    G = np.zeros((nb, nb), dtype=bool)
    G[:global_blocks, :] = True
    G[:, :global_blocks] = True
    return G


def attention_block_mask(nb: int, max_stride: int, global_blocks: int = 0) -> np.ndarray:
    """Attention score mask: flat block butterfly (square, nb x nb block
    units) plus the global stripes, as a union of supports (the paper adds
    the sparse and the low-rank parts)."""
    return square_block_mask(nb, max_stride) | global_block_mask(nb, global_blocks)


def attention_layout(seq: int, b: int, max_stride: int, global_blocks: int = 0):
    """Block mask and block-CSR of the attention mask for sequence length seq."""
    assert seq % b == 0
    M = attention_block_mask(seq // b, max_stride, global_blocks)
    return M, block_csr(M)


def block_cover(M: np.ndarray, b1: int, b2: int) -> np.ndarray:
    """(b1, b2)-block cover of a 0/1 mask (definition in the appendix on the
    cost model: the block-aligned mask with the fewest nonzeros that
    contains M): every b1 x b2 block that holds a nonzero becomes all ones.
    The shape must be a multiple of (b1, b2)."""
    m, n = M.shape
    assert m % b1 == 0 and n % b2 == 0
    C = np.zeros_like(M, dtype=bool)
    for i in range(0, m, b1):
        for j in range(0, n, b2):
            if M[i:i + b1, j:j + b2].any():
                C[i:i + b1, j:j + b2] = True
    return C


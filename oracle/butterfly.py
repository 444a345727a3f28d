"""Residual butterfly product and its flat first-order term.

Test infrastructure only.  Section 3 (residual form of a butterfly matrix):
    M = (I + lam B_n)(I + lam B_{n/2}) ... (I + lam B_2)
and the flat butterfly  I + lam (B_2 + B_4 + ... + B_n)  is its first-order
term in lam.  The second-order term is sum over ordered pairs (a left of c in
the product) of B_a B_c.
"""
from __future__ import annotations

import numpy as np

from .mask import factor_matrix_support, element_mask


def random_factor_matrix(n: int, k: int, b: int, rng, fro: float | None = 1.0):
    """Dense (n*b) x (n*b) matrix with the support of B_k^{(n, b)} and
    N(0, 1) values on it, optionally scaled to the given Frobenius norm."""
    S = element_mask(factor_matrix_support(n, k), b)
    A = np.where(S, rng.standard_normal(S.shape), 0.0)
    if fro is not None:
        A *= fro / np.linalg.norm(A)
    return A


def strides(n: int, max_stride: int):
    """Strides 2, 4, ..., min(max_stride, n)."""
    out, k = [], 2
    while k <= min(max_stride, n):
        out.append(k)
        k *= 2
    return out


def residual_product(factors: dict, lam: float, dim: int) -> np.ndarray:
    """(I + lam B_kmax) ... (I + lam B_2), largest stride leftmost."""
    M = np.eye(dim)
    for k in sorted(factors, reverse=True):
        M = M @ (np.eye(dim) + lam * factors[k])
    return M


def flat(factors: dict, lam: float, dim: int) -> np.ndarray:
    """I + lam * sum_k B_k (definition of flat butterfly)."""
    return np.eye(dim) + lam * sum(factors.values())


def second_order(factors: dict, dim: int) -> np.ndarray:
    """Coefficient of lam^2 in the residual product: sum over pairs of factors
    taken in product order (larger stride on the left)."""
    ks = sorted(factors, reverse=True)
    C = np.zeros((dim, dim))
    for ia in range(len(ks)):
        for ic in range(ia + 1, len(ks)):
            C += factors[ks[ia]] @ factors[ks[ic]]
    return C

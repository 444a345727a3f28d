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


def product_layer_forward(X, factors):
    """The product form as a layer on token rows.  `factors` lists dense
    F_1 .. F_L in application order (smallest stride first), so the matrix is
    M = F_L ... F_1 (Section 3.2's product of factors, each a general matrix
    on the support of its I + B_k) and Y = X M^T, computed factor by factor:
    x_0 = X, x_f = x_{f-1} F_f^T.  Returns (Y, [x_0, ..., x_{L-1}]), the
    input of every factor."""
    xs, x = [], X
    for F in factors:
        xs.append(x)
        x = x @ F.T
    return x, xs


def product_layer_backward(xs, factors, supports, dY):
    """Gradients of L = <dY, Y> for product_layer_forward: g_L = dY,
    g_{f-1} = g_f F_f, and each factor's gradient restricted to its support,
    dF_f = (g_f^T x_{f-1}) o S_f (the masked-gradient rule of the appendix on
    gradient computation, applied to each factor).  `supports` holds the
    element masks S_f.  Returns (dX, [dF_1 .. dF_L], [g_1 .. g_L])."""
    L = len(factors)
    g = dY
    dF, gs = [None] * L, [None] * L
    for f in range(L - 1, -1, -1):
        gs[f] = g
        dF[f] = (g.T @ xs[f]) * supports[f]
        g = g @ factors[f]
    return g, dF, gs


def product_factor_mask(nb: int, L: int) -> np.ndarray:
    """Block mask of all factors' gradients at once: an (L nb) x (L nb)
    block-diagonal whose f-th diagonal block is the support of the factor of
    stride 2^(f+1) (block units), so that the gradients of every factor are
    one masked product of the stacked output gradients and inputs."""
    from .mask import factor_matrix_support
    M = np.zeros((L * nb, L * nb), dtype=bool)
    for f in range(L):
        M[f * nb:(f + 1) * nb, f * nb:(f + 1) * nb] = factor_matrix_support(nb, 2 ** (f + 1))
    return M

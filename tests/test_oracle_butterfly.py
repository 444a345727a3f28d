"""Pin: the flat butterfly is the first-order term of the residual butterfly
product, with an O(lam^2) remainder bounded as in the flat-approximation
theorem (Section 4)."""
import math

import numpy as np
import pytest

from oracle import butterfly as ob
from oracle import mask as om


@pytest.mark.parametrize("n,b", [(4, 1), (8, 1), (16, 1), (4, 2), (8, 2)])
def test_flat_is_first_order_term(n, b):
    rng = np.random.default_rng(n * 10 + b)
    dim = n * b
    F = {k: ob.random_factor_matrix(n, k, b, rng, fro=1.0) for k in ob.strides(n, n)}
    C2 = ob.second_order(F, dim)
    ratios, resid, lams = [], [], [1e-1, 1e-2, 1e-3, 1e-4]
    for lam in lams:
        E = ob.residual_product(F, lam, dim) - ob.flat(F, lam, dim)
        ratios.append(np.linalg.norm(E) / lam ** 2)
        resid.append(np.linalg.norm(E / lam ** 2 - C2))
    # ||E|| / lam^2 settles to ||C2||; the remainder of E / lam^2 is O(lam)
    for a, c in zip(ratios[1:], ratios[2:]):
        assert abs(a / c - 1) < 0.15
    assert abs(ratios[-1] / np.linalg.norm(C2) - 1) < 1e-3
    # (with only two factors the lam^2 term is the whole remainder, so the
    # residual is roundoff, about 1e-15 / lam^2)
    for a, c, lam in zip(resid, resid[1:], lams[1:]):
        assert c < a * 0.2 + 1e-14 / lam ** 2
    # derivative of the product at lam = 0 is the sum of the factors
    h = 1e-6
    D = (ob.residual_product(F, h, dim) - ob.residual_product(F, -h, dim)) / (2 * h)
    assert np.allclose(D, sum(F.values()), atol=1e-8)


@pytest.mark.parametrize("n", [4, 8, 16, 32])
def test_theorem_bound(n):
    """With |lam| <= c sqrt(eps) / (log n * B_max), c = 1/2: ||E||_F <= eps."""
    rng = np.random.default_rng(n)
    F = {k: ob.random_factor_matrix(n, k, 1, rng, fro=1.0) for k in ob.strides(n, n)}
    Bmax = max(np.linalg.norm(v) for v in F.values())
    for eps in [1e-2, 1e-4]:
        lam = 0.5 * math.sqrt(eps) / (math.log2(n) * Bmax)
        E = ob.residual_product(F, lam, n) - ob.flat(F, lam, n)
        assert np.linalg.norm(E) <= eps


@pytest.mark.parametrize("n,ms", [(8, 2), (8, 4), (8, 8), (16, 4), (16, 16)])
def test_flat_support_is_the_mask(n, ms):
    rng = np.random.default_rng(1)
    F = {k: ob.random_factor_matrix(n, k, 1, rng, fro=None) for k in ob.strides(n, ms)}
    Mf = ob.flat(F, 0.3, n)
    assert np.array_equal(Mf != 0, om.flat_butterfly_support(n, ms))

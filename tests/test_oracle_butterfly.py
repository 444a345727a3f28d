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


def _product_case(nb, b, L, T, seed):
    rng = np.random.default_rng(seed)
    dim = nb * b
    ks = [2 ** (f + 1) for f in range(L)]
    F = [ob.random_factor_matrix(nb, k, b, rng, fro=None) for k in ks]
    S = [om.element_mask(om.factor_matrix_support(nb, k), b) for k in ks]
    X = rng.standard_normal((T, dim))
    dY = rng.standard_normal((T, dim))
    return F, S, X, dY


@pytest.mark.parametrize("nb,b,L", [(8, 2, 3), (4, 3, 2), (8, 1, 1)])
def test_product_layer_gradients_by_finite_differences(nb, b, L):
    """L = <dY, Y> is linear in X and in each factor separately, so central
    differences give the gradients to roundoff."""
    F, S, X, dY = _product_case(nb, b, L, 5, seed=nb + b + L)
    Y, xs = ob.product_layer_forward(X, F)
    dX, dF, _ = ob.product_layer_backward(xs, F, S, dY)
    loss = lambda X_, F_: float(np.sum(dY * ob.product_layer_forward(X_, F_)[0]))
    h, rng = 1e-3, np.random.default_rng(7)
    for _ in range(6):
        i, j = rng.integers(0, X.shape[0]), rng.integers(0, X.shape[1])
        E = np.zeros_like(X)
        E[i, j] = h
        fd = (loss(X + E, F) - loss(X - E, F)) / (2 * h)
        assert abs(fd - dX[i, j]) < 1e-8 * max(1.0, abs(fd))
    for f in range(L):
        rows, cols = np.nonzero(S[f])
        for q in rng.integers(0, len(rows), 5):
            Fp = [x.copy() for x in F]
            Fm = [x.copy() for x in F]
            Fp[f][rows[q], cols[q]] += h
            Fm[f][rows[q], cols[q]] -= h
            fd = (loss(X, Fp) - loss(X, Fm)) / (2 * h)
            assert abs(fd - dF[f][rows[q], cols[q]]) < 1e-8 * max(1.0, abs(fd))
        assert not np.any(dF[f][~S[f]])  # nothing outside the support


def test_product_layer_single_factor_is_the_linear_layer():
    """One factor: the product layer is the sparse layer with that factor as
    its masked weight (oracle.linear, a separate implementation)."""
    from oracle import linear as ol
    F, S, X, dY = _product_case(8, 4, 1, 6, seed=3)
    Y, xs = ob.product_layer_forward(X, F)
    dX, dF, gs = ob.product_layer_backward(xs, F, S, dY)
    Yl, _ = ol.forward(X, F[0])
    g = ol.backward(X, F[0], S[0], dY)
    assert np.allclose(Y, Yl, atol=1e-12) and np.allclose(dX, g["dX"], atol=1e-12)
    assert np.allclose(dF[0], g["dW"], atol=1e-12) and np.array_equal(gs[0], dY)


@pytest.mark.parametrize("nb", [4, 8, 16])
def test_product_layer_residual_form(nb):
    """Factors I + lam B_k applied smallest stride first give X M^T with the
    residual product M of Section 3.2, and differ from the flat butterfly
    layer by O(lam^2)."""
    rng = np.random.default_rng(nb)
    B = {k: ob.random_factor_matrix(nb, k, 1, rng, fro=1.0) for k in ob.strides(nb, nb)}
    X = rng.standard_normal((7, nb))
    errs = []
    for lam in (1e-2, 1e-3):
        F = [np.eye(nb) + lam * B[k] for k in sorted(B)]
        Y, _ = ob.product_layer_forward(X, F)
        assert np.allclose(Y, X @ ob.residual_product(B, lam, nb).T, atol=1e-12)
        errs.append(np.linalg.norm(Y - X @ ob.flat(B, lam, nb).T))
    assert 70 < errs[0] / errs[1] < 130  # second order: 10x smaller lam, ~100x smaller gap


def test_product_factor_mask_rows_and_blocks():
    """Each diagonal block of the stacked mask is its factor's support: two
    blocks per row (p and p XOR 2^f), nothing off the diagonal blocks."""
    nb, L = 16, 4
    M = ob.product_factor_mask(nb, L)
    assert M.sum(axis=1).tolist() == [2] * (L * nb)
    for f in range(L):
        for p in range(nb):
            row = M[f * nb + p]
            assert set(np.nonzero(row)[0]) == {f * nb + p, f * nb + (p ^ 2 ** f)}

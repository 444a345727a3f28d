"""Pins for the oracle's block-sparse attention (CPU only): all-kept mask is
dense softmax attention (scipy softmax), block-diagonal mask is independent
per-block attention, log-sum-exp matches scipy, and the backward matches
finite differences of L = <dO, O>."""
import numpy as np
import pytest
from scipy.special import logsumexp, softmax

from oracle import attention as oa
from oracle import mask as om


def test_all_kept_is_dense_attention():
    rng = np.random.default_rng(0)
    S, d, b = 8, 4, 4
    M, _ = om.layout(S, S, b, 2)
    assert M.all()
    Q, K, V = (rng.standard_normal((S, d)) for _ in range(3))
    O, lse, _ = oa.forward_head(Q, K, V, om.element_mask(M, b), 0.5)
    ref = softmax(Q @ K.T * 0.5, axis=1) @ V
    assert np.allclose(O, ref)
    assert np.allclose(lse, logsumexp(Q @ K.T * 0.5, axis=1))


def test_block_diagonal_is_per_block_attention():
    rng = np.random.default_rng(1)
    S, d, b = 16, 4, 4
    M, _ = om.layout(S, S, b, 1)
    Q, K, V = (rng.standard_normal((S, d)) for _ in range(3))
    O, _, P = oa.forward_head(Q, K, V, om.element_mask(M, b), 0.3)
    for i in range(S // b):
        sl = slice(i * b, (i + 1) * b)
        ref = softmax(Q[sl] @ K[sl].T * 0.3, axis=1) @ V[sl]
        assert np.allclose(O[sl], ref)
    assert np.allclose(P.sum(1), 1.0)


def test_masked_entries_have_zero_probability():
    rng = np.random.default_rng(2)
    S, d, b = 32, 4, 4
    M, _ = om.layout(S, S, b, 4)
    Mel = om.element_mask(M, b)
    Q, K, V = (rng.standard_normal((S, d)) for _ in range(3))
    _, lse, P = oa.forward_head(Q, K, V, Mel, 0.5)
    assert (P[~Mel] == 0).all() and np.allclose(P.sum(1), 1)
    Sc = Q @ K.T * 0.5
    for r in range(S):
        assert np.isclose(lse[r], logsumexp(Sc[r][Mel[r]]))


@pytest.mark.parametrize("ms", [2, 4])
def test_finite_differences(ms):
    rng = np.random.default_rng(3)
    S, d, b = 8, 3, 2
    M, _ = om.layout(S, S, b, ms)
    Mel = om.element_mask(M, b)
    Q, K, V, dO = (rng.standard_normal((S, d)) for _ in range(4))
    scale = 0.7
    dQ, dK, dV = oa.backward_head(Q, K, V, Mel, scale, dO)
    L = lambda Q_, K_, V_: float((dO * oa.forward_head(Q_, K_, V_, Mel, scale)[0]).sum())
    h = 1e-6
    for G_ref, A, pos in [(dQ, Q, 0), (dK, K, 1), (dV, V, 2)]:
        G = np.zeros_like(A)
        for e in np.ndindex(A.shape):
            ap, am = [Q, K, V], [Q, K, V]
            Ap, Am = A.copy(), A.copy()
            Ap[e] += h
            Am[e] -= h
            ap[pos], am[pos] = Ap, Am
            G[e] = (L(*ap) - L(*am)) / (2 * h)
        assert np.allclose(G_ref, G, atol=1e-7)

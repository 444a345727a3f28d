"""Pins for the oracle's layer with the learnable mixing weight gamma
(Section 3.3, model sparsification: W = gamma B + (1 - gamma) U V^T), CPU only.

Pinned by central finite differences of L = <dY, Y> with respect to every
input including gamma (L is linear in each argument, so the differences are
exact up to rounding), by the endpoints (gamma = 1 is the sparse layer alone,
gamma = 0 the low-rank product alone, each against the unmixed oracle), by
linearity in gamma, and by the mixed weight written out as a dense matrix
(numpy matmul against X).
"""
import numpy as np
import pytest

from oracle import linear as ol
from oracle import mask as om


def _case(seed=0, T=6, n_out=8, n_in=12, b=2, ms=2, r=2):
    rng = np.random.default_rng(seed)
    M, _ = om.layout(n_out, n_in, b, ms)
    Mel = om.element_mask(M, b)
    X = rng.standard_normal((T, n_in))
    Wd = rng.standard_normal((n_out, n_in)) * Mel
    U = rng.standard_normal((n_out, r))
    V = rng.standard_normal((r, n_in))
    dY = rng.standard_normal((T, n_out))
    return X, Wd, Mel, U, V, dY


@pytest.mark.parametrize("gamma", [0.0, 0.3, 1.0])
def test_finite_differences(gamma):
    X, Wd, Mel, U, V, dY = _case()
    g = ol.backward_mixed(X, Wd, Mel, dY, U, V, gamma)
    L = lambda X, Wd, U, V, gm: np.sum(dY * ol.forward_mixed(X, Wd, U, V, gm)[0])
    h = 1e-6
    for name, arr, mask in [("dX", X, None), ("dW", Wd, Mel), ("dU", U, None), ("dV", V, None)]:
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            if mask is not None and not mask[idx]:
                continue
            e = np.zeros_like(arr)
            e[idx] = h
            args = {"dX": (X, Wd, U, V), "dW": (X, Wd, U, V), "dU": (X, Wd, U, V), "dV": (X, Wd, U, V)}[name]
            a = list(args)
            pos = {"dX": 0, "dW": 1, "dU": 2, "dV": 3}[name]
            a[pos] = arr + e
            lp = L(*a, gamma)
            a[pos] = arr - e
            lm = L(*a, gamma)
            num[idx] = (lp - lm) / (2 * h)
        assert np.allclose(g[name], num, atol=1e-6), name
    dg = (L(X, Wd, U, V, gamma + h) - L(X, Wd, U, V, gamma - h)) / (2 * h)
    assert abs(g["dgamma"] - dg) < 1e-6


def test_endpoints_reduce_to_unmixed_layer():
    X, Wd, Mel, U, V, dY = _case(1)
    Y1, _ = ol.forward_mixed(X, Wd, U, V, 1.0)
    assert np.allclose(Y1, ol.forward(X, Wd)[0])
    Y0, _ = ol.forward_mixed(X, Wd, U, V, 0.0)
    assert np.allclose(Y0, ol.forward(X, np.zeros_like(Wd), U, V)[0])
    g1 = ol.backward_mixed(X, Wd, Mel, dY, U, V, 1.0)
    assert np.allclose(g1["dX"], ol.backward(X, Wd, Mel, dY)["dX"])
    assert np.allclose(g1["dU"], 0) and np.allclose(g1["dV"], 0)


def test_linear_in_gamma_and_dense_weight():
    X, Wd, Mel, U, V, dY = _case(2)
    Y0, Y1 = ol.forward_mixed(X, Wd, U, V, 0.0)[0], ol.forward_mixed(X, Wd, U, V, 1.0)[0]
    for gm in [0.25, 0.6, -0.5, 1.7]:
        Yg = ol.forward_mixed(X, Wd, U, V, gm)[0]
        assert np.allclose(Yg, gm * Y1 + (1 - gm) * Y0)
        assert np.allclose(Yg, np.matmul(X, ol.mixed_weight(Wd, U, V, gm).T))
        g = ol.backward_mixed(X, Wd, Mel, dY, U, V, gm)
        assert np.isclose(g["dgamma"], np.sum(dY * (Y1 - Y0)))

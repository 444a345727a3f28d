"""Pins for the oracle's sparse + low-rank linear layer (CPU only):
hand-worked fixture, finite differences of L = <dY, Y>, integer exactness of
the block loop vs the dense masked product, and special cases that reduce to
library routines."""
import os

import numpy as np
import pytest

from oracle import linear as ol
from oracle import mask as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load_worked():
    d = {}
    for line in open(os.path.join(GOLDEN, "linear_worked_n4.txt")):
        if line.startswith("#") or ":" not in line:
            continue
        k, v = line.split(":")
        d[k.strip()] = np.array([float(x) for x in v.split()])
    return d


def test_worked_example():
    g = _load_worked()
    M, (row_ptr, col_idx, *_r) = om.layout(4, 4, 1, 2)
    Mel = om.element_mask(M, 1)
    W = g["W"].reshape(4, 4) * Mel
    X, U, V = g["X"].reshape(1, 4), g["U"].reshape(4, 1), g["V"].reshape(1, 4)
    Y, _ = ol.forward(X, W, U, V)
    assert np.array_equal(Y[0], g["Y"])
    gr = ol.backward(X, W, Mel, g["dY"].reshape(1, 4), U, V)
    assert np.array_equal(gr["dW"].ravel(), g["dW"])
    assert np.array_equal(gr["dX"][0], g["dX"])
    assert np.array_equal(gr["dU"].ravel(), g["dU"])
    assert np.array_equal(gr["dV"].ravel(), g["dV"])


def _tiny(n_out, n_in, b, ms, T, r, seed):
    rng = np.random.default_rng(seed)
    M, (row_ptr, col_idx, *_r) = om.layout(n_out, n_in, b, ms)
    Mel = om.element_mask(M, b)
    X = rng.standard_normal((T, n_in))
    W = rng.standard_normal((n_out, n_in)) * Mel
    U = rng.standard_normal((n_out, r))
    V = rng.standard_normal((r, n_in))
    dY = rng.standard_normal((T, n_out))
    return M, Mel, row_ptr, col_idx, X, W, U, V, dY


@pytest.mark.parametrize("n_out,n_in,b,ms", [(8, 8, 2, 2), (8, 8, 2, 4), (12, 6, 2, 2), (6, 12, 3, 2)])
def test_finite_differences(n_out, n_in, b, ms):
    """L = <dY, Y> is linear in each of X, W, U, V separately, so central
    differences are exact up to roundoff."""
    M, Mel, _, _, X, W, U, V, dY = _tiny(n_out, n_in, b, ms, T=3, r=2, seed=5)
    gr = ol.backward(X, W, Mel, dY, U, V)
    L = lambda X_, W_, U_, V_: float((dY * ol.forward(X_, W_ * Mel, U_, V_)[0]).sum())
    h = 0.5
    for name, A, idx in [("dX", X, 0), ("dW", W, 1), ("dU", U, 2), ("dV", V, 3)]:
        G = np.zeros_like(A)
        for e in np.ndindex(A.shape):
            args = [X, W, U, V]
            Ap, Am = A.copy(), A.copy()
            Ap[e] += h
            Am[e] -= h
            args[idx] = Ap
            lp = L(*args)
            args[idx] = Am
            G[e] = (lp - L(*args)) / (2 * h)
        assert np.allclose(gr[name], G, atol=1e-10), name
    # the weight gradient is zero off the mask (it is the masked product)
    assert (gr["dW"][~Mel] == 0).all()


def test_blockloop_equals_dense_on_integers():
    rng = np.random.default_rng(2)
    for (n_out, n_in, b, ms) in [(64, 64, 8, 4), (96, 24, 4, 16), (32, 128, 8, 8)]:
        M, (row_ptr, col_idx, *_r) = om.layout(n_out, n_in, b, ms)
        Mel = om.element_mask(M, b)
        X = rng.integers(-2, 3, (16, n_in)).astype(float)
        Wd = rng.integers(-2, 3, (n_out, n_in)).astype(float) * Mel
        Wblk = ol.pack(Wd, row_ptr, col_idx, n_out // b, b)
        assert np.array_equal(ol.unpack(Wblk, row_ptr, col_idx, n_out // b, n_in // b, b), Wd)
        Yb = ol.forward_blockloop(X, Wblk, row_ptr, col_idx, n_out // b, b)
        Yd, _ = ol.forward(X, Wd)
        assert np.array_equal(Yb, Yd)


def test_special_cases_reduce_to_library_routines():
    rng = np.random.default_rng(4)
    # all-kept mask (square side 2 with stride >= 2): plain matmul
    M, _ = om.layout(16, 16, 8, 2)
    assert M.all()
    X, W = rng.standard_normal((5, 16)), rng.standard_normal((16, 16))
    assert np.allclose(ol.forward(X, W * om.element_mask(M, 8))[0], np.matmul(X, W.T))
    # W = 0: low-rank only, X (U V)^T
    U, V = rng.standard_normal((16, 4)), rng.standard_normal((4, 16))
    Y, _ = ol.forward(X, np.zeros((16, 16)), U, V)
    assert np.allclose(Y, np.linalg.multi_dot([X, np.dot(U, V).T]))
    # stride 1: block-diagonal, equal to a batched per-block product
    M, (row_ptr, col_idx, *_r) = om.layout(32, 32, 8, 1)
    Wd = rng.standard_normal((32, 32)) * om.element_mask(M, 8)
    X = rng.standard_normal((7, 32))
    blocks = np.stack([Wd[i * 8:(i + 1) * 8, i * 8:(i + 1) * 8] for i in range(4)])
    ref = np.einsum("tik,ijk->tij", X.reshape(7, 4, 8), blocks).reshape(7, 32)
    assert np.allclose(ol.forward(X, Wd)[0], ref)


def test_gelu_closed_forms():
    assert ol.gelu(np.array([0.0]))[0] == 0.0
    assert abs(ol.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15
    assert abs(ol.gelu(np.array([-1.0]))[0] + 0.15865525393145707) < 1e-15
    x = np.linspace(-4, 4, 33)
    h = 1e-6
    fd = (ol.gelu(x + h) - ol.gelu(x - h)) / (2 * h)
    assert np.allclose(ol.gelu_grad(x), fd, atol=1e-8)


def test_mlp_pair_finite_differences():
    rng = np.random.default_rng(6)
    M1, _ = om.layout(12, 6, 2, 2)
    M2, _ = om.layout(6, 12, 2, 2)
    E1, E2 = om.element_mask(M1, 2), om.element_mask(M2, 2)
    X = rng.standard_normal((3, 6))
    W1 = rng.standard_normal((12, 6)) * E1
    W2 = rng.standard_normal((6, 12)) * E2
    U1, V1 = rng.standard_normal((12, 2)), rng.standard_normal((2, 6))
    U2, V2 = rng.standard_normal((6, 2)), rng.standard_normal((2, 12))
    dY = rng.standard_normal((3, 6))
    g = ol.mlp_pair_backward(X, W1, E1, U1, V1, W2, E2, U2, V2, dY)
    L = lambda X_, W1_: float((dY * ol.mlp_pair_forward(X_, W1_ * E1, U1, V1, W2, U2, V2)["Y"]).sum())
    h = 1e-6
    for name, A, pos in [("dX", X, 0), ("dW", W1, 1)]:
        G = np.zeros_like(A)
        for e in np.ndindex(A.shape):
            Ap, Am = A.copy(), A.copy()
            Ap[e] += h
            Am[e] -= h
            args_p = [X, W1]
            args_m = [X, W1]
            args_p[pos], args_m[pos] = Ap, Am
            G[e] = (L(*args_p) - L(*args_m)) / (2 * h)
        assert np.allclose(g["l1"][name], G, atol=1e-6), name

"""Sparse + low-rank linear layer, dense masked, float64.

Test infrastructure only.

Layer (Section 3.3, model sparsification; the learnable mixing weight of the
same section is in forward_mixed / backward_mixed below):
    Y = X (M o W)^T + (X V^T) U^T
with X: T x K, W: N x K kept on the b x b blocks of the flat block butterfly
mask M, U: N x r, V: r x K.  The low-rank product is applied as U (V^T x)
(appendix on efficient implementation), so T_lr = X V^T is an explicit
intermediate.

Backward (gradient Lemma of the appendix on gradient computation, sparse
training algorithm: the weight gradient is (input . output-gradient^T)
restricted to the mask), with dY the output gradient:
    dX = dY (M o W) + (dY U) V
    dW = (dY^T X) o M
    dU = dY^T (X V^T)
    dV = (dY U)^T X
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf


def unpack(Wblk, row_ptr, col_idx, nb_out: int, nb_in: int, b: int):
    """Packed blocks [nnzb][b][b] (block-CSR order) -> dense N x K with zeros
    outside the mask.  Within a block, Wblk[p][q, c] = W[i*b + q, j*b + c]."""
    W = np.zeros((nb_out * b, nb_in * b))
    for i in range(nb_out):
        for p in range(row_ptr[i], row_ptr[i + 1]):
            j = col_idx[p]
            W[i * b:(i + 1) * b, j * b:(j + 1) * b] = Wblk[p]
    return W


def pack(Wd, row_ptr, col_idx, nb_out: int, b: int):
    """Dense N x K -> packed kept blocks [nnzb][b][b] in block-CSR order."""
    out = np.zeros((int(row_ptr[-1]), b, b))
    for i in range(nb_out):
        for p in range(row_ptr[i], row_ptr[i + 1]):
            j = col_idx[p]
            out[p] = Wd[i * b:(i + 1) * b, j * b:(j + 1) * b]
    return out


def forward(X, Wd, U=None, V=None):
    """Y = X Wd^T + (X V^T) U^T, Wd already masked.  Returns (Y, T_lr)."""
    Y = X @ Wd.T
    T_lr = None
    if U is not None and U.shape[1] > 0:
        T_lr = X @ V.T
        Y = Y + T_lr @ U.T
    return Y, T_lr


def backward(X, Wd, Mel, dY, U=None, V=None):
    """Gradients of L = <dY, Y> for the layer above.

    Returns dict with dX, dW (dense, zero outside the element mask Mel), and
    dU, dV, S = dY U when the low-rank term is present."""
    out = {"dX": dY @ Wd, "dW": (dY.T @ X) * Mel}
    if U is not None and U.shape[1] > 0:
        lr = lowrank_grads(X, dY, U, V)
        out.update(lr)
        out["dX"] = out["dX"] + lr["S"] @ V
    return out


def lowrank_grads(X, dY, U, V):
    """The low-rank part of the backward alone: S = dY U, dU = dY^T (X V^T),
    dV = S^T X (backward() adds S V to dX)."""
    S = dY @ U
    return {"S": S, "dU": dY.T @ (X @ V.T), "dV": S.T @ X}


def forward_blockloop(X, Wblk, row_ptr, col_idx, nb_out: int, b: int):
    """Sparse part of the forward computed block by block over the packed
    kept blocks: Y[:, i] = sum_{j kept in row i} X[:, j] W_blk(i, j)^T."""
    Y = np.zeros((X.shape[0], nb_out * b))
    for i in range(nb_out):
        for p in range(row_ptr[i], row_ptr[i + 1]):
            j = col_idx[p]
            Y[:, i * b:(i + 1) * b] += X[:, j * b:(j + 1) * b] @ Wblk[p].T
    return Y


def gelu(x):
    """Exact (erf) GELU: x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def gelu_grad(x):
    """d/dx [x Phi(x)] = Phi(x) + x phi(x)."""
    Phi = 0.5 * (1.0 + erf(x / np.sqrt(2.0)))
    phi = np.exp(-0.5 * x * x) / np.sqrt(2.0 * np.pi)
    return Phi + x * phi


def mlp_pair_forward(X, W1d, U1, V1, W2d, U2, V2):
    """Two layers with GELU between: H_pre = layer1(X), H = gelu(H_pre),
    Y = layer2(H)."""
    H_pre, T1 = forward(X, W1d, U1, V1)
    H = gelu(H_pre)
    Y, T2 = forward(H, W2d, U2, V2)
    return {"H_pre": H_pre, "H": H, "Y": Y, "T1": T1, "T2": T2}


def mlp_pair_backward(X, W1d, M1, U1, V1, W2d, M2, U2, V2, dY, fwd=None):
    """Backward of mlp_pair_forward for L = <dY, Y>."""
    if fwd is None:
        fwd = mlp_pair_forward(X, W1d, U1, V1, W2d, U2, V2)
    g2 = backward(fwd["H"], W2d, M2, dY, U2, V2)
    dH_pre = g2["dX"] * gelu_grad(fwd["H_pre"])
    g1 = backward(X, W1d, M1, dH_pre, U1, V1)
    return {"l2": g2, "l1": g1, "dH": g2["dX"], "dH_pre": dH_pre}


def mixed_weight(Wd, U, V, gamma):
    """The layer's weight with the learnable mixing weight of Section 3.3
    (model sparsification): gamma B + (1 - gamma) (low-rank product), with B
    the masked sparse matrix Wd (N x K) and the low-rank product U V (U: N x r,
    V: r x K; the paper's U V^T with its V transposed)."""
    return gamma * Wd + (1.0 - gamma) * (U @ V)


def forward_mixed(X, Wd, U, V, gamma):
    """Y = X W^T for the mixed weight, evaluated as the method does it:
    gamma X Wd^T + (1 - gamma) (X V^T) U^T.  Returns (Y, T_lr)."""
    T_lr = X @ V.T
    return gamma * (X @ Wd.T) + (1.0 - gamma) * (T_lr @ U.T), T_lr


def backward_mixed(X, Wd, Mel, dY, U, V, gamma):
    """Gradients of L = <dY, Y> for forward_mixed: with respect to X, the
    sparse blocks (restricted to the mask, gradient Lemma of the appendix on
    gradient computation), U, V and gamma.

        dX     = gamma dY Wd + (1 - gamma) (dY U) V
        dW     = gamma (dY^T X) o M
        dU     = (1 - gamma) dY^T (X V^T)
        dV     = (1 - gamma) (dY U)^T X
        dgamma = <dY, X Wd^T> - <dY, (X V^T) U^T>
               = <(dY^T X) o M, Wd> - <dY U, X V^T>
    (S = dY U and T_lr = X V^T are the unscaled intermediates.)"""
    S = dY @ U
    T_lr = X @ V.T
    G = dY.T @ X
    return {
        "dX": gamma * (dY @ Wd) + (1.0 - gamma) * (S @ V),
        "dW": gamma * G * Mel,
        "dU": (1.0 - gamma) * (dY.T @ T_lr),
        "dV": (1.0 - gamma) * (S.T @ X),
        "dgamma": float(np.sum(dY * (X @ Wd.T)) - np.sum(dY * (T_lr @ U.T))),
        "S": S,
    }

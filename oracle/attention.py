"""Block-sparse softmax attention, dense masked, float64, one head at a time.

Test infrastructure only.

The score matrix keeps only the b x b blocks of the flat block butterfly mask
(the same mask family as the weights; appendix on method details, sparse +
low-rank in attention).  Reading: non-causal, scale 1/sqrt(d), masked scores
are -inf, softmax over each row, no dropout.  Every row keeps its diagonal
block, so no row is empty.

Forward:  S = Q K^T * scale;  S[~M] = -inf;  P = softmax_row(S);  O = P V;
          lse = log sum_j exp(S_ij) (natural log).
Backward (standard softmax calculus, L = <dO, O>):
          delta = rowsum(dO o O);  dV = P^T dO;  dP = dO V^T;
          dS = P o (dP - delta);  dQ = dS K * scale;  dK = dS^T Q * scale.
"""
from __future__ import annotations

import numpy as np


def forward_head(Q, K, V, Mel, scale):
    """One head.  Q, K, V: S x d; Mel: S x S bool.  Returns (O, lse, P)."""
    Sc = (Q @ K.T) * scale
    Sc = np.where(Mel, Sc, -np.inf)
    m = Sc.max(axis=1, keepdims=True)
    E = np.exp(Sc - m)
    l = E.sum(axis=1, keepdims=True)
    P = E / l
    O = P @ V
    lse = (m + np.log(l))[:, 0]
    return O, lse, P


def backward_head(Q, K, V, Mel, scale, dO):
    """One head; returns dQ, dK, dV."""
    O, _, P = forward_head(Q, K, V, Mel, scale)
    delta = (dO * O).sum(axis=1, keepdims=True)
    dV = P.T @ dO
    dP = dO @ V.T
    dS = P * (dP - delta)
    dQ = (dS @ K) * scale
    dK = (dS.T @ Q) * scale
    return dQ, dK, dV


def forward(Q, K, V, Mel, scale, heads=None):
    """Q, K, V: [B][H][S][d].  Returns O, lse for the listed (b, h) pairs
    (all when heads is None) as dicts keyed by (b, h)."""
    Bn, Hn = Q.shape[:2]
    heads = heads if heads is not None else [(x, y) for x in range(Bn) for y in range(Hn)]
    O, L = {}, {}
    for (x, y) in heads:
        o, lse, _ = forward_head(Q[x, y], K[x, y], V[x, y], Mel, scale)
        O[(x, y)], L[(x, y)] = o, lse
    return O, L


def backward(Q, K, V, Mel, scale, dO, heads=None):
    """Gradients for the listed (b, h) pairs, as dicts keyed by (b, h)."""
    Bn, Hn = Q.shape[:2]
    heads = heads if heads is not None else [(x, y) for x in range(Bn) for y in range(Hn)]
    dQ, dK, dV = {}, {}, {}
    for (x, y) in heads:
        dQ[(x, y)], dK[(x, y)], dV[(x, y)] = backward_head(
            Q[x, y], K[x, y], V[x, y], Mel, scale, dO[x, y])
    return dQ, dK, dV

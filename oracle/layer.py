"""SA layer with its projections, in fp64 numpy.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; it shares nothing with the GPU library.

Forward, in the order of Appendix G.3 (one SA layer, "SA FLOPs") and section 3.1:

    Q = P W_Q                       prototype projection   [M, d]
    K = X W_K                       key projection         [L, d]
    S = scale * Q K^T               affinities             [M, L]
    A = softmax over prototypes     (each token's column sums to one)
    sketch = A X                    aggregation of the unprojected history
    lse[t] = log sum_m exp(S[m, t])

per user (the rows of X between two offsets) and per head (heads are
independent SA instances with their own P[h], W_Q[h], W_K[h]; H = 1 is the
paper).  Matrices are materialised per user; matmul is numpy's, in fp64.

Backward, by the chain rule of the forward (the paper prints no gradients):

    dY      = sum_r dsketch[b, r]          (a user's sketch reused by R targets, section 4.2)
    dX     += A^T dY                       (through the aggregation: X is the value)
    dA      = dY X^T
    dS      = A * (dA - colsum(A * dA))    (softmax over prototypes, per token)
    dQ     += scale dS K                   (summed over every user)
    dK      = scale dS^T Q
    dX     += dK W_K^T,   dW_K += X^T dK   (through the key projection)
    dW_Q    = P^T dQ,     dP    = dQ W_Q^T (through the prototype projection)
"""
from __future__ import annotations

import numpy as np


def _check(X, P, Wq, Wk, offsets):
    X = np.asarray(X, np.float64)
    P = np.asarray(P, np.float64)
    Wq = np.asarray(Wq, np.float64)
    Wk = np.asarray(Wk, np.float64)
    offsets = np.asarray(offsets, np.int64)
    T, H, d = X.shape
    if P.shape[0] != H or P.shape[2] != d or Wq.shape != (H, d, d) or Wk.shape != (H, d, d):
        raise ValueError(f"shape mismatch X{X.shape} P{P.shape} Wq{Wq.shape} Wk{Wk.shape}")
    if offsets[0] != 0 or offsets[-1] != T or np.any(np.diff(offsets) < 0):
        raise ValueError("bad offsets")
    return X, P, Wq, Wk, offsets


def _weights(Q, K, scale):
    """A [M, L] (softmax over prototypes, stable form) and lse [L] from Q [M,d], K [L,d]."""
    S = scale * (Q @ K.T)
    mu = S.max(axis=0)
    E = np.exp(S - mu)
    z = E.sum(axis=0)
    return E / z, mu + np.log(z)


def layer_fwd(X, P, Wq, Wk, offsets, scale=None):
    """X [T,H,d], P [H,M,d], Wq/Wk [H,d,d], offsets [B+1] -> (sketch [B,H,M,d], lse [T,H])."""
    X, P, Wq, Wk, offsets = _check(X, P, Wq, Wk, offsets)
    T, H, d = X.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    sketch = np.zeros((B, H, M, d))
    lse = np.full((T, H), np.nan)
    for h in range(H):
        Q = P[h] @ Wq[h]
        for b in range(B):
            t0, t1 = offsets[b], offsets[b + 1]
            if t1 == t0:
                continue
            Xb = X[t0:t1, h]
            A, l = _weights(Q, Xb @ Wk[h], scale)
            sketch[b, h] = A @ Xb
            lse[t0:t1, h] = l
    return sketch, lse


def layer_bwd(X, P, Wq, Wk, offsets, dsketch, scale=None):
    """Gradients of <dsketch summed over R, sketch>: (dX [T,H,d], dP [H,M,d], dWq, dWk [H,d,d])."""
    X, P, Wq, Wk, offsets = _check(X, P, Wq, Wk, offsets)
    T, H, d = X.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    dsketch = np.asarray(dsketch, np.float64)
    if dsketch.shape[0] != B or dsketch.shape[2:] != (H, M, d):
        raise ValueError(f"dsketch shape {dsketch.shape}")
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    dY = dsketch.sum(axis=1)
    dX = np.zeros((T, H, d))
    dP = np.zeros((H, M, d))
    dWq = np.zeros((H, d, d))
    dWk = np.zeros((H, d, d))
    for h in range(H):
        Q = P[h] @ Wq[h]
        dQ = np.zeros((M, d))
        for b in range(B):
            t0, t1 = offsets[b], offsets[b + 1]
            if t1 == t0:
                continue
            Xb = X[t0:t1, h]
            K = Xb @ Wk[h]
            A, _ = _weights(Q, K, scale)
            dXb = A.T @ dY[b, h]
            dA = dY[b, h] @ Xb.T
            dS = A * (dA - (A * dA).sum(axis=0))
            dQ += scale * (dS @ K)
            dK = scale * (dS.T @ Q)
            dXb += dK @ Wk[h].T
            dWk[h] += Xb.T @ dK
            dX[t0:t1, h] = dXb
        dWq[h] = P[h].T @ dQ
        dP[h] = dQ @ Wq[h].T
    return dX, dP, dWq, dWk

"""Stacked SA block (section 3.3, stacked refinement), in fp64 numpy.
TEST INFRASTRUCTURE ONLY: used by tests/ and the smoke check, never by the library.

Starting from the shared prototypes, each of the N_sa layers does, per user and
head (heads are independent instances; H = 1 is the paper):

    S     = scale (Xt W_Q)(X W_K)^T            Xt: the current sketch state [M, d]
    A     = softmax over prototypes (each token's column sums to one)
    Xhat  = A X                                the history itself is aggregated
    Xbar  = LN1(Xt + Xhat)                     residual + layer norm
    Xt    = LN2(Xbar + FFN(Xbar))              SwiGLU FFN with intermediate width 2d

with Xt = P for the first layer (Xt W_Q is then the shared query of Appendix
G.3) and Xt per user afterwards.  FFN(x) = (silu(x W1) * (x W3)) W2 with W1, W3
[d, 2d] and W2 [2d, d] (gate, up and down projections; Appendix G.3 counts
12 M d^2 FLOPs for it).  LN(x) = (x - mean) / sqrt(var + eps) * gamma + beta over
the d features, biased variance.

Readings where the paper is silent: no biases in the FFN; layer norms with an
affine gain and bias and eps = 1e-5; a user with no tokens has a zero sketch
Xhat, so its state is refined from the prototypes alone.

Parameter layout (L = N_sa layers):
    Wq, Wk  [L, H, d, d]      W1, W3 [L, H, d, 2d]      W2 [L, H, 2d, d]
    ln      [L, 4, H, d]      (gamma1, beta1, gamma2, beta2)
"""
from __future__ import annotations

import numpy as np


def layer_norm(x, gamma, beta, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gamma + beta


def swiglu(x, W1, W3, W2):
    g = x @ W1
    return (g / (1.0 + np.exp(-g)) * (x @ W3)) @ W2


def block_fwd(X, P, Wq, Wk, ln, W1, W3, W2, offsets, scale=None, eps=1e-5):
    """Returns (out [B,H,M,d], lse [L,T,H]): the refined sketch and each layer's
    per-token log-sum-exp over the prototypes."""
    X = np.asarray(X, np.float64)
    P = np.asarray(P, np.float64)
    Wq, Wk, ln, W1, W3, W2 = (np.asarray(a, np.float64) for a in (Wq, Wk, ln, W1, W3, W2))
    offsets = np.asarray(offsets, np.int64)
    T, H, d = X.shape
    M = P.shape[1]
    L = Wq.shape[0]
    B = offsets.shape[0] - 1
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((B, H, M, d))
    lse = np.full((L, T, H), np.nan)
    for b in range(B):
        t0, t1 = offsets[b], offsets[b + 1]
        for h in range(H):
            Xb = X[t0:t1, h]
            Xt = P[h]
            for l in range(L):
                Xhat = np.zeros((M, d))
                if t1 > t0:
                    S = scale * ((Xt @ Wq[l, h]) @ (Xb @ Wk[l, h]).T)      # [M, L_b]
                    mu = S.max(axis=0)
                    E = np.exp(S - mu)
                    z = E.sum(axis=0)
                    Xhat = (E / z) @ Xb
                    lse[l, t0:t1, h] = mu + np.log(z)
                Xbar = layer_norm(Xt + Xhat, ln[l, 0, h], ln[l, 1, h], eps)
                Xt = layer_norm(Xbar + swiglu(Xbar, W1[l, h], W3[l, h], W2[l, h]), ln[l, 2, h], ln[l, 3, h], eps)
            out[b, h] = Xt
    return out, lse

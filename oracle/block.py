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


def _ln_bwd(dy, y_in, gamma, eps):
    """Gradients of LN(y_in) * gamma + beta w.r.t. y_in, gamma, beta (rows over the last axis)."""
    mu = y_in.mean(axis=-1, keepdims=True)
    var = ((y_in - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xh = (y_in - mu) * rstd
    g = dy * gamma
    dx = rstd * (g - g.mean(axis=-1, keepdims=True) - xh * (g * xh).mean(axis=-1, keepdims=True))
    return dx, (dy * xh).reshape(-1, dy.shape[-1]).sum(axis=0), dy.reshape(-1, dy.shape[-1]).sum(axis=0)


def block_bwd(X, P, Wq, Wk, ln, W1, W3, W2, offsets, dout, scale=None, eps=1e-5):
    """Gradients of <dout, out> (out of block_fwd): dict with dX [T,H,d], dP [H,M,d],
    dWq, dWk [L,H,d,d], dln [L,4,H,d], dW1, dW3 [L,H,d,2d], dW2 [L,H,2d,d].

    Per user and head the forward is replayed storing each layer's state, sums
    and FFN activations, then the chain rule runs from the last layer down:
    LN2, the FFN (through the gate silu(g) u, silu' = s (1 + g (1 - s))), LN1, then
    the sketch with the state as queries (the softmax-over-prototypes Jacobian of
    the layer oracle) and the two projections.  The state's gradient of the first
    layer is the prototypes' gradient, summed over users; weight gradients are
    summed over users.
    """
    X = np.asarray(X, np.float64)
    P = np.asarray(P, np.float64)
    Wq, Wk, ln, W1, W3, W2 = (np.asarray(a, np.float64) for a in (Wq, Wk, ln, W1, W3, W2))
    dout = np.asarray(dout, np.float64)
    offsets = np.asarray(offsets, np.int64)
    T, H, d = X.shape
    M = P.shape[1]
    L = Wq.shape[0]
    B = offsets.shape[0] - 1
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    g = {"dX": np.zeros_like(X), "dP": np.zeros_like(P), "dWq": np.zeros_like(Wq), "dWk": np.zeros_like(Wk),
         "dln": np.zeros_like(ln), "dW1": np.zeros_like(W1), "dW3": np.zeros_like(W3), "dW2": np.zeros_like(W2)}
    for b in range(B):
        t0, t1 = offsets[b], offsets[b + 1]
        for h in range(H):
            Xb = X[t0:t1, h]
            Xt = P[h]
            saved = []
            for l in range(L):
                Q = Xt @ Wq[l, h]
                K = Xb @ Wk[l, h]
                A = np.zeros((M, 0))
                Xhat = np.zeros((M, d))
                if t1 > t0:
                    S = scale * (Q @ K.T)
                    E = np.exp(S - S.max(axis=0))
                    A = E / E.sum(axis=0)
                    Xhat = A @ Xb
                Y1 = Xt + Xhat
                Xbar = layer_norm(Y1, ln[l, 0, h], ln[l, 1, h], eps)
                G = Xbar @ W1[l, h]
                U = Xbar @ W3[l, h]
                sg = 1.0 / (1.0 + np.exp(-G))
                Z = G * sg * U
                Y2 = Xbar + Z @ W2[l, h]
                saved.append((Xt, Q, K, A, Y1, Xbar, G, U, sg, Z, Y2))
                Xt = layer_norm(Y2, ln[l, 2, h], ln[l, 3, h], eps)
            dXt = dout[b, h]
            for l in range(L - 1, -1, -1):
                Xt, Q, K, A, Y1, Xbar, G, U, sg, Z, Y2 = saved[l]
                dY2, dg2, db2 = _ln_bwd(dXt, Y2, ln[l, 2, h], eps)
                g["dln"][l, 2, h] += dg2
                g["dln"][l, 3, h] += db2
                dZ = dY2 @ W2[l, h].T
                g["dW2"][l, h] += Z.T @ dY2
                dG = dZ * U * sg * (1.0 + G * (1.0 - sg))
                dU = dZ * G * sg
                g["dW1"][l, h] += Xbar.T @ dG
                g["dW3"][l, h] += Xbar.T @ dU
                dXbar = dY2 + dG @ W1[l, h].T + dU @ W3[l, h].T
                dY1, dg1, db1 = _ln_bwd(dXbar, Y1, ln[l, 0, h], eps)
                g["dln"][l, 0, h] += dg1
                g["dln"][l, 1, h] += db1
                dXt = dY1.copy()               # residual
                if t1 > t0:
                    dA = dY1 @ Xb.T            # Xhat = A X: dXhat = dY1
                    g["dX"][t0:t1, h] += A.T @ dY1
                    dS = A * (dA - (A * dA).sum(axis=0))
                    dQ = scale * (dS @ K)
                    dK = scale * (dS.T @ Q)
                    g["dX"][t0:t1, h] += dK @ Wk[l, h].T
                    g["dWk"][l, h] += Xb.T @ dK
                    g["dWq"][l, h] += Xt.T @ dQ
                    dXt += dQ @ Wq[l, h].T
            g["dP"][h] += dXt
    return g

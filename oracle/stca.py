"""Single-query target-to-history cross attention over the adapted sketch, in the
reordered form of Appendix G.2, in fp64 numpy.
TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the bench's CPU
baseline, never by the library.

The sketch branch of section 3.4 runs STCA (recapped in section 2.1, Eq. of Attn)
over the adapted sketch Xs = sketch W_A [k, D] of a user, with one query per
target.  The R targets of a user (the MRLB group of section 4.2) share its
sketch.  Per user b, target r and head i (h heads, d_h = D / h; W^(i) is the
column block i d_h .. (i + 1) d_h of W_Q, W_K, W_V in R^{D x D}):

    u      = (q W_Q^(i)) W_K^(i)T                    in R^D
    alpha  = softmax over the k sketch rows of scale * u Xs^T
    o^(i)  = (alpha Xs) W_V^(i)                       in R^{d_h}

out[b, r] = the heads' o^(i) side by side (in R^D), and lse[b, r, i] = the
log-sum-exp of the scaled logits.  Appendix G.2 shows this equals
softmax(scale (q W_Q^(i))(Xs W_K^(i))^T)(Xs W_V^(i)) without forming the
length-k projections; scale = 1/sqrt(d_h).

Readings where the paper is silent: W_Q, W_K, W_V are square D x D matrices cut
into h column blocks (the paper's W in R^{D x d_h} per head); the output
projection W_O, the query-side FFN and the history-side pre-FFN of a full STCA
layer are separate dense products, not part of this step.

Layout: Xs [B, k, D], q [B, R, D], weights [D, D] (row = input feature).
"""
from __future__ import annotations

import numpy as np


def _heads(W, h):
    D = W.shape[1]
    dh = D // h
    return [W[:, i * dh:(i + 1) * dh] for i in range(h)]


def stca_fwd(Xs, q, Wq, Wk, Wv, h, scale=None):
    """Returns (out [B, R, D], lse [B, R, h])."""
    Xs = np.asarray(Xs, np.float64)
    q = np.asarray(q, np.float64)
    Wq, Wk, Wv = (np.asarray(a, np.float64) for a in (Wq, Wk, Wv))
    B, k, D = Xs.shape
    R = q.shape[1]
    dh = D // h
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    Q, K, V = _heads(Wq, h), _heads(Wk, h), _heads(Wv, h)
    out = np.zeros((B, R, D))
    lse = np.zeros((B, R, h))
    for b in range(B):
        X = Xs[b]
        for r in range(R):
            for i in range(h):
                u = (q[b, r] @ Q[i]) @ K[i].T          # [D]
                s = scale * (X @ u)                    # [k]
                mu = s.max()
                e = np.exp(s - mu)
                z = e.sum()
                alpha = e / z
                out[b, r, i * dh:(i + 1) * dh] = (alpha @ X) @ V[i]
                lse[b, r, i] = mu + np.log(z)
    return out, lse


def stca_bwd(Xs, q, Wq, Wk, Wv, h, dout, scale=None):
    """Gradients of <dout, out> (out of stca_fwd): dict with dXs [B, k, D],
    dq [B, R, D], dWq, dWk, dWv [D, D].

    Per (user, target, head), by the chain rule of the forward: with c = alpha Xs,
    dc = do^(i) W_V^(i)T, dW_V^(i) += c^T do^(i); dalpha = Xs dc, dXs += alpha dc^T;
    ds = alpha (dalpha - <alpha, dalpha>) (softmax Jacobian); du = scale ds Xs,
    dXs += scale ds u^T; with p = q W_Q^(i): dp = du W_K^(i), dW_K^(i) += du^T p,
    dq += dp W_Q^(i)T, dW_Q^(i) += q^T dp.
    """
    Xs = np.asarray(Xs, np.float64)
    q = np.asarray(q, np.float64)
    Wq, Wk, Wv = (np.asarray(a, np.float64) for a in (Wq, Wk, Wv))
    dout = np.asarray(dout, np.float64)
    B, k, D = Xs.shape
    R = q.shape[1]
    dh = D // h
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    Q, K, V = _heads(Wq, h), _heads(Wk, h), _heads(Wv, h)
    g = {"dXs": np.zeros_like(Xs), "dq": np.zeros_like(q), "dWq": np.zeros_like(Wq),
         "dWk": np.zeros_like(Wk), "dWv": np.zeros_like(Wv)}
    for b in range(B):
        X = Xs[b]
        for r in range(R):
            for i in range(h):
                cols = slice(i * dh, (i + 1) * dh)
                p = q[b, r] @ Q[i]                     # [d_h]
                u = p @ K[i].T                         # [D]
                s = scale * (X @ u)
                e = np.exp(s - s.max())
                alpha = e / e.sum()                    # [k]
                c = alpha @ X                          # [D]
                do = dout[b, r, cols]                  # [d_h]
                g["dWv"][:, cols] += np.outer(c, do)
                dc = V[i] @ do                         # [D]
                dalpha = X @ dc                        # [k]
                g["dXs"][b] += np.outer(alpha, dc)
                ds = alpha * (dalpha - alpha @ dalpha)
                du = scale * (ds @ X)                  # [D]
                g["dXs"][b] += scale * np.outer(ds, u)
                dp = du @ K[i]                         # [d_h]
                g["dWk"][:, cols] += np.outer(du, p)
                g["dq"][b, r] += Q[i] @ dp
                g["dWq"][:, cols] += np.outer(q[b, r], dp)
    return g

"""Pins of the SA-layer oracle (Appendix G.3: Q = P W_Q, K = X W_K, S = Q K^T /
sqrt(d), A = softmax over prototypes, sketch = A X; section 3.1) and of its
chain-rule backward.

Each check takes a route other than the oracle's own code:
* identity projections reduce it to the separately pinned C oracle with
  K = V = X (and dX = dK + dV);
* torch float64 autograd of an independently written formulation;
* central finite differences along random directions;
* the gauge invariance W_Q -> W_Q G, W_K -> W_K G^-T (S depends only on W_Q W_K^T);
* the absorbed form S = scale (P W_Q W_K^T) X^T, on dyadic inputs where it is exact;
* mass conservation (sum over prototypes of the sketch = sum of the user's X).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import layer


def case(seed, lengths, H, M, d, wscale=None, dyadic=False):
    rng = np.random.default_rng(seed)
    T = int(sum(lengths))
    if dyadic:
        X = rng.integers(-8, 9, (T, H, d)) / 8.0
        P = rng.integers(-8, 9, (H, M, d)) / 8.0
        Wq = rng.integers(-4, 5, (H, d, d)) / 8.0
        Wk = rng.integers(-4, 5, (H, d, d)) / 8.0
    else:
        ws = wscale if wscale is not None else 1.0 / np.sqrt(d)
        X = rng.standard_normal((T, H, d))
        P = rng.standard_normal((H, M, d))
        Wq = rng.standard_normal((H, d, d)) * ws
        Wk = rng.standard_normal((H, d, d)) * ws
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    return X, P, Wq, Wk, off


def test_identity_projections_reduce_to_c_oracle():
    # exact fp32 inputs so the C oracle (fp32 in, fp64 arithmetic) sees the same values
    X, P, _, _, off = case(1, [7, 0, 12, 3], 2, 6, 8)
    X = X.astype(np.float32).astype(np.float64)
    P = P.astype(np.float32).astype(np.float64)
    H, d = 2, 8
    eye = np.broadcast_to(np.eye(d), (H, d, d)).copy()
    dsk = np.random.default_rng(2).standard_normal((4, 3, H, 6, d)).astype(np.float32)
    sk, lse = layer.layer_fwd(X, P, eye, eye, off)
    rs, rl = oracle.fwd(X, X, P, off)
    np.testing.assert_allclose(sk, rs, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rl, rtol=0, atol=1e-12)
    dX, dP, dWq, dWk = layer.layer_bwd(X, P, eye, eye, off, dsk.astype(np.float64))
    rK, rV, rP = oracle.bwd(X, X, P, off, dsk)
    np.testing.assert_allclose(dX, rK + rV, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dP, rP, rtol=0, atol=1e-11)
    # with W = I: dW_Q = P^T dQ and dW_K = dQ^T P (dQ = dP here)
    for h in range(H):
        np.testing.assert_allclose(dWq[h], P[h].T @ rP[h], rtol=0, atol=1e-11)
        np.testing.assert_allclose(dWk[h], rP[h].T @ P[h], rtol=0, atol=1e-11)


def _torch_layer(X, P, Wq, Wk, off, scale):
    """Independent formulation: one masked [H, T, M] logits tensor, softmax over M."""
    T, H, d = X.shape
    Q = torch.einsum("hmi,hij->hmj", P, Wq)                     # [H, M, d]
    K = torch.einsum("thi,hij->thj", X, Wk)                     # [T, H, d]
    S = scale * torch.einsum("thj,hmj->htm", K, Q)              # [H, T, M]
    A = torch.softmax(S, dim=-1)
    lse = torch.logsumexp(S, dim=-1).T                          # [T, H]
    B = len(off) - 1
    owner = torch.zeros((B, T), dtype=X.dtype)
    for b in range(B):
        owner[b, off[b]:off[b + 1]] = 1.0
    sketch = torch.einsum("bt,htm,thj->bhmj", owner, A, X)
    return sketch, lse


def test_matches_torch_autograd():
    X, P, Wq, Wk, off = case(3, [5, 9, 1, 0, 4], 2, 7, 6)
    dsk = np.random.default_rng(4).standard_normal((5, 2, 2, 7, 6))
    scale = 0.41
    sk, lse = layer.layer_fwd(X, P, Wq, Wk, off, scale=scale)
    dX, dP, dWq, dWk = layer.layer_bwd(X, P, Wq, Wk, off, dsk, scale=scale)
    tX, tP, tWq, tWk = (torch.tensor(a, requires_grad=True) for a in (X, P, Wq, Wk))
    ts, tl = _torch_layer(tX, tP, tWq, tWk, off, scale)
    np.testing.assert_allclose(sk, ts.detach().numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, tl.detach().numpy(), rtol=0, atol=1e-12)
    (ts * torch.tensor(dsk.sum(axis=1))).sum().backward()
    for mine, ref in ((dX, tX), (dP, tP), (dWq, tWq), (dWk, tWk)):
        np.testing.assert_allclose(mine, ref.grad.numpy(), rtol=0, atol=1e-11)


def test_finite_differences():
    X, P, Wq, Wk, off = case(5, [4, 6], 1, 3, 4, wscale=0.7)
    dsk = np.random.default_rng(6).standard_normal((2, 1, 1, 3, 4))
    g = layer.layer_bwd(X, P, Wq, Wk, off, dsk)
    rng = np.random.default_rng(7)
    params = [X, P, Wq, Wk]

    def f(ps):
        sk, _ = layer.layer_fwd(*ps, off)
        return float((sk * dsk.sum(axis=1)).sum())

    eps = 1e-5
    for i in range(4):
        v = rng.standard_normal(params[i].shape)
        plus = [p.copy() for p in params]
        minus = [p.copy() for p in params]
        plus[i] += eps * v
        minus[i] -= eps * v
        fd = (f(plus) - f(minus)) / (2 * eps)
        an = float((g[i] * v).sum())
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (i, fd, an)


def test_gauge_invariance():
    # S = scale P W_Q W_K^T X^T depends on W_Q, W_K only through W_Q W_K^T
    X, P, Wq, Wk, off = case(8, [6, 11], 2, 5, 4)
    G = np.random.default_rng(9).standard_normal((4, 4)) + 3 * np.eye(4)
    Wq2 = Wq @ G
    Wk2 = Wk @ np.linalg.inv(G).T
    a, la = layer.layer_fwd(X, P, Wq, Wk, off)
    b, lb = layer.layer_fwd(X, P, Wq2, Wk2, off)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-11)
    np.testing.assert_allclose(la, lb, rtol=0, atol=1e-11)
    # the projected-key sketch changes with W_K alone
    c, _ = layer.layer_fwd(X, P, Wq, Wk2, off)
    assert np.abs(c - a).max() > 1e-3


def test_absorbed_form_on_dyadic_inputs():
    # on dyadic inputs P' = P W_Q W_K^T is exact in fp32, so the C oracle with
    # K = V = X and prototypes P' evaluates the same logits
    X, P, Wq, Wk, off = case(10, [5, 3, 8], 2, 4, 4, dyadic=True)
    Pp = np.einsum("hmi,hij,hkj->hmk", P, Wq, Wk)
    assert np.array_equal(Pp.astype(np.float32).astype(np.float64), Pp)
    sk, lse = layer.layer_fwd(X, P, Wq, Wk, off, scale=0.5)
    rs, rl = oracle.fwd(X, X, Pp, off, scale=0.5)
    np.testing.assert_allclose(sk, rs, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rl, rtol=0, atol=1e-12)


def test_mass_conservation_and_empty_user():
    X, P, Wq, Wk, off = case(11, [9, 0, 4], 3, 5, 4)
    sk, lse = layer.layer_fwd(X, P, Wq, Wk, off)
    for b in range(3):
        np.testing.assert_allclose(sk[b].sum(axis=1), X[off[b]:off[b + 1]].sum(axis=0), rtol=0, atol=1e-12)
    assert np.all(sk[1] == 0)
    dsk = np.ones((3, 1, 3, 5, 4))
    dX, dP, dWq, dWk = layer.layer_bwd(X, P, Wq, Wk, off, dsk)
    # dY equal across prototypes: the softmax gradient vanishes, dX = dY row, no
    # gradient reaches P or the projections
    np.testing.assert_allclose(dX, 1.0, rtol=0, atol=1e-12)
    for g in (dP, dWq, dWk):
        np.testing.assert_allclose(g, 0.0, rtol=0, atol=1e-12)

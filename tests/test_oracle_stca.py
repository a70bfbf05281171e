"""Pins of the reordered single-query STCA oracle (Appendix G.2; STCA recap in
section 2.1; sketch-side STCA in section 3.4).

Routes other than the oracle's own code:
* torch float64, the standard form softmax(scale (q W_Q)(Xs W_K)^T)(Xs W_V) with
  the length-k projections formed explicitly and all users, targets and heads
  batched (the equality Appendix G.2 states);
* k = 1: every weight is one, so the output is Xs_0 W_V whatever the query and
  lse is the single logit;
* W_Q = 0: uniform weights 1/k, output mean(Xs) W_V, lse = log k;
* heads are independent: changing W_V's columns of one head leaves the others;
* backward: torch float64 autograd of the standard form (all five gradients)
  and central finite differences along random directions.
"""
import numpy as np
import torch

from oracle import stca


def inputs(seed, B, R, k, D):
    rng = np.random.default_rng(seed)
    Xs = rng.standard_normal((B, k, D))
    q = rng.standard_normal((B, R, D))
    W = [rng.standard_normal((D, D)) / np.sqrt(D) for _ in range(3)]
    return Xs, q, W


def torch_standard(Xs, q, Wq, Wk, Wv, h, scale):
    B, k, D = Xs.shape
    R = q.shape[1]
    dh = D // h
    Qp = (q @ Wq).reshape(B, R, h, dh)                      # query projection
    Kp = (Xs @ Wk).reshape(B, k, h, dh)                     # explicit key projection
    Vp = (Xs @ Wv).reshape(B, k, h, dh)                     # explicit value projection
    S = scale * torch.einsum("brhj,bkhj->brhk", Qp, Kp)
    A = torch.softmax(S, dim=-1)
    o = torch.einsum("brhk,bkhj->brhj", A, Vp)
    return o.reshape(B, R, D), torch.logsumexp(S, dim=-1)


def test_matches_standard_form():
    Xs, q, W = inputs(1, 3, 4, 7, 8)
    out, lse = stca.stca_fwd(Xs, q, *W, h=2)
    t = [torch.tensor(a) for a in (Xs, q, *W)]
    ref, rlse = torch_standard(*t, h=2, scale=1 / np.sqrt(4))
    np.testing.assert_allclose(out, ref.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rlse.numpy(), rtol=0, atol=1e-12)


def test_single_sketch_row():
    Xs, q, W = inputs(2, 2, 5, 1, 8)
    out, lse = stca.stca_fwd(Xs, q, *W, h=4)
    for b in range(2):
        for r in range(5):
            np.testing.assert_allclose(out[b, r], Xs[b, 0] @ W[2], rtol=0, atol=1e-12)
    # the single logit: scale (q W_Q^(i)) W_K^(i)T Xs_0, d_h = 2
    dh = 2
    for i in range(4):
        cols = slice(i * dh, (i + 1) * dh)
        u = (q @ W[0][:, cols]) @ W[1][:, cols].T                  # [B, R, D]
        np.testing.assert_allclose(lse[..., i], np.einsum("brd,bd->br", u, Xs[:, 0]) / np.sqrt(dh),
                                   rtol=0, atol=1e-12)


def test_zero_query_weights_average():
    Xs, q, (Wq, Wk, Wv) = inputs(3, 2, 3, 9, 8)
    out, lse = stca.stca_fwd(Xs, q, np.zeros_like(Wq), Wk, Wv, h=2)
    for b in range(2):
        np.testing.assert_allclose(out[b], np.broadcast_to(Xs[b].mean(0) @ Wv, (3, 8)), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.log(9.0), rtol=0, atol=1e-12)


def test_heads_are_independent():
    Xs, q, (Wq, Wk, Wv) = inputs(4, 2, 3, 6, 12)
    out, _ = stca.stca_fwd(Xs, q, Wq, Wk, Wv, h=3)
    Wv2 = Wv.copy()
    Wv2[:, 4:8] = 0.0
    Wk2 = Wk.copy()
    Wk2[:, 4:8] *= 3.0
    out2, _ = stca.stca_fwd(Xs, q, Wq, Wk2, Wv2, h=3)
    np.testing.assert_array_equal(out2[..., :4], out[..., :4])
    np.testing.assert_array_equal(out2[..., 8:], out[..., 8:])
    assert np.all(out2[..., 4:8] == 0)


def test_backward_matches_torch_autograd():
    Xs, q, W = inputs(5, 3, 4, 6, 8)
    dout = np.random.default_rng(6).standard_normal((3, 4, 8))
    g = stca.stca_bwd(Xs, q, *W, h=2, dout=dout)
    t = [torch.tensor(a, requires_grad=True) for a in (Xs, q, *W)]
    out, _ = torch_standard(*t, h=2, scale=1 / np.sqrt(4))
    (out * torch.tensor(dout)).sum().backward()
    for name, tt in zip(("dXs", "dq", "dWq", "dWk", "dWv"), t):
        np.testing.assert_allclose(g[name], tt.grad.numpy(), rtol=0, atol=1e-11, err_msg=name)


def test_backward_finite_differences():
    Xs, q, W = inputs(7, 2, 3, 5, 8)
    dout = np.random.default_rng(8).standard_normal((2, 3, 8))
    g = stca.stca_bwd(Xs, q, *W, h=4, dout=dout)
    rng = np.random.default_rng(9)
    args = [Xs, q, *W]
    eps = 1e-6
    for idx, name in enumerate(("dXs", "dq", "dWq", "dWk", "dWv")):
        v = rng.standard_normal(args[idx].shape)
        up = list(args)
        dn = list(args)
        up[idx] = args[idx] + eps * v
        dn[idx] = args[idx] - eps * v
        fu = (stca.stca_fwd(*up, h=4)[0] * dout).sum()
        fd_ = (stca.stca_fwd(*dn, h=4)[0] * dout).sum()
        fd = (fu - fd_) / (2 * eps)
        assert abs(fd - (g[name] * v).sum()) < 1e-6 * max(1.0, abs(fd)), name

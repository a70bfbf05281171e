"""Pins of the stacked SA block oracle (section 3.3: per-layer allocation and
aggregation with the current sketch state as queries, residual + LN, SwiGLU FFN +
residual + LN; Appendix G.3 for the projections and the FFN width).

Routes other than the oracle's own code:
* torch float64: an independently written batched formulation (masked logits
  over all tokens at once, torch's layer_norm and silu);
* one layer with a zero FFN and unit norms reduces to LN(LN(P + sketch)) with the
  sketch of the separately pinned layer oracle;
* unit-gain, zero-bias norms give rows of zero mean and variance var/(var+eps);
* token order within a user does not matter; an empty user depends on P only;
* backward: torch float64 autograd of the independent formulation (all eight
  gradients) and central finite differences along random directions.
"""
import numpy as np
import torch

from oracle import block, layer


def params(seed, L, H, d, unit_ln=False, zero_ffn=False):
    rng = np.random.default_rng(seed)
    s = 1.0 / np.sqrt(d)
    Wq = rng.standard_normal((L, H, d, d)) * s
    Wk = rng.standard_normal((L, H, d, d)) * s
    W1 = rng.standard_normal((L, H, d, 2 * d)) * s
    W3 = rng.standard_normal((L, H, d, 2 * d)) * s
    W2 = rng.standard_normal((L, H, 2 * d, d)) / np.sqrt(2 * d)
    if zero_ffn:
        W2 = np.zeros_like(W2)
    ln = np.empty((L, 4, H, d))
    ln[:, 0] = 1.0 + 0.1 * rng.standard_normal((L, H, d))
    ln[:, 1] = 0.1 * rng.standard_normal((L, H, d))
    ln[:, 2] = 1.0 + 0.1 * rng.standard_normal((L, H, d))
    ln[:, 3] = 0.1 * rng.standard_normal((L, H, d))
    if unit_ln:
        ln[:, 0] = ln[:, 2] = 1.0
        ln[:, 1] = ln[:, 3] = 0.0
    return Wq, Wk, ln, W1, W3, W2


def inputs(seed, lengths, H, M, d):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((int(sum(lengths)), H, d))
    P = rng.standard_normal((H, M, d)) / np.sqrt(d)
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    return X, P, off


def torch_block(X, P, Wq, Wk, ln, W1, W3, W2, off, scale, eps):
    X, P, Wq, Wk, ln, W1, W3, W2 = (torch.tensor(a) for a in (X, P, Wq, Wk, ln, W1, W3, W2))
    T, H, d = X.shape
    B = len(off) - 1
    M = P.shape[1]
    L = Wq.shape[0]
    owner = torch.zeros((B, T), dtype=torch.float64)
    for b in range(B):
        owner[b, off[b]:off[b + 1]] = 1.0
    state = P.unsqueeze(0).expand(B, H, M, d)                         # [B, H, M, d]
    for l in range(L):
        q = torch.einsum("bhmi,hij->bhmj", state, Wq[l])
        k = torch.einsum("thi,hij->thj", X, Wk[l])
        S = scale * torch.einsum("bhmj,thj->bhmt", q, k)
        S = S.masked_fill(owner[:, None, None, :] == 0, float("-inf"))
        A = torch.softmax(S, dim=2).nan_to_num(0.0)                  # over prototypes
        xhat = torch.einsum("bhmt,thj->bhmj", A, X)
        xbar = torch.stack([torch.nn.functional.layer_norm(state[:, h] + xhat[:, h], (d,), ln[l, 0, h], ln[l, 1, h], eps)
                            for h in range(H)], dim=1)
        g = torch.einsum("bhmi,hij->bhmj", xbar, W1[l])
        u = torch.einsum("bhmi,hij->bhmj", xbar, W3[l])
        f = torch.einsum("bhmi,hij->bhmj", torch.nn.functional.silu(g) * u, W2[l])
        state = torch.stack([torch.nn.functional.layer_norm(xbar[:, h] + f[:, h], (d,), ln[l, 2, h], ln[l, 3, h], eps)
                             for h in range(H)], dim=1)
    return state.numpy()


def test_matches_torch_formulation():
    X, P, off = inputs(1, [6, 0, 11, 3], 2, 5, 4)
    prm = params(2, 2, 2, 4)
    out, lse = block.block_fwd(X, P, *prm, off, scale=0.4)
    ref = torch_block(X, P, *prm, off, 0.4, 1e-5)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-11)
    assert np.all(np.isfinite(lse[:, :20])) and lse.shape == (2, 20, 2)


def test_one_layer_reduces_to_layer_oracle():
    X, P, off = inputs(3, [7, 4, 9], 2, 6, 4)
    Wq, Wk, ln, W1, W3, W2 = params(4, 1, 2, 4, unit_ln=True, zero_ffn=True)
    out, lse = block.block_fwd(X, P, Wq, Wk, ln, W1, W3, W2, off)
    sk, l_lse = layer.layer_fwd(X, P, Wq[0], Wk[0], off)
    np.testing.assert_allclose(lse[0], l_lse, rtol=0, atol=1e-12)
    eps = 1e-5
    for b in range(3):
        for h in range(2):
            z = P[h] + sk[b, h]
            z = (z - z.mean(-1, keepdims=True)) / np.sqrt(z.var(-1, keepdims=True) + eps)
            z = (z - z.mean(-1, keepdims=True)) / np.sqrt(z.var(-1, keepdims=True) + eps)
            np.testing.assert_allclose(out[b, h], z, rtol=0, atol=1e-12)


def test_unit_norm_rows_are_standardised():
    X, P, off = inputs(5, [12, 5], 1, 8, 6)
    prm = params(6, 2, 1, 6, unit_ln=True)
    out, _ = block.block_fwd(X, P, *prm, off)
    np.testing.assert_allclose(out.mean(-1), 0.0, atol=1e-12)
    var = out.var(-1)
    assert np.all(var < 1.0) and np.all(var > 1.0 - 1e-3)


def test_token_permutation_and_empty_users():
    X, P, off = inputs(7, [10, 0, 0, 8], 2, 4, 4)
    prm = params(8, 2, 2, 4)
    out, _ = block.block_fwd(X, P, *prm, off)
    perm = np.concatenate([np.random.default_rng(9).permutation(10), 10 + np.arange(8)[::-1]])
    out2, _ = block.block_fwd(X[perm], P, *prm, off)
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-12)
    # the two empty users see the prototypes only, and identically
    np.testing.assert_array_equal(out[1], out[2])
    alone, _ = block.block_fwd(X[:0], P, *prm, np.array([0, 0], np.int64))
    np.testing.assert_allclose(out[1], alone[0], rtol=0, atol=1e-13)


def test_backward_matches_torch_autograd():
    X, P, off = inputs(21, [6, 0, 9, 3], 2, 5, 4)
    prm = params(22, 2, 2, 4)
    dout = np.random.default_rng(23).standard_normal((4, 2, 5, 4))
    g = block.block_bwd(X, P, *prm, off, dout, scale=0.45)
    tX, tP = torch.tensor(X, requires_grad=True), torch.tensor(P, requires_grad=True)
    tw = [torch.tensor(a, requires_grad=True) for a in prm]
    out = _torch_block_t(tX, tP, *tw, off, 0.45, 1e-5)
    (out * torch.tensor(dout)).sum().backward()
    ref = {"dX": tX.grad, "dP": tP.grad, "dWq": tw[0].grad, "dWk": tw[1].grad, "dln": tw[2].grad,
           "dW1": tw[3].grad, "dW3": tw[4].grad, "dW2": tw[5].grad}
    for k, v in ref.items():
        np.testing.assert_allclose(g[k], v.numpy(), rtol=0, atol=1e-10, err_msg=k)


def _torch_block_t(X, P, Wq, Wk, ln, W1, W3, W2, off, scale, eps):
    T, H, d = X.shape
    B = len(off) - 1
    M = P.shape[1]
    L = Wq.shape[0]
    owner = torch.zeros((B, T), dtype=torch.float64)
    for b in range(B):
        owner[b, off[b]:off[b + 1]] = 1.0
    state = P.unsqueeze(0).expand(B, H, M, d)
    for l in range(L):
        q = torch.einsum("bhmi,hij->bhmj", state, Wq[l])
        k = torch.einsum("thi,hij->thj", X, Wk[l])
        S = scale * torch.einsum("bhmj,thj->bhmt", q, k)
        S = S.masked_fill(owner[:, None, None, :] == 0, float("-inf"))
        A = torch.softmax(S, dim=2).nan_to_num(0.0)
        xhat = torch.einsum("bhmt,thj->bhmj", A, X)
        xbar = torch.stack([torch.nn.functional.layer_norm(state[:, h] + xhat[:, h], (d,), ln[l, 0, h], ln[l, 1, h], eps)
                            for h in range(H)], dim=1)
        gg = torch.einsum("bhmi,hij->bhmj", xbar, W1[l])
        u = torch.einsum("bhmi,hij->bhmj", xbar, W3[l])
        f = torch.einsum("bhmi,hij->bhmj", torch.nn.functional.silu(gg) * u, W2[l])
        state = torch.stack([torch.nn.functional.layer_norm(xbar[:, h] + f[:, h], (d,), ln[l, 2, h], ln[l, 3, h], eps)
                             for h in range(H)], dim=1)
    return state


def test_backward_finite_differences():
    X, P, off = inputs(24, [5, 7], 1, 3, 4)
    prm = list(params(25, 2, 1, 4))
    dout = np.random.default_rng(26).standard_normal((2, 1, 3, 4))
    g = block.block_bwd(X, P, *prm, off, dout)
    rng = np.random.default_rng(27)

    def f(Xa, Pa, pr):
        out, _ = block.block_fwd(Xa, Pa, *pr, off)
        return float((out * dout).sum())

    eps = 1e-6
    names = ["dWq", "dWk", "dln", "dW1", "dW3", "dW2"]
    for name, arr in (("dX", X), ("dP", P)):
        v = rng.standard_normal(arr.shape)
        a, b = (X + eps * v, P) if name == "dX" else (X, P + eps * v)
        c, e = (X - eps * v, P) if name == "dX" else (X, P - eps * v)
        fd = (f(a, b, prm) - f(c, e, prm)) / (2 * eps)
        assert abs(fd - (g[name] * v).sum()) < 1e-6 * max(1.0, abs(fd)), name
    for i, name in enumerate(names):
        v = rng.standard_normal(prm[i].shape)
        up = [p.copy() for p in prm]
        dn = [p.copy() for p in prm]
        up[i] += eps * v
        dn[i] -= eps * v
        fd = (f(X, P, up) - f(X, P, dn)) / (2 * eps)
        assert abs(fd - (g[name] * v).sum()) < 1e-6 * max(1.0, abs(fd)), name

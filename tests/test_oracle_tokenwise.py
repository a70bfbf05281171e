"""Pins of the token-wise normalised oracle (the paper's alternative to SA's
prototype-wise normalisation: weights normalised over each user's tokens for
every prototype; appendix on prototype-wise normalisation, Table 1 baseline).

Each pin checks the oracle against something other than its own code: torch's
scaled-dot-product attention (prototypes as queries), a materialised
long-double formulation, closed forms, and invariances that hold for this
normalisation and not for the other.
"""
import numpy as np
import pytest
import torch

import oracle


def _inputs(rng, lengths, H, M, d):
    T = int(sum(lengths))
    K = rng.standard_normal((T, H, d)).astype(np.float32)
    V = rng.standard_normal((T, H, d)).astype(np.float32)
    P = (rng.standard_normal((H, M, d)) / np.sqrt(d)).astype(np.float32)
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    return K, V, P, off


def test_matches_torch_attention_with_prototype_queries():
    # softmax over a user's tokens for each prototype is attention with the M
    # prototypes as queries and the user's tokens as keys / values
    rng = np.random.default_rng(11)
    lengths = [7, 1, 20, 3]
    H, M, d = 2, 5, 8
    K, V, P, off = _inputs(rng, lengths, H, M, d)
    scale = 0.37
    sk, lse = oracle.fwd_tokenwise(K, V, P, off, scale=scale)
    for b in range(len(lengths)):
        t0, t1 = off[b], off[b + 1]
        for h in range(H):
            q = torch.from_numpy(P[h].astype(np.float64))[None, None]
            k = torch.from_numpy(K[t0:t1, h].astype(np.float64))[None, None]
            v = torch.from_numpy(V[t0:t1, h].astype(np.float64))[None, None]
            ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale)[0, 0].numpy()
            np.testing.assert_allclose(sk[b, h], ref, rtol=0, atol=1e-12)
            ref_lse = torch.logsumexp(scale * (q[0, 0] @ k[0, 0].T), dim=-1).numpy()
            np.testing.assert_allclose(lse[b, h], ref_lse, rtol=0, atol=1e-12)


def test_brute_force_longdouble():
    rng = np.random.default_rng(12)
    lengths = [3, 5, 2]
    H, M, d = 1, 4, 3
    K, V, P, off = _inputs(rng, lengths, H, M, d)
    scale = 0.5
    sk, lse = oracle.fwd_tokenwise(K, V, P, off, scale=scale)
    for b in range(len(lengths)):
        Kb = K[off[b]:off[b + 1], 0].astype(np.longdouble)
        Vb = V[off[b]:off[b + 1], 0].astype(np.longdouble)
        S = np.longdouble(scale) * (P[0].astype(np.longdouble) @ Kb.T)     # [M, L]
        W = np.exp(S) / np.exp(S).sum(axis=1, keepdims=True)               # over tokens
        np.testing.assert_allclose(sk[b, 0], (W @ Vb).astype(np.float64), rtol=0, atol=1e-13)
        np.testing.assert_allclose(lse[b, 0], np.log(np.exp(S).sum(axis=1)).astype(np.float64),
                                   rtol=0, atol=1e-13)


def test_weights_sum_to_one_over_tokens():
    # V = 1 gives sketch rows equal to the sum of the weights over the tokens
    rng = np.random.default_rng(13)
    lengths = [9, 4, 1]
    H, M, d = 3, 6, 4
    K, V, P, off = _inputs(rng, lengths, H, M, d)
    sk, _ = oracle.fwd_tokenwise(K, np.ones_like(V), P, off)
    np.testing.assert_allclose(sk, 1.0, rtol=0, atol=1e-13)


def test_single_token_and_uniform_logits():
    rng = np.random.default_rng(14)
    H, M, d = 2, 3, 4
    # one token: every prototype's sketch row is that token's V, lse_m = s_m
    K, V, P, off = _inputs(rng, [1], H, M, d)
    sk, lse = oracle.fwd_tokenwise(K, V, P, off, scale=0.3)
    for h in range(H):
        np.testing.assert_allclose(sk[0, h], np.broadcast_to(V[0, h], (M, d)), rtol=0, atol=1e-15)
        np.testing.assert_allclose(lse[0, h], 0.3 * (P[h].astype(np.float64) @ K[0, h].astype(np.float64)),
                                   rtol=0, atol=1e-14)
    # P = 0: every weight is 1/L, the sketch is the mean of V, lse = log L
    K, V, P, off = _inputs(rng, [5, 8], H, M, d)
    sk, lse = oracle.fwd_tokenwise(K, V, np.zeros_like(P), off)
    for b, L in enumerate([5, 8]):
        mean = V[off[b]:off[b + 1]].astype(np.float64).mean(axis=0)     # [H, d]
        np.testing.assert_allclose(sk[b], np.broadcast_to(mean[:, None, :], (H, M, d)), rtol=0, atol=1e-14)
        np.testing.assert_allclose(lse[b], np.log(L), rtol=0, atol=1e-14)


def test_empty_user():
    rng = np.random.default_rng(15)
    K, V, P, off = _inputs(rng, [3, 0, 2], 1, 2, 4)
    sk, lse = oracle.fwd_tokenwise(K, V, P, off)
    assert np.all(sk[1] == 0.0) and np.all(np.isneginf(lse[1]))


def test_common_key_shift_invariance():
    # adding one vector w to every K row shifts each prototype's logits by the
    # token-independent scale*w.P_m: the token-wise weights do not change (the
    # prototype-wise ones do), and lse_m moves by exactly that amount
    rng = np.random.default_rng(16)
    lengths = [6, 11]
    H, M, d = 1, 4, 8
    K, V, P, off = _inputs(rng, lengths, H, M, d)
    w = np.array([2.0, -1.0, 0.5, 0.0, 1.0, 0.0, -2.0, 0.25], np.float32)   # dyadic, exact sums
    Kd = np.round(K * 64) / 64
    sk0, lse0 = oracle.fwd_tokenwise(Kd, V, P, off, scale=0.25)
    sk1, lse1 = oracle.fwd_tokenwise(Kd + w, V, P, off, scale=0.25)
    np.testing.assert_allclose(sk1, sk0, rtol=0, atol=1e-12)
    shift = 0.25 * (P[0].astype(np.float64) @ w.astype(np.float64))
    np.testing.assert_allclose(lse1[:, 0] - lse0[:, 0], np.broadcast_to(shift, (2, M)), rtol=0, atol=1e-12)
    # the prototype-wise sketch is not invariant to this shift
    pw0, _ = oracle.fwd(Kd, V, P, off, scale=0.25)
    pw1, _ = oracle.fwd(Kd + w, V, P, off, scale=0.25)
    assert np.max(np.abs(pw1 - pw0)) > 1e-3


def test_split_merge_by_lse():
    # a user cut into chunks: each chunk's normalised sketch weighted by
    # exp(lse_chunk - lse) and summed gives the whole user's sketch, and the
    # chunk lse's combine by log-sum-exp (the merge a split-L implementation uses)
    rng = np.random.default_rng(17)
    H, M, d = 2, 5, 6
    K, V, P, off = _inputs(rng, [23], H, M, d)
    whole, lse = oracle.fwd_tokenwise(K, V, P, off)
    cuts = np.array([0, 4, 5, 17, 23], np.int64)
    parts, plse = oracle.fwd_tokenwise(K, V, P, cuts)
    L = np.logaddexp.reduce(plse, axis=0)                          # [H, M]
    merged = (np.exp(plse - L)[..., None] * parts).sum(axis=0)
    np.testing.assert_allclose(L, lse[0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(merged, whole[0], rtol=0, atol=1e-12)


def test_permutation_within_user():
    rng = np.random.default_rng(18)
    H, M, d = 1, 3, 4
    K, V, P, off = _inputs(rng, [12], H, M, d)
    perm = rng.permutation(12)
    a, la = oracle.fwd_tokenwise(K, V, P, off)
    b, lb = oracle.fwd_tokenwise(K[perm], V[perm], P, off)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)
    np.testing.assert_allclose(la, lb, rtol=0, atol=1e-13)

"""Pins of the fp64 CPU oracle against facts the paper and the mathematics fix.

None of these re-types the oracle's loops: each check uses an independent
route (a materialised matrix formulation, a library softmax / autograd, a
closed form, an invariant, or finite differences) chosen so that a plausible
mistake in the oracle (normalising over tokens instead of prototypes, a
dropped scale, a transposed operand, a wrong user range, a sign error in the
softmax Jacobian) fails at least one of them.

Paper passages: section 3.1 (S = Q K^T / sqrt(d), A = softmax over prototypes
with sum_j A_{j,i} = 1, sketch = A X), Appendix B, Appendix C (per-token
conservation), section 4.2 (MRLB: a user's sketch reused by R targets).
"""
import math

import numpy as np
import pytest
import scipy.special

import oracle
from paper_2609_08443_amd import workloads as wl


def rand_case(seed, lengths, H, M, d, scale_p=None, dyadic=False):
    rng = np.random.default_rng(seed)
    T = int(sum(lengths))
    if dyadic:
        # values k * 2^-6, exactly representable with room for 2^-12 steps
        K = (rng.integers(-64, 65, (T, H, d)) / 64.0).astype(np.float32)
        V = (rng.integers(-64, 65, (T, H, d)) / 64.0).astype(np.float32)
        P = (rng.integers(-64, 65, (H, M, d)) / 64.0).astype(np.float32)
    else:
        K = rng.standard_normal((T, H, d)).astype(np.float32)
        V = rng.standard_normal((T, H, d)).astype(np.float32)
        sp = scale_p if scale_p is not None else 1.0
        P = (rng.standard_normal((H, M, d)) * sp).astype(np.float32)
    off = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=off[1:])
    return K, V, P, off


def brute_force_fwd(K, V, P, off, scale):
    """Materialised formulation in long double: S (k x n), A = softmax over axis k, X~ = A X."""
    B = len(off) - 1
    T, H, d = K.shape
    M = P.shape[1]
    ld = np.longdouble
    sketch = np.zeros((B, H, M, d), ld)
    lse = np.zeros((T, H), ld)
    for b in range(B):
        s, e = off[b], off[b + 1]
        for h in range(H):
            X = V[s:e, h, :].astype(ld)                       # n x d
            Kh = K[s:e, h, :].astype(ld)                      # n x d
            Q = P[h].astype(ld)                               # k x d
            S = (Q @ Kh.T) * ld(scale)                        # k x n  (paper orientation)
            if e > s:
                mx = S.max(axis=0, keepdims=True)
                E = np.exp(S - mx)
                A = E / E.sum(axis=0, keepdims=True)          # normalise over prototypes
                sketch[b, h] = A @ X                          # k x d
                lse[s:e, h] = (mx + np.log(E.sum(axis=0, keepdims=True)))[0]
    return sketch, lse


# ---------------------------------------------------------------- P1
def test_conservation_per_token():
    """Appendix C / section 3.1: sum over prototypes of A_{j,i} is 1 for every token."""
    K, V, P, off = rand_case(1, [37], 3, 40, 16)
    A, _ = oracle.weights(K, P)
    assert np.all(A >= 0)
    np.testing.assert_allclose(A.sum(axis=-1), 1.0, rtol=0, atol=1e-12)
    # and it is NOT a softmax over tokens: the column sums over tokens are not 1
    assert np.abs(A.sum(axis=0) - 1.0).max() > 0.1


# ---------------------------------------------------------------- P2
@pytest.mark.parametrize("lengths", [[5, 0, 17, 1], [64], [3, 3, 3]])
def test_mass_conservation_of_sketch(lengths):
    """sum_m sketch[b,h,m,:] = sum_{t in b} V[t,h,:] (follows from sum_m A = 1 and X~ = A X)."""
    K, V, P, off = rand_case(2, lengths, 2, 24, 8, scale_p=0.5)
    sk, _ = oracle.fwd(K, V, P, off)
    for b in range(len(lengths)):
        ref = V[off[b]:off[b + 1]].astype(np.float64).sum(axis=0)     # [H, d]
        np.testing.assert_allclose(sk[b].sum(axis=1), ref, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- P3
def test_token_permutation_invariance():
    """The sketch is a sum over a user's tokens: reordering them changes nothing;
    lse moves with its token."""
    K, V, P, off = rand_case(3, [9, 14], 2, 16, 8)
    rng = np.random.default_rng(7)
    perm = np.concatenate([rng.permutation(9), 9 + rng.permutation(14)])
    sk, lse = oracle.fwd(K, V, P, off)
    sk2, lse2 = oracle.fwd(K[perm], V[perm], P, off)
    np.testing.assert_allclose(sk2, sk, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(lse2, lse[perm])


# ---------------------------------------------------------------- P4
def test_single_token_closed_form():
    """L = 1: sketch_m = softmax_m(s) V_t with s = scale * P K_t (library softmax)."""
    K, V, P, off = rand_case(4, [1, 1], 2, 12, 8)
    sc = 1.0 / math.sqrt(8)
    sk, lse = oracle.fwd(K, V, P, off)
    for b in range(2):
        for h in range(2):
            s = sc * (P[h].astype(np.float64) @ K[b, h].astype(np.float64))
            a = scipy.special.softmax(s)
            np.testing.assert_allclose(sk[b, h], np.outer(a, V[b, h]), rtol=1e-12, atol=1e-14)
            np.testing.assert_allclose(lse[b, h], scipy.special.logsumexp(s), rtol=1e-13)


def test_single_prototype_closed_form():
    """M = 1: every weight is 1, the sketch is the plain sum of V, lse = the logit."""
    K, V, P, off = rand_case(5, [7, 3], 2, 1, 8)
    sk, lse = oracle.fwd(K, V, P, off)
    for b in range(2):
        np.testing.assert_allclose(sk[b, :, 0, :], V[off[b]:off[b + 1]].astype(np.float64).sum(0), rtol=1e-12,
                                   atol=1e-12)
    s = np.einsum("thd,hd->th", K.astype(np.float64), P[:, 0, :].astype(np.float64)) / math.sqrt(8)
    np.testing.assert_allclose(lse, s, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("zero", ["P", "K", "equal_rows"])
def test_uniform_logits_closed_form(zero):
    """Equal logits for all prototypes: every weight is 1/M; lse = log M + common logit."""
    K, V, P, off = rand_case(6, [6, 11], 2, 10, 8)
    if zero == "P":
        P[:] = 0
    elif zero == "K":
        K[:] = 0
    else:
        P[:] = P[:, :1, :]
    sk, lse = oracle.fwd(K, V, P, off)
    for b in range(2):
        ref = V[off[b]:off[b + 1]].astype(np.float64).sum(0) / 10.0     # [H, d]
        for m in range(10):
            np.testing.assert_allclose(sk[b, :, m, :], ref, rtol=1e-12, atol=1e-13)
    common = np.einsum("thd,hd->th", K.astype(np.float64), P[:, 0, :].astype(np.float64)) / math.sqrt(8)
    np.testing.assert_allclose(lse, math.log(10.0) + common, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- P5, P6
def test_prototype_shift_invariance():
    """Adding one vector u to every prototype shifts all logits of a token equally."""
    K, V, P, off = rand_case(8, [13, 4], 2, 16, 8)
    P = (np.round(P * 64) / 64).astype(np.float32)   # dyadic, so P + u is exact in fp32
    u = np.asarray([0.5, -0.25, 1.0, 0.0, 0.125, -1.0, 0.75, 0.25], np.float32)
    sk, _ = oracle.fwd(K, V, P, off)
    sk2, _ = oracle.fwd(K, V, (P + u).astype(np.float32), off)
    np.testing.assert_allclose(sk2, sk, rtol=1e-10, atol=1e-12)


def test_linearity_in_values():
    K, V1, P, off = rand_case(9, [8, 5], 2, 16, 8)
    # dyadic values so that a V1 + b V2 is exact in fp32
    V1 = (np.round(V1 * 64) / 64).astype(np.float32)
    V2 = (np.random.default_rng(10).integers(-64, 65, V1.shape) / 64).astype(np.float32)
    a, b = 0.5, -2.0
    s1, _ = oracle.fwd(K, V1, P, off)
    s2, _ = oracle.fwd(K, V2, P, off)
    s3, _ = oracle.fwd(K, (a * V1 + b * V2).astype(np.float32), P, off)
    np.testing.assert_allclose(s3, a * s1 + b * s2, rtol=1e-10, atol=1e-12)


def test_scale_is_applied_to_logits():
    """Doubling K at scale c equals keeping K at scale 2c (the 1/sqrt(d) of section 3.1)."""
    K, V, P, off = rand_case(11, [9], 1, 8, 4)
    s1, l1 = oracle.fwd(K, V, P, off, scale=1.0)
    s2, l2 = oracle.fwd((2 * K).astype(np.float32), V, P, off, scale=0.5)
    np.testing.assert_allclose(s1, s2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=1e-13)
    # default scale is 1/sqrt(d) with d the per-head width
    s3, _ = oracle.fwd(K, V, P, off)
    s4, _ = oracle.fwd(K, V, P, off, scale=0.5)
    np.testing.assert_array_equal(s3, s4)


# ---------------------------------------------------------------- P7
@pytest.mark.parametrize("seed,lengths,H,M,d", [
    (12, [3, 0, 5], 2, 4, 4), (13, [1, 2], 1, 3, 2), (14, [5, 5, 1], 3, 4, 3)])
def test_brute_force_tiny(seed, lengths, H, M, d):
    K, V, P, off = rand_case(seed, lengths, H, M, d)
    sc = 1.0 / math.sqrt(d)
    sk, lse = oracle.fwd(K, V, P, off)
    bsk, blse = brute_force_fwd(K, V, P, off, sc)
    np.testing.assert_allclose(sk, bsk.astype(np.float64), rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse, blse.astype(np.float64), rtol=1e-13, atol=1e-14)


def test_empty_user_gives_zero_sketch():
    K, V, P, off = rand_case(15, [0, 4, 0], 2, 8, 4)
    sk, _ = oracle.fwd(K, V, P, off)
    assert np.all(sk[0] == 0) and np.all(sk[2] == 0)
    assert np.any(sk[1] != 0)


def test_large_logits_are_stable():
    """Logits of several hundred do not overflow: the stable form is exact."""
    K, V, P, off = rand_case(16, [6], 1, 5, 4)
    K *= 200.0
    sk, lse = oracle.fwd(K, V, P, off)
    assert np.all(np.isfinite(sk)) and np.all(np.isfinite(lse))
    bsk, blse = brute_force_fwd(K, V, P, off, 0.5)
    np.testing.assert_allclose(sk, bsk.astype(np.float64), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, blse.astype(np.float64), rtol=1e-13)


# ---------------------------------------------------------------- P8 (finite differences)
def _f(K, V, P, off, dY, sc):
    sk, _ = oracle.fwd(K, V, P, off, scale=sc)
    return float((sk * dY).sum())


def test_backward_finite_differences():
    """Central differences of f = <dY, sketch> on dyadic inputs (exact +/- h in fp32)."""
    lengths, H, M, d = [3, 2], 2, 4, 3
    K, V, P, off = rand_case(17, lengths, H, M, d, dyadic=True)
    B = len(lengths)
    rng = np.random.default_rng(18)
    dS = (rng.integers(-32, 33, (B, 1, H, M, d)) / 32.0).astype(np.float32)
    dY = dS.astype(np.float64).sum(axis=1)
    sc = 0.75
    dK, dV, dP = oracle.bwd(K, V, P, off, dS, scale=sc)
    h = 2.0 ** -12

    def fd(arr, idx):
        a0 = arr[idx]
        arr[idx] = a0 + h
        fp = _f(K, V, P, off, dY, sc)
        arr[idx] = a0 - h
        fm = _f(K, V, P, off, dY, sc)
        arr[idx] = a0
        return (fp - fm) / (2 * h)

    for name, arr, grad in (("K", K, dK), ("V", V, dV), ("P", P, dP)):
        num = np.zeros_like(grad)
        for idx in np.ndindex(arr.shape):
            num[idx] = fd(arr, idx)
        err = np.abs(num - grad).max() / max(np.abs(grad).max(), 1e-30)
        assert err < 1e-6, (name, err)


def test_backward_matches_torch_autograd():
    """Library route: torch float64 autograd of the materialised formulation."""
    torch = pytest.importorskip("torch")
    lengths, H, M, d = [7, 0, 12], 2, 6, 5
    K, V, P, off = rand_case(19, lengths, H, M, d)
    B = len(lengths)
    R = 3
    dS = np.random.default_rng(20).standard_normal((B, R, H, M, d)).astype(np.float32)
    sc = 1.0 / math.sqrt(d)
    dK, dV, dP = oracle.bwd(K, V, P, off, dS)
    tK = torch.tensor(K, dtype=torch.float64, requires_grad=True)
    tV = torch.tensor(V, dtype=torch.float64, requires_grad=True)
    tP = torch.tensor(P, dtype=torch.float64, requires_grad=True)
    loss = 0
    for b in range(B):
        s, e = off[b], off[b + 1]
        for h in range(H):
            S = sc * tP[h] @ tK[s:e, h, :].T            # k x n
            A = torch.softmax(S, dim=0)                  # over prototypes
            X = A @ tV[s:e, h, :]
            for r in range(R):
                loss = loss + (X * torch.tensor(dS[b, r, h], dtype=torch.float64)).sum()
    loss.backward()
    np.testing.assert_allclose(dK, tK.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, tV.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dP, tP.grad.numpy(), rtol=1e-10, atol=1e-12)


# ---------------------------------------------------------------- P9 invariants
def test_backward_invariants():
    lengths, H, M, d = [11, 4, 9], 2, 12, 8
    K, V, P, off = rand_case(21, lengths, H, M, d, scale_p=0.4)
    B = len(lengths)
    dS = np.random.default_rng(22).standard_normal((B, 2, H, M, d)).astype(np.float32)
    dY = dS.astype(np.float64).sum(axis=1)
    dK, dV, dP = oracle.bwd(K, V, P, off, dS)
    sk, _ = oracle.fwd(K, V, P, off)
    # shift invariance in P  =>  sum over prototypes of dP is zero
    np.testing.assert_allclose(dP.sum(axis=1), 0.0, atol=1e-10)
    # logits are bilinear in (K, P)  =>  <dK, K> = <dP, P> per head
    for h in range(H):
        np.testing.assert_allclose((dK[:, h] * K[:, h]).sum(), (dP[h] * P[h]).sum(),
                                   rtol=1e-9, atol=1e-10)
    # the sketch is linear in V  =>  <dV, V> = <dY, sketch> per (user, head)
    for b in range(B):
        for h in range(H):
            lhs = (dV[off[b]:off[b + 1], h] * V[off[b]:off[b + 1], h]).sum()
            np.testing.assert_allclose(lhs, (dY[b, h] * sk[b, h]).sum(), rtol=1e-10, atol=1e-11)


# ---------------------------------------------------------------- P10 closed forms
def test_backward_closed_forms():
    lengths, H, M, d = [5, 6], 2, 7, 4
    K, V, P, off = rand_case(23, lengths, H, M, d)
    B = len(lengths)
    g = np.random.default_rng(24).standard_normal((B, 1, H, 1, d)).astype(np.float32)
    # the same upstream gradient for every prototype: dV_t = g, dK = dP = 0
    dS = np.broadcast_to(g, (B, 1, H, M, d)).copy()
    dK, dV, dP = oracle.bwd(K, V, P, off, dS)
    for b in range(B):
        np.testing.assert_allclose(dV[off[b]:off[b + 1]], np.broadcast_to(g[b, 0, :, 0, :], (lengths[b], H, d)),
                                   rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dK, 0.0, atol=1e-12)
    np.testing.assert_allclose(dP, 0.0, atol=1e-12)
    # M = 1: dV_t = dY_0, dK = dP = 0
    K1, V1, P1, off1 = rand_case(25, lengths, H, 1, d)
    dS1 = np.random.default_rng(26).standard_normal((B, 1, H, 1, d)).astype(np.float32)
    dK1, dV1, dP1 = oracle.bwd(K1, V1, P1, off1, dS1)
    for b in range(B):
        np.testing.assert_allclose(dV1[off1[b]:off1[b + 1]], np.broadcast_to(dS1[b, 0, :, 0, :], (lengths[b], H, d)),
                                   rtol=1e-12)
    assert np.all(dK1 == 0) and np.all(dP1 == 0)
    # V = 0: no gradient flows into the logits
    dS2 = np.random.default_rng(27).standard_normal((B, 1, H, M, d)).astype(np.float32)
    dK2, dV2, dP2 = oracle.bwd(K, np.zeros_like(V), P, off, dS2)
    assert np.all(dK2 == 0) and np.all(dP2 == 0)


# ---------------------------------------------------------------- P11 MRLB
def test_mrlb_sum_of_target_gradients():
    """Section 4.2: one sketch reused by R targets receives the sum of their gradients."""
    lengths, H, M, d = [6, 3], 2, 8, 4
    K, V, P, off = rand_case(28, lengths, H, M, d)
    dS = np.random.default_rng(29).standard_normal((2, 4, H, M, d)).astype(np.float32)
    gR = oracle.bwd(K, V, P, off, dS)
    g1 = oracle.bwd(K, V, P, off, dS.astype(np.float64).sum(axis=1, keepdims=True).astype(np.float32))
    # fp32 rounding of the summed dY is the only difference
    for a, b in zip(gR, g1):
        np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-6)


# ---------------------------------------------------------------- P12 exact integer case
def test_exact_integer_sketch_with_uniform_weights():
    """P = 0 and M a power of two: A = 1/M exactly, V small integers => every sketch value
    is an exactly representable fp32 (the bit-exact ragged GPU test relies on this)."""
    lengths = [5, 0, 33, 1, 70]
    H, M, d = 2, 8, 4
    T = sum(lengths)
    off = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=off[1:])
    K = np.random.default_rng(30).standard_normal((T, H, d)).astype(np.float32)
    P = np.zeros((H, M, d), np.float32)
    V = np.zeros((T, H, d), np.float32)
    for b in range(len(lengths)):
        V[off[b]:off[b + 1], :, 0] = b + 1
    V[:, :, 1] = (np.arange(T) % 4)[:, None]
    sk, lse = oracle.fwd(K, V, P, off)
    for b in range(len(lengths)):
        exp0 = lengths[b] * (b + 1) / M
        assert np.all(sk[b, :, :, 0] == exp0)
        assert np.all(sk[b, :, :, 1] == (np.arange(off[b], off[b + 1]) % 4).sum() / M)
    np.testing.assert_allclose(lse, math.log(M), rtol=0, atol=1e-15)


# ---------------------------------------------------------------- generator sanity
def test_generator_is_seeded_and_per_user():
    w = wl.custom([4, 0, 6], H=2, M=8, d=4, seed=99)
    a = wl.host_tensors(w)
    b = wl.host_tensors(w)
    np.testing.assert_array_equal(a["K"], b["K"])
    # regenerating one user alone gives the same slice
    u2 = wl.host_user(w, 2)
    np.testing.assert_array_equal(u2["K"], a["K"][4:10])
    # bf16 values are exactly representable
    assert np.array_equal(wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(a["K"])), a["K"])


def test_loguniform_lengths_recipe():
    w = wl.config(3)
    assert w.B == 32 and w.lengths.min() >= 1000 and w.lengths.max() <= 100_000
    assert np.array_equal(w.lengths, wl.config(5).lengths)

"""GPU parity of the SA layer with its projections (sa_layer_fwd / sa_layer_bwd:
Q = P W_Q, K = X W_K, sketch = softmax_proto(scale Q K^T) X; Appendix G.3)
against the fp64 numpy layer oracle, through the C ABI.

Tolerances as for the sketching step: normwise max relative error per (user,
head) slice for the sketch and dX, per head for dP, dW_Q and dW_K, <= 2e-2
(bf16) / 1e-4 (fp32); lse absolute error <= 1e-3 (bf16) / 1e-5 (fp32).  In
bf16 mode the library rounds P' = P W_Q W_K^T to bf16 once; the error budget
of that rounding is the same 2^-9 relative as the bf16 inputs.
"""
import numpy as np
import pytest

from oracle import layer as olayer
from paper_2609_08443_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "fp32": 1e-4}
LSE_TOL = {"bf16": 1e-3, "fp32": 1e-5}


@pytest.fixture(scope="module")
def sa():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_08443_amd import sa_sketch
    sa_sketch.lib()
    return sa_sketch


def normwise(gpu, ref, axes):
    err = np.abs(gpu.astype(np.float64) - ref).max(axis=axes)
    den = np.abs(ref).max(axis=axes)
    return err / np.maximum(den, 1e-30)


def make(lengths, H, M, d, dtype, seed, R=2):
    w = wl.custom(lengths, H, M, d, dtype, seed=seed, R=R, bwd=True)
    host = wl.host_tensors(w)
    host.update(wl.host_projections(w))
    host["X"] = host.pop("V")
    del host["K"]
    return w, host, wl.to_device(host, dtype)


def check(sa, lengths, H, M, d, dtype, seed):
    w, host, dev = make(lengths, H, M, d, dtype, seed)
    print(f"layer case lengths={lengths} H={H} M={M} d={d} {dtype}", flush=True)
    sk, lse = sa.layer_fwd(dev["X"], dev["P"], dev["Wq"], dev["Wk"], dev["offsets"], w.scale)
    dX, dP, dWq, dWk = sa.layer_bwd(dev["X"], dev["P"], dev["Wq"], dev["Wk"], dev["offsets"],
                                    dev["dsketch"], lse, w.scale)
    torch.cuda.synchronize()
    args = (host["X"], host["P"], host["Wq"], host["Wk"], host["offsets"])
    rs, rl = olayer.layer_fwd(*args, scale=w.scale)
    rX, rP, rWq, rWk = olayer.layer_bwd(*args, host["dsketch"], scale=w.scale)
    tol = TOL[dtype]
    nonempty = np.asarray(w.lengths) > 0
    e = normwise(sk.cpu().numpy(), rs, (2, 3))
    assert np.all(e[nonempty] <= tol), ("sketch", e[nonempty].max())
    assert np.all(sk.cpu().numpy()[~nonempty] == 0)
    le = np.abs(lse.cpu().numpy() - rl).max() if w.T else 0.0
    assert le <= LSE_TOL[dtype], ("lse", le)
    gX = dX.cpu().numpy()
    off = host["offsets"]
    for b in range(w.B):
        if off[b + 1] == off[b]:
            continue
        eb = normwise(gX[off[b]:off[b + 1]], rX[off[b]:off[b + 1]], (0, 2))
        assert np.all(eb <= tol), ("dX", b, eb.max())
    for name, g, r in (("dP", dP, rP), ("dWq", dWq, rWq), ("dWk", dWk, rWk)):
        eh = normwise(g.cpu().numpy(), r, (1, 2))
        assert np.all(eh <= tol), (name, eh.max())


FUSED_CASES = [
    ([37, 0, 70, 1, 5], 2, 128, 64),
    ([300, 17, 64], 2, 512, 128),
    ([96, 31, 200], 2, 256, 64),
    ([2000, 3, 513], 4, 512, 128),
]


@pytest.mark.parametrize("lengths,H,M,d", FUSED_CASES)
def test_layer_fused_matches_oracle(sa, lengths, H, M, d):
    check(sa, lengths, H, M, d, "bf16", seed=3 * sum(lengths) + M + d)


PLAIN_CASES = [
    ([40, 0, 77], 2, 64, 64, "fp32"),
    ([50, 9], 1, 200, 128, "fp32"),
    ([33, 64], 2, 64, 64, "bf16"),     # M not a multiple of 128: plain path in bf16
]


@pytest.mark.parametrize("lengths,H,M,d,dtype", PLAIN_CASES)
def test_layer_plain_matches_oracle(sa, lengths, H, M, d, dtype):
    check(sa, lengths, H, M, d, dtype, seed=5 * sum(lengths) + M + d)


def test_identity_projections_equal_sketching_step(sa):
    # W_Q = W_K = I: P' = P exactly, so the layer forward is the sketching forward
    # with K = V = X bit for bit; its dX is dK + dV of the sketching backward
    w, host, dev = make([150, 0, 61, 300], 2, 256, 128, "bf16", seed=21)
    eye = torch.eye(w.d, dtype=torch.bfloat16, device="cuda").expand(w.H, w.d, w.d).contiguous()
    X, P, off = dev["X"], dev["P"], dev["offsets"]
    sk, lse = sa.layer_fwd(X, P, eye, eye, off, w.scale)
    sk2, lse2 = sa.sketch_fwd(X, X, P, off, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(sk, sk2) and torch.equal(lse, lse2)
    dX, dP, _, _ = sa.layer_bwd(X, P, eye, eye, off, dev["dsketch"], lse, w.scale)
    dK, dV, dP2 = sa.sketch_bwd(X, X, P, off, dev["dsketch"], lse2, w.scale)
    torch.cuda.synchronize()
    ref = (dK + dV).cpu().numpy().astype(np.float64)
    err = np.abs(dX.cpu().numpy() - ref).max() / np.abs(ref).max()
    assert err <= 1e-2, err
    np.testing.assert_array_equal(dP.cpu().numpy(), dP2.cpu().numpy())


def test_layer_deterministic(sa):
    w, host, dev = make([700, 41, 0, 333], 2, 256, 128, "bf16", seed=23)
    a = [dev[k] for k in ("X", "P", "Wq", "Wk", "offsets")]
    s1, l1 = sa.layer_fwd(*a, w.scale)
    g1 = sa.layer_bwd(*a, dev["dsketch"], l1, w.scale)
    s2, l2 = sa.layer_fwd(*a, w.scale)
    g2 = sa.layer_bwd(*a, dev["dsketch"], l2, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(l1, l2)
    for x, y in zip(g1, g2):
        assert torch.equal(x, y)

"""GPU parity of the reordered single-query STCA over the sketch (sa_stca_fwd /
sa_stca_bwd, Appendix G.2) against the fp64 numpy oracle, through the C ABI.

Tolerances: normwise max relative error <= 2e-2 (bf16) / 1e-4 (fp32) per
(user, target) row block for the output and dq, per user for dXs, per head's
column block for dW_Q, dW_K, dW_V.  lse absolute error: fp32 1e-4; bf16 mode
rounds q W_Q, u = (q W_Q) W_K^T and the logits themselves to bf16 once each, so a
logit of magnitude |s| moves by up to about 3 * 2^-9 |s|; the bound is
2^-7 max(1, max |s|).
The cases mix products that run on the matrix cores (every contraction length
a multiple of 64) with ones that do not (the register-tiled fallback).
"""
import numpy as np
import pytest

from oracle import stca as ostca
from paper_2609_08443_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "fp32": 1e-4}


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


def run(sa, B, R, k, D, h, dtype, seed, bwd=True):
    host = wl.host_stca(seed, B, R, k, D, dtype)
    dev = wl.to_device(host, dtype)
    print(f"stca case B={B} R={R} k={k} D={D} h={h} {dtype}", flush=True)
    args = [dev[n] for n in ("Xs", "q", "Wq", "Wk", "Wv")]
    out, lse = sa.stca_fwd(*args, h=h, want_lse=True)
    g = sa.stca_bwd(*args, h=h, dout=dev["dout"]) if bwd else None
    torch.cuda.synchronize()
    hargs = [host[n] for n in ("Xs", "q", "Wq", "Wk", "Wv")]
    rout, rlse = ostca.stca_fwd(*hargs, h=h)
    ref = ostca.stca_bwd(*hargs, h=h, dout=host["dout"]) if bwd else None
    return host, out.cpu().numpy(), lse.cpu().numpy(), rout, rlse, \
        ({k_: v.cpu().numpy() for k_, v in g.items()} if bwd else None), ref


def check(res, h, dtype):
    host, out, lse, rout, rlse, g, ref = res
    tol = TOL[dtype]
    e = normwise(out, rout, (2,))
    assert np.all(e <= tol), ("out", e.max())
    if dtype == "fp32":
        lt = 1e-4
    else:
        s_max = np.abs(rlse).max() + np.log(host["Xs"].shape[1])
        lt = 2.0 ** -7 * max(1.0, s_max)
    assert np.abs(lse - rlse).max() <= lt, ("lse", np.abs(lse - rlse).max(), lt)
    if g is None:
        return
    e = normwise(g["dXs"], ref["dXs"], (1, 2))
    assert np.all(e <= tol), ("dXs", e.max())
    e = normwise(g["dq"], ref["dq"], (2,))
    assert np.all(e <= tol), ("dq", e.max())
    D = out.shape[-1]
    dh = D // h
    for name in ("dWq", "dWk", "dWv"):
        for i in range(h):
            cols = slice(i * dh, (i + 1) * dh)
            e = normwise(g[name][:, cols], ref[name][:, cols], (0, 1))
            assert e <= tol, (name, i, e)


CASES = [
    (4, 16, 192, 256, 4, "bf16"),    # every product on the matrix cores
    (3, 5, 128, 256, 4, "bf16"),     # weight gradients and dXs (k = 15, 20 rows) on the fallback
    (2, 16, 256, 512, 8, "bf16"),
    (2, 8, 100, 128, 2, "bf16"),     # k = 100: partial tiles, aggregation on the fallback
    (1, 4, 600, 128, 2, "bf16"),     # k = 600: the widest register-resident softmax rows, partly filled
    (2, 3, 50, 64, 2, "fp32"),
    (1, 7, 33, 96, 3, "fp32"),
]


@pytest.mark.parametrize("B,R,k,D,h,dtype", CASES)
def test_stca_matches_oracle(sa, B, R, k, D, h, dtype):
    check(run(sa, B, R, k, D, h, dtype, seed=7 * B + R + k + D + h), h, dtype)


def test_stca_single_sketch_row_and_determinism(sa):
    # k = 1: every weight is one and the output is Xs_0 W_V for every target
    res = run(sa, 2, 4, 1, 128, 2, "bf16", seed=3)
    check(res, 2, "bf16")
    res2 = run(sa, 2, 4, 1, 128, 2, "bf16", seed=3)
    for a, b in zip(res[1:3], res2[1:3]):
        np.testing.assert_array_equal(a, b)
    for key in res[5]:
        np.testing.assert_array_equal(res[5][key], res2[5][key])


def test_stca_zero_users_is_a_no_op(sa):
    dev = wl.to_device(wl.host_stca(5, 0, 3, 64, 128, "bf16"), "bf16")
    out, _ = sa.stca_fwd(*[dev[n] for n in ("Xs", "q", "Wq", "Wk", "Wv")], h=2)
    torch.cuda.synchronize()
    assert out.shape == (0, 3, 128)

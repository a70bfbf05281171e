"""GPU parity of the token-wise normalised forward (sa_sketch_fwd_tokenwise)
against the fp64 CPU oracle, through the C ABI.

Tolerances as for the prototype-wise forward: normwise max relative error per
(user, head) slice <= 2e-2 (bf16) / 1e-4 (fp32); per-prototype lse absolute
error <= 1e-3 (bf16) / 1e-5 (fp32).  Empty users must give a zero sketch and
lse_m = -inf.  Small token counts make the work-list ranges short, so most
users are cut across several ranges and the log-sum-exp merge is exercised.
"""
import numpy as np
import pytest

import oracle
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


def run_case(sa, w):
    host = wl.host_tensors(w)
    dev = wl.to_device(host, w.dtype)
    print(f"tokenwise case {w.name} B={w.B} T={w.T} H={w.H} M={w.M} d={w.d} {w.dtype}", flush=True)
    sk, lse = sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    torch.cuda.synchronize()
    ref_sk, ref_lse = oracle.fwd_tokenwise(host["K"], host["V"], host["P"], host["offsets"], w.scale)
    g = sk.cpu().numpy()
    gl = lse.cpu().numpy()
    nonempty = np.asarray(w.lengths) > 0
    e = normwise(g, ref_sk, (2, 3))
    assert np.all(e[nonempty] <= TOL[w.dtype]), (w.name, e[nonempty].max())
    assert np.all(g[~nonempty] == 0), "empty users must get a zero sketch"
    assert np.all(np.isneginf(gl[~nonempty])), "empty users must get lse_m = -inf"
    le = np.abs(gl[nonempty] - ref_lse[nonempty]).max() if nonempty.any() else 0.0
    assert le <= LSE_TOL[w.dtype], (w.name, le)
    return sk, lse


FUSED_CASES = [
    ([37, 0, 70, 1, 5], 2, 128, 64),
    ([100, 33], 1, 256, 64),
    ([300, 17, 64], 2, 1024, 64),
    ([29, 70, 0, 95], 2, 128, 128),
    ([260, 1], 1, 512, 128),
    ([96, 31, 200], 2, 384, 128),
    ([2000, 3, 513], 4, 512, 128),
]


@pytest.mark.parametrize("lengths,H,M,d", FUSED_CASES)
def test_tokenwise_fused_matches_oracle(sa, lengths, H, M, d):
    w = wl.custom(lengths, H, M, d, "bf16", seed=7 * sum(lengths) + M + d)
    run_case(sa, w)


PLAIN_CASES = [
    ([40, 0, 77], 2, 64, 64, "fp32"),
    ([50, 9], 1, 200, 128, "fp32"),
    ([33, 64], 2, 64, 64, "bf16"),      # M not a multiple of 128: plain path
    ([2048], 1, 64, 64, "fp32"),        # the single-user fp32 configuration's shape
]


@pytest.mark.parametrize("lengths,H,M,d,dtype", PLAIN_CASES)
def test_tokenwise_plain_matches_oracle(sa, lengths, H, M, d, dtype):
    w = wl.custom(lengths, H, M, d, dtype, seed=11 * sum(lengths) + M + d)
    run_case(sa, w)


def test_tokenwise_deterministic(sa):
    w = wl.custom([700, 41, 0, 333], 2, 256, 128, "bf16", seed=5)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, w.dtype)
    a, la = sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    b, lb = sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_tokenwise_single_token_users(sa):
    # one token: every prototype's row is that token's V (exactly, up to the
    # bf16 MFMA round trip of a weight equal to 1)
    w = wl.custom([1, 1, 1], 2, 128, 64, "bf16", seed=3)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, w.dtype)
    sk, _ = sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    torch.cuda.synchronize()
    g = sk.cpu().numpy()
    V = host["V"].astype(np.float64)
    for b in range(3):
        np.testing.assert_array_equal(g[b], np.broadcast_to(V[b][:, None, :], (2, 128, 64)))


def test_tokenwise_sums_to_one(sa):
    # V = 1: each sketch row is the sum of its weights over the user's tokens
    w = wl.custom([333, 64, 5], 2, 256, 64, "bf16", seed=9)
    host = wl.host_tensors(w)
    host["V"] = np.ones_like(host["V"])
    dev = wl.to_device(host, w.dtype)
    sk, _ = sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    torch.cuda.synchronize()
    np.testing.assert_allclose(sk.cpu().numpy(), 1.0, rtol=0, atol=1e-2)

"""GPU parity of the HIP path against the fp64 CPU oracle, through the C ABI.

Tolerances (stated by the benchmark spec, applied as in the oracle's
reading): normwise max relative error per (user, head) slice,
max|gpu - ref| / max|ref|, <= 2e-2 for bf16 inputs and <= 1e-4 in fp32 mode;
lse absolute error <= 1e-3 (bf16) / 1e-5 (fp32).  Integer work (the work
list) and the exactly representable ragged case are compared bit for bit.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import worklist as wlref
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


def run_case(sa, w, check_lse=True):
    host = wl.host_tensors(w)
    dev = wl.to_device(host, w.dtype)
    print(f"case {w.name} B={w.B} T={w.T}", flush=True)
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    torch.cuda.synchronize()
    ref_sk, ref_lse = oracle.fwd(host["K"], host["V"], host["P"], host["offsets"], w.scale)
    g = sk.cpu().numpy()
    e = normwise(g, ref_sk, (2, 3))
    nonempty = np.asarray(w.lengths) > 0
    assert np.all(e[nonempty] <= TOL[w.dtype]), (w.name, e.max())
    assert np.all(g[~nonempty] == 0), "empty users must get a zero sketch"
    if check_lse and w.T:
        le = np.abs(lse.cpu().numpy() - ref_lse).max()
        assert le <= LSE_TOL[w.dtype], (w.name, le)
    return host, dev, sk, lse, e


# shapes: several 32-token tiles with ragged tails, empty users, both paths
FUSED_CASES = [
    ([37, 0, 70, 1, 5], 2, 128, 64),
    ([100, 33], 1, 256, 64),
    ([65, 3, 0, 130], 3, 512, 64),
    ([300, 17, 64], 2, 1024, 64),
    ([29, 70, 0, 95], 2, 128, 128),
    ([260, 1], 1, 512, 128),
    ([96, 31, 200], 2, 384, 128),
    # every other fused instance: d = 64 with 3, 5, 6, 7 prototype tiles per wave,
    # d = 128 with 2
    ([45, 0, 97, 3], 2, 384, 64),
    ([70, 33, 1], 1, 640, 64),
    ([130, 0, 64], 2, 768, 64),
    ([99, 1, 40], 1, 896, 64),
    ([61, 0, 140, 2], 2, 256, 128),
]


@pytest.mark.parametrize("lengths,H,M,d", FUSED_CASES)
def test_fused_fwd_matches_oracle(sa, lengths, H, M, d):
    w = wl.custom(lengths, H, M, d, "bf16", seed=sum(lengths) + M + d)
    run_case(sa, w)


GENERIC_CASES = [
    ([40, 0, 77], 2, 64, 64, "fp32"),
    ([50, 9], 1, 200, 128, "fp32"),
    ([33, 64], 2, 64, 64, "bf16"),     # M not a multiple of 128 -> plain path
    ([45], 1, 100, 128, "bf16"),
    ([70, 2], 1, 256, 64, "fp32"),
]


@pytest.mark.parametrize("lengths,H,M,d,dtype", GENERIC_CASES)
def test_plain_path_fwd_matches_oracle(sa, lengths, H, M, d, dtype):
    w = wl.custom(lengths, H, M, d, dtype, seed=7 + sum(lengths))
    run_case(sa, w)


def test_config1_fp32_single_user(sa):
    w = wl.config(1)
    _, _, _, _, e = run_case(sa, w)
    assert e.max() <= 1e-4


@pytest.mark.parametrize("M,d", [(256, 64), (512, 128)])
def test_fused_split_users_across_ranges(sa, M, d):
    """Users longer than a workgroup range: the split-L merge sums partial sketches."""
    w = wl.custom([5000, 12, 7000, 0, 2500], 2, M, d, "bf16", seed=5)
    host, dev, sk, lse, e = run_case(sa, w)
    C = sa.fwd_chunk_tokens(w.B, w.T, w.H, w.M, w.d, 0)
    assert C < 5000 * 2, "the case must actually split users across ranges"


def test_exact_ragged_sketch_bit_for_bit(sa):
    """P = 0, M = 128: every weight is exactly 1/128; V holds small integers tagging the user.
    Every sketch value is then an exact fp32, so the GPU must match the oracle bit for bit
    (catches offset, work-list, split-L and cross-user leakage mistakes)."""
    lengths = [5, 0, 33, 1, 70, 2048, 9000, 31, 32, 64]
    H, M, d = 2, 128, 64
    w = wl.custom(lengths, H, M, d, "bf16", seed=11)
    host = wl.host_tensors(w)
    host["P"][:] = 0
    V = np.zeros_like(host["V"])
    off = host["offsets"]
    for b in range(w.B):
        V[off[b]:off[b + 1], :, 0] = b + 1
        V[off[b]:off[b + 1], 1, 2] = -(b + 1)
    V[:, :, 1] = (np.arange(w.T) % 4)[:, None]
    host["V"] = V
    dev = wl.to_device(host, "bf16")
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
    ref, ref_lse = oracle.fwd(host["K"], host["V"], host["P"], off, w.scale)
    g = sk.cpu().numpy()
    assert np.array_equal(g, ref.astype(np.float32)), np.abs(g - ref).max()
    assert np.array_equal(ref.astype(np.float32).astype(np.float64), ref)


@pytest.mark.parametrize("offsets,H,C", [
    ([0, 5, 5, 17, 18], 2, 4), ([0, 100], 3, 32), ([0, 0, 0], 2, 7), ([0, 1, 2, 3], 1, 1),
    ([0, 64, 64, 200], 2, 64), ([0, 1000, 1500, 99999], 4, 2688), ([0, 3], 5, 100000)])
def test_worklist_bit_exact(sa, offsets, H, C):
    T = offsets[-1]
    off = torch.tensor(offsets, dtype=torch.int64, device="cuda")
    items = sa.build_worklist(off, T, H, C).cpu().numpy()
    ref = np.asarray(wlref.worklist(offsets, T, H, C), dtype=np.int32).reshape(-1, 8)
    assert items.shape == ref.shape
    assert np.array_equal(items, ref)


def test_worklist_of_config3(sa):
    w = wl.config(3)
    off = torch.from_numpy(w.offsets).cuda()
    C = sa.fwd_chunk_tokens(w.B, w.T, w.H, w.M, w.d, 0)
    items = sa.build_worklist(off, w.T, w.H, C).cpu().numpy()
    ref = np.asarray(wlref.worklist(list(w.offsets), w.T, w.H, C), dtype=np.int32).reshape(-1, 8)
    assert np.array_equal(items, ref)


def test_fwd_is_deterministic(sa):
    w = wl.custom([3000, 50, 4100], 2, 512, 64, "bf16", seed=3)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, "bf16")
    a1, l1 = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    a2, l2 = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    assert torch.equal(a1, a2) and torch.equal(l1, l2)


def test_fwd_properties_mass_and_permutation(sa):
    """sum_m sketch = sum_t V (per-token weights sum to 1), and token order inside a
    user does not matter (up to the fp32 summation order)."""
    w = wl.custom([500, 77], 2, 256, 64, "bf16", seed=8)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, "bf16")
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    g = sk.cpu().numpy().astype(np.float64)
    for b in range(w.B):
        vs = host["V"][w.offsets[b]:w.offsets[b + 1]].astype(np.float64).sum(0)
        err = np.abs(g[b].sum(axis=1) - vs).max() / np.abs(vs).max()
        assert err < 2e-2
    perm = np.concatenate([np.random.default_rng(1).permutation(500), 500 + np.arange(77)[::-1]])
    host2 = dict(host, K=host["K"][perm], V=host["V"][perm])
    dev2 = wl.to_device(host2, "bf16")
    sk2, lse2 = sa.sketch_fwd(dev2["K"], dev2["V"], dev2["P"], dev2["offsets"])
    assert np.abs(sk2.cpu().numpy() - g).max() / np.abs(g).max() < 1e-5
    # per-token work is position independent: lse moves with its token, bit for bit
    assert torch.equal(lse2.cpu(), lse.cpu()[torch.from_numpy(perm)])


def test_fwd_without_lse_and_zero_users(sa):
    w = wl.custom([40, 90], 1, 128, 64, "bf16", seed=4)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, "bf16")
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"], want_lse=False)
    assert lse is None
    ref, _ = oracle.fwd(host["K"], host["V"], host["P"], host["offsets"])
    assert normwise(sk.cpu().numpy(), ref, (2, 3)).max() <= 2e-2
    # all users empty: zero sketches
    w0 = wl.custom([0, 0, 0], 2, 128, 64, "bf16", seed=4)
    dev0 = wl.to_device(wl.host_tensors(w0), "bf16")
    sk0, _ = sa.sketch_fwd(dev0["K"], dev0["V"], dev0["P"], dev0["offsets"])
    assert torch.count_nonzero(sk0).item() == 0


# ------------------------------------------------------------------ backward
BWD_CASES = [
    ([37, 0, 70, 5], 2, 128, 64, "bf16", 1),
    ([100, 33], 1, 256, 64, "bf16", 4),
    ([29, 70, 0, 95], 2, 128, 128, "bf16", 2),
    ([260, 1], 1, 512, 128, "bf16", 4),
    ([40, 0, 77], 2, 64, 64, "fp32", 3),
    ([33, 64], 2, 64, 128, "bf16", 1),
    # d = 64 with M a multiple of 512: the dP kernel with two prototype tiles per
    # wave and its P / dY slices in LDS; an empty user, and users long enough to be
    # cut into several segments, so dP sums partials of several ranges
    ([300, 0, 1200, 7], 2, 512, 64, "bf16", 2),
    ([700, 0, 45, 1500], 2, 1024, 64, "bf16", 4),
]


@pytest.mark.parametrize("lengths,H,M,d,dtype,R", BWD_CASES)
def test_bwd_matches_oracle(sa, lengths, H, M, d, dtype, R):
    w = wl.custom(lengths, H, M, d, dtype, seed=100 + sum(lengths), R=R, bwd=True)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, dtype)
    print(f"bwd case {w.name}", flush=True)
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    dK, dV, dP = sa.sketch_bwd(dev["K"], dev["V"], dev["P"], dev["offsets"], dev["dsketch"], lse)
    torch.cuda.synchronize()
    rK, rV, rP = oracle.bwd(host["K"], host["V"], host["P"], host["offsets"], host["dsketch"])
    tol = TOL[dtype]
    off = host["offsets"]
    for b in range(w.B):
        s, e = off[b], off[b + 1]
        if e == s:
            continue
        for h in range(H):
            for name, gg, rr in (("dK", dK, rK), ("dV", dV, rV)):
                gs = gg[s:e, h].cpu().numpy().astype(np.float64)
                rs = rr[s:e, h]
                err = np.abs(gs - rs).max() / max(np.abs(rs).max(), 1e-30)
                assert err <= tol, (name, b, h, err)
    gP = dP.cpu().numpy().astype(np.float64)
    for h in range(H):
        err = np.abs(gP[h] - rP[h]).max() / max(np.abs(rP[h]).max(), 1e-30)
        assert err <= tol, ("dP", h, err)


def test_bwd_users_split_across_ranges(sa):
    """Long users are cut into several segments; dK/dV are per token, dP sums every segment."""
    w = wl.custom([3000, 5, 2100, 0, 700], 2, 256, 64, "bf16", seed=77, R=2, bwd=True)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, "bf16")
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    dK, dV, dP = sa.sketch_bwd(dev["K"], dev["V"], dev["P"], dev["offsets"], dev["dsketch"], lse)
    torch.cuda.synchronize()
    rK, rV, rP = oracle.bwd(host["K"], host["V"], host["P"], host["offsets"], host["dsketch"])
    off = host["offsets"]
    for b in range(w.B):
        s, e = off[b], off[b + 1]
        if e == s:
            continue
        for h in range(w.H):
            for gg, rr in ((dK, rK), (dV, rV)):
                g = gg[s:e, h].cpu().numpy().astype(np.float64)
                assert np.abs(g - rr[s:e, h]).max() / np.abs(rr[s:e, h]).max() <= 2e-2
    g = dP.cpu().numpy().astype(np.float64)
    for h in range(w.H):
        assert np.abs(g[h] - rP[h]).max() / np.abs(rP[h]).max() <= 2e-2


def test_bwd_is_deterministic(sa):
    w = wl.custom([1500, 40, 900], 2, 512, 128, "bf16", seed=78, R=4, bwd=True)
    dev = wl.to_device(wl.host_tensors(w), "bf16")
    _, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    g1 = sa.sketch_bwd(dev["K"], dev["V"], dev["P"], dev["offsets"], dev["dsketch"], lse)
    g2 = sa.sketch_bwd(dev["K"], dev["V"], dev["P"], dev["offsets"], dev["dsketch"], lse)
    for a_, b_ in zip(g1, g2):
        assert torch.equal(a_, b_)


# (M, d) = (256, 64) reads the next tile's operands after the bound check, the
# other two before it (four or more prototype tiles per wave)
@pytest.mark.parametrize("M,d", [(256, 64), (512, 128), (1024, 64)])
def test_fwd_loose_bound_falls_back_to_exact_max(sa, M, d):
    """Keys of huge norm nearly orthogonal to every prototype: the logits sit far below
    the Cauchy-Schwarz shift, so exp(logit - shift) would underflow; the tile is
    recomputed with the exact per-token max and still matches the oracle."""
    rng = np.random.default_rng(5)
    lengths = [70, 33, 129]
    w = wl.custom(lengths, 2, M, d, "bf16", seed=9)
    host = wl.host_tensors(w)
    T = w.T
    K = np.zeros((T, 2, d), np.float32)
    K[:, :, 0] = 2048.0                                  # |K_t| = 2048 along axis 0
    K[:, :, 1:] = rng.standard_normal((T, 2, d - 1)).astype(np.float32)
    P = (rng.standard_normal((2, M, d)) * 4.0).astype(np.float32)
    P[:, :, 0] = (rng.integers(-8, 9, (2, M)) / 512.0)   # tiny overlap with axis 0
    # every other token gets an ordinary key, so tiles mix both regimes
    K[::2] = rng.standard_normal((len(K[::2]), 2, d)).astype(np.float32)
    host["K"] = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(K))
    host["P"] = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(P))
    dev = wl.to_device(host, "bf16")
    sk, lse = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    ref, ref_lse = oracle.fwd(host["K"], host["V"], host["P"], host["offsets"])
    # the bound is far above the logits (otherwise this case tests nothing)
    s_max = np.max(np.einsum("thd,hmd->thm", host["K"].astype(np.float64),
                             host["P"].astype(np.float64)), axis=2) / math.sqrt(d)
    bound = np.linalg.norm(host["K"], axis=2) * np.linalg.norm(host["P"], axis=2).max(axis=1) / math.sqrt(d)
    assert (bound - s_max).max() > 200
    g = sk.cpu().numpy()
    assert np.all(np.isfinite(g)) and np.all(np.isfinite(lse.cpu().numpy()))
    assert normwise(g, ref, (2, 3)).max() <= 2e-2
    assert np.abs(lse.cpu().numpy() - ref_lse).max() <= 1e-3 * max(1.0, np.abs(ref_lse).max())


# ------------------------------------------------------------------ offsets validation
# With SA_DEBUG_VALIDATE=1 every entry point copies the offsets to the host and
# rejects malformed ones with SA_ERR_BAD_OFFSETS before any launch; valid
# offsets give the same results as without the check.
def test_debug_validate_rejects_malformed_offsets(sa, monkeypatch):
    w = wl.custom([40, 0, 70], 2, 128, 64, "bf16", seed=91, R=2, bwd=True)
    host = wl.host_tensors(w)
    dev = wl.to_device(host, "bf16")
    sk0, lse0 = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    torch.cuda.synchronize()
    monkeypatch.setenv("SA_DEBUG_VALIDATE", "1")
    sk1, lse1 = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"])
    sa.sketch_bwd(dev["K"], dev["V"], dev["P"], dev["offsets"], dev["dsketch"], lse1)
    torch.cuda.synchronize()
    assert torch.equal(sk0, sk1) and torch.equal(lse0, lse1)
    T = w.T
    bad = {"first not zero": [1, 40, 40, T], "decreasing": [0, 50, 40, T], "last not T": [0, 40, 40, T - 1]}
    for name, o in bad.items():
        off = torch.tensor(o, dtype=torch.int64, device="cuda")
        print(f"malformed offsets case: {name}", flush=True)
        for call in (lambda: sa.sketch_fwd(dev["K"], dev["V"], dev["P"], off),
                     lambda: sa.sketch_bwd(dev["K"], dev["V"], dev["P"], off, dev["dsketch"], lse1),
                     lambda: sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], off)):
            with pytest.raises(sa.SAError) as ei:
                call()
            assert ei.value.status == 4, (name, ei.value)

"""GPU parity of stacked SA (sa_block_fwd: per layer the sketch with the
current state as queries, residual + LN, SwiGLU FFN + residual + LN; section
3.3) against the fp64 numpy block oracle, through the C ABI.

Output tolerance: normwise max relative error per (user, head) slice <= 2e-2
(bf16) / 1e-4 (fp32), as for the other paths.  The first layer's lse keeps the
sketching step's absolute bounds (1e-3 bf16, 1e-5 fp32).

A later layer's logits use per-user prototypes P' = state W_Q W_K^T computed on
the device from the device's own state (and rounded once to bf16 in bf16
mode), so its lse carries two errors, checked separately:
* the sketching step itself: the kernel's lse against the fp64 oracle fed the
  device's own P' (read back from the training forward's saved buffer) must
  meet the first layer's bound;
* the error of P' (the state's error from the earlier layers, plus the bf16
  rounding of P'): changing the prototypes by dP'_m moves lse_t by
  sum_m A_tm scale <X_t, dP'_m>, a weighted mean, so by at most
  scale |X_t| max_m |dP'_m| (Cauchy-Schwarz).  The oracle fed the device's P'
  and the oracle's own block must differ by no more than that, token by token.
"""
import numpy as np
import pytest

from block_lse_check import later_layer_lse
from oracle import block as oblock
from paper_2609_08443_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "fp32": 1e-4}
LSE0 = {"bf16": 1e-3, "fp32": 1e-5}


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


NAMES = ("Wq", "Wk", "ln", "W1", "W3", "W2")


def run(sa, lengths, H, M, d, L, dtype, seed):
    w = wl.custom(lengths, H, M, d, dtype, seed=seed)
    host = wl.host_tensors(w)
    host.update(wl.host_block_params(w, L))
    host["X"] = host.pop("V")
    del host["K"]
    dev = wl.to_device(host, dtype)
    print(f"block case lengths={lengths} H={H} M={M} d={d} L={L} {dtype}", flush=True)
    saved = sa.block_saved_buffer(dev["X"], dev["P"], dev["Wq"], dev["offsets"])
    out, lse = sa.block_fwd(dev["X"], dev["P"], *[dev[k] for k in NAMES], dev["offsets"], w.scale,
                            want_lse=True, saved=saved)
    torch.cuda.synchronize()
    code = sa.SA_BF16 if dtype == "bf16" else sa.SA_FP32
    views = sa.block_saved_views(saved, w.B, w.T, H, M, d, L, code)
    Pp = [None] + [views[l]["Pp"].float().cpu().numpy() for l in range(1, L)]
    ref, rlse = oblock.block_fwd(host["X"], host["P"], *[host[k] for k in NAMES], host["offsets"],
                                 scale=w.scale)
    return w, out.cpu().numpy(), lse.cpu().numpy(), ref, rlse, (host, Pp)


def check(w, out, lse, ref, rlse, extra, dtype):
    e = normwise(out, ref, (2, 3))
    assert np.all(e <= TOL[dtype]), ("out", e.max())
    if w.T:
        assert np.abs(lse[0] - rlse[0]).max() <= LSE0[dtype], ("lse0", np.abs(lse[0] - rlse[0]).max())
        host, Pp = extra
        later_layer_lse(w.scale, host["X"], host["P"], [host[k] for k in NAMES], host["offsets"], Pp, lse, rlse,
                        LSE0[dtype], TOL[dtype])


FUSED = [
    ([37, 0, 70, 1, 5], 2, 128, 64, 2),
    ([300, 17, 64], 2, 512, 128, 2),
    ([96, 31, 200], 1, 256, 64, 3),
    ([2000, 3, 513], 4, 512, 128, 2),
]


@pytest.mark.parametrize("lengths,H,M,d,L", FUSED)
def test_block_fused_matches_oracle(sa, lengths, H, M, d, L):
    check(*run(sa, lengths, H, M, d, L, "bf16", seed=13 * sum(lengths) + M + d + L), "bf16")


PLAIN = [
    ([40, 0, 77], 2, 64, 64, 2, "fp32"),
    ([50, 9], 1, 200, 128, 2, "fp32"),
    ([33, 64], 2, 64, 64, 2, "bf16"),
]


@pytest.mark.parametrize("lengths,H,M,d,L,dtype", PLAIN)
def test_block_plain_matches_oracle(sa, lengths, H, M, d, L, dtype):
    check(*run(sa, lengths, H, M, d, L, dtype, seed=17 * sum(lengths) + M + d), dtype)


def test_block_empty_users_and_determinism(sa):
    # users without tokens get the refinement of the prototypes alone: equal rows
    w, out, lse, ref, rlse, extra = run(sa, [0, 120, 0], 2, 128, 64, 2, "bf16", seed=31)
    np.testing.assert_array_equal(out[0], out[2])
    check(w, out, lse, ref, rlse, extra, "bf16")
    _, out2, lse2, _, _, _ = run(sa, [0, 120, 0], 2, 128, 64, 2, "bf16", seed=31)
    np.testing.assert_array_equal(out, out2)
    np.testing.assert_array_equal(lse, lse2)


# ------------------------------------------------------------------ backward
# sa_block_bwd against the block oracle's chain rule (itself pinned by torch
# autograd and finite differences).  Same bars as the forward: normwise max
# relative error <= 2e-2 (bf16) / 1e-4 (fp32) per (user, head) slice for dX,
# per head for dP and per (layer, head) for each weight and norm gradient.
GNAMES = ("dWq", "dWk", "dln", "dW1", "dW3", "dW2")


def run_bwd(sa, lengths, H, M, d, L, dtype, seed):
    w = wl.custom(lengths, H, M, d, dtype, seed=seed, R=1, bwd=True)
    host = wl.host_tensors(w)
    host.update(wl.host_block_params(w, L))
    host["X"] = host.pop("V")
    del host["K"]
    dout = np.ascontiguousarray(host.pop("dsketch")[:, 0])
    dev = wl.to_device(host, dtype)
    print(f"block bwd case lengths={lengths} H={H} M={M} d={d} L={L} {dtype}", flush=True)
    g = sa.block_bwd(dev["X"], dev["P"], *[dev[k] for k in NAMES], dev["offsets"],
                     torch.tensor(dout, dtype=torch.float32, device="cuda"), w.scale)
    torch.cuda.synchronize()
    ref = oblock.block_bwd(host["X"], host["P"], *[host[k] for k in NAMES], host["offsets"], dout,
                           scale=w.scale)
    return w, host, {k: v.cpu().numpy() for k, v in g.items()}, ref


def check_bwd(w, host, g, ref, dtype):
    tol = TOL[dtype]
    off = host["offsets"]
    for b in range(w.B):
        if off[b + 1] == off[b]:
            continue
        eb = normwise(g["dX"][off[b]:off[b + 1]], ref["dX"][off[b]:off[b + 1]], (0, 2))
        assert np.all(eb <= tol), ("dX", b, eb.max())
    eh = normwise(g["dP"], ref["dP"], (1, 2))
    assert np.all(eh <= tol), ("dP", eh.max())
    for name in GNAMES:
        axes = (3,) if name == "dln" else (2, 3)   # dln: per (layer, parameter, head)
        e = normwise(g[name], ref[name], axes)
        assert np.all(e <= tol), (name, e.max())


BWD_FUSED = [
    ([37, 0, 70, 1, 5], 2, 128, 64, 2),
    ([300, 17, 64], 2, 512, 128, 2),
    ([96, 31, 200], 1, 256, 64, 3),
]


@pytest.mark.parametrize("lengths,H,M,d,L", BWD_FUSED)
def test_block_bwd_fused_matches_oracle(sa, lengths, H, M, d, L):
    check_bwd(*run_bwd(sa, lengths, H, M, d, L, "bf16", seed=19 * sum(lengths) + M + d + L), "bf16")


BWD_PLAIN = [
    ([40, 0, 77], 2, 64, 64, 2, "fp32"),
    ([50, 9], 1, 200, 128, 1, "fp32"),
    ([33, 64], 2, 64, 64, 2, "bf16"),
]


@pytest.mark.parametrize("lengths,H,M,d,L,dtype", BWD_PLAIN)
def test_block_bwd_plain_matches_oracle(sa, lengths, H, M, d, L, dtype):
    check_bwd(*run_bwd(sa, lengths, H, M, d, L, dtype, seed=23 * sum(lengths) + M + d), dtype)


def test_block_bwd_all_users_empty(sa):
    # no tokens at all: every sketch is zero, the gradients flow through the
    # refinement of the prototypes only (dW_Q, dW_K vanish)
    w, host, g, ref = run_bwd(sa, [0, 0], 2, 128, 64, 2, "bf16", seed=37)
    assert g["dX"].shape == (0, 2, 64)
    assert np.count_nonzero(g["dWq"]) == 0 and np.count_nonzero(g["dWk"]) == 0
    check_bwd(w, host, g, ref, "bf16")


def test_block_bwd_deterministic(sa):
    _, _, g1, _ = run_bwd(sa, [500, 0, 77, 260], 2, 256, 128, 2, "bf16", seed=41)
    _, _, g2, _ = run_bwd(sa, [500, 0, 77, 260], 2, 256, 128, 2, "bf16", seed=41)
    for k in g1:
        np.testing.assert_array_equal(g1[k], g2[k], err_msg=k)


# ------------------------------------------------------------------ training mode
# The training forward keeps every layer's intermediates in a caller buffer and
# the backward reads them instead of replaying the forward: the same kernels on
# the same inputs in the same order, so outputs and gradients are bit-identical
# to the inference forward and the replaying backward, and the backward leaves
# the buffer unchanged.
@pytest.mark.parametrize("lengths,H,M,d,L,dtype", [
    ([37, 0, 70, 1, 5], 2, 128, 64, 2, "bf16"),
    ([96, 31, 200], 1, 256, 64, 3, "bf16"),
    ([40, 0, 77], 2, 64, 64, 2, "fp32"),
])
def test_block_saved_matches_replay(sa, lengths, H, M, d, L, dtype):
    w = wl.custom(lengths, H, M, d, dtype, seed=7 * sum(lengths) + L, R=1, bwd=True)
    host = wl.host_tensors(w)
    host.update(wl.host_block_params(w, L))
    host["X"] = host.pop("V")
    del host["K"]
    dout = torch.tensor(np.ascontiguousarray(host.pop("dsketch")[:, 0]), dtype=torch.float32, device="cuda")
    dev = wl.to_device(host, dtype)
    args = (dev["X"], dev["P"], *[dev[k] for k in NAMES], dev["offsets"])
    print(f"block saved case lengths={lengths} H={H} M={M} d={d} L={L} {dtype}", flush=True)
    out0, lse0 = sa.block_fwd(*args, w.scale, want_lse=True)
    g0 = sa.block_bwd(*args, dout, w.scale)
    saved = sa.block_saved_buffer(dev["X"], dev["P"], dev["Wq"], dev["offsets"])
    out1, lse1 = sa.block_fwd(*args, w.scale, want_lse=True, saved=saved)
    before = saved.clone()
    g1 = sa.block_bwd(*args, dout, w.scale, saved=saved)
    g2 = sa.block_bwd(*args, dout, w.scale, saved=saved)
    torch.cuda.synchronize()
    assert torch.equal(out0, out1) and torch.equal(lse0, lse1)
    assert torch.equal(saved, before)
    for k in g0:
        assert torch.equal(g0[k], g1[k]), k
        assert torch.equal(g1[k], g2[k]), k

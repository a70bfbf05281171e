"""Benchmark of the SA sketching step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c5] [--no-cpu-baseline]

A step is one pass of the whole hot path over one batch: sa_sketch_fwd
(work list, fused forward, split-L merge) then sa_sketch_bwd (MRLB target sum,
backward kernels).  The default workload is the ragged 100K batch trained with
4 target instances per user (32 users, log-uniform lengths in [1e3, 1e5],
H = 4, d = 128, M = 512, bf16, R = 4).  Inputs are synthetic, drawn on the
device with fixed seeds, resident in HBM before timing starts.

Prints one JSON line.  ``value`` is history tokens per second of the whole
step; ``fwd_tokens_per_s`` is the forward alone.  ``roofline`` describes the
kernel with the largest share of the step against the roof that binds at its
algorithmic FLOPs (GEMM convention of Appendix G: 4 M d per (token, head) in the
forward, 8 M d in the backward) and algorithmic bytes: the one with the larger
ideal time, so a kernel below the ridge point is measured in bytes per second
over its live HIP-event time.  ``cpu_baseline`` times the CPU oracle on a
bounded sample of the same batch.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2609_08443_amd import workloads as wl  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
METRIC = "history tokens sketched/sec (fwd+bwd step; fwd alone in fwd_tokens_per_s), ragged 100K batch"

WORKLOADS = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}

# HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE (scaled by the
# same counters on a plain 1 GiB copy) on the default workload, keyed by the sha256 of
# the kernel's source file at the time: a changed kernel reports traffic = null.
# Source: profiles/hbm_bytes_c5_ragged100k_fwd_bwd.md
MEASURED_TRAFFIC = {
    "bwd_token": ("paper_2609_08443_amd/csrc/bwd_fused.hip",
                  "57d0367bf7b2a9a5441602519ebfd053502bcd504f2584431bfee195eb7587c3",
                  1.310e9 + 2.250e9),
    "bwd_proto": ("paper_2609_08443_amd/csrc/bwd_fused.hip",
                  "57d0367bf7b2a9a5441602519ebfd053502bcd504f2584431bfee195eb7587c3",
                  1.220e9 + 0.100e9),
    "fused_fwd": ("paper_2609_08443_amd/csrc/fwd_fused.hip",
                  "221f8a9cd9d47e29d8f3d3ad2c3d6abb3048e9c1b17f5877add84c3f71458562",
                  0.658e9 + 0.135e9),
}


def measured_traffic(kernel: str, workload: str):
    """Bytes per launch if counters were taken on this workload and kernel source."""
    import hashlib
    if workload != "c5" or kernel not in MEASURED_TRAFFIC:
        return None
    path, digest, nbytes = MEASURED_TRAFFIC[kernel]
    try:
        with open(os.path.join(ROOT, path), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    except OSError:
        return None
    return nbytes


# ---------------------------------------------------------------- accounting
def fwd_algorithmic_flops(w: wl.Workload) -> float:
    """Affinity GEMM + aggregation GEMM, 2 L_s L d each, per head (Appendix G.3)."""
    return 4.0 * w.M * w.d * float(w.T) * w.H


def bwd_algorithmic_flops(w: wl.Workload) -> float:
    """Four gradient GEMMs of the same size: dA = V dY^T, dV = A dY, dK = dS P, dP = dS^T K."""
    return 8.0 * w.M * w.d * float(w.T) * w.H


def fwd_algorithmic_bytes(w: wl.Workload) -> float:
    el = 2 if w.dtype == "bf16" else 4
    return (2.0 * w.T * w.H * w.d * el          # K, V read once
            + w.H * w.M * w.d * el              # P
            + 4.0 * w.B * w.H * w.M * w.d       # sketch written
            + 4.0 * w.T * w.H)                  # lse written


def bwd_algorithmic_bytes(w: wl.Workload) -> float:
    el = 2 if w.dtype == "bf16" else 4
    return (2.0 * w.T * w.H * w.d * el          # K, V
            + 4.0 * w.T * w.H                   # lse
            + 4.0 * w.B * w.R * w.H * w.M * w.d  # dsketch
            + 2.0 * 4.0 * w.T * w.H * w.d       # dK, dV written (fp32)
            + 4.0 * w.H * w.M * w.d)            # dP


# kernel name -> (algorithmic flops, executed matrix flops, algorithmic bytes, bound) of one
# launch.  Algorithmic = the GEMMs of the method (Appendix G convention); executed also
# counts the recomputation of S (and of dA) that the backward kernels do instead of storing.
def kernel_work(name: str, w: wl.Workload):
    th = float(w.T) * w.H
    md = float(w.M) * w.d
    el = 2 if w.dtype == "bf16" else 4
    if name == "fused_fwd":
        return 4 * md * th, 4 * md * th, fwd_algorithmic_bytes(w), "mfma"
    if name == "bwd_token":   # dA, dV, dK (+ S twice)
        return 6 * md * th, 10 * md * th, th * w.d * (2 * el + 8) + 4 * th, "mfma"
    if name == "bwd_proto":   # dP (+ S and dA)
        return 2 * md * th, 6 * md * th, th * w.d * 2 * el + 8 * th, "mfma"
    if name == "plain_fwd":
        return 4 * md * th, 0.0, fwd_algorithmic_bytes(w), "alu"
    if name == "plain_bwd":
        return 8 * md * th, 0.0, bwd_algorithmic_bytes(w), "alu"
    return None


# ---------------------------------------------------------------- CPU baseline
def cpu_baseline(w: wl.Workload, dev: dict, budget_tokens: int) -> dict:
    """The fp64 oracle (fwd, plus bwd when the step has it) on the shortest users of the
    batch whose total length reaches budget_tokens; reported in tokens/s."""
    import numpy as np
    import oracle

    order = list(np.argsort(w.lengths, kind="stable"))
    users, tot = [], 0
    for b in order:
        users.append(int(b))
        tot += int(w.lengths[b])
        if tot >= budget_tokens:
            break
    users.sort()
    off = w.offsets
    K = np.concatenate([dev["K"][off[b]:off[b + 1]].float().cpu().numpy() for b in users])
    V = np.concatenate([dev["V"][off[b]:off[b + 1]].float().cpu().numpy() for b in users])
    P = dev["P"].float().cpu().numpy()
    lens = w.lengths[users]
    o = np.zeros(len(users) + 1, np.int64)
    np.cumsum(lens, out=o[1:])
    threads = oracle.max_threads()
    t0 = time.perf_counter()
    oracle.fwd(K, V, P, o, w.scale)
    if w.bwd:
        dS = dev["dsketch"][users].cpu().numpy()
        oracle.bwd(K, V, P, o, dS, w.scale)
    dt = time.perf_counter() - t0
    ntok = int(lens.sum())
    return {"value": ntok / dt, "unit": "tokens/s", "cores": min(threads, len(users) * w.H),
            "kind": "oracle",
            "sample": f"{len(users)} shortest users ({ntok} tokens, all {w.H} heads, "
                      f"{'fwd+bwd' if w.bwd else 'fwd'}) of the same batch, fp64, {dt:.1f} s"}


# ---------------------------------------------------------------- main
def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the timings of the token-wise variant and of the SA layer")
    ap.add_argument("--cpu-tokens", type=int, default=300000,
                    help="tokens of the CPU-baseline sample (shortest users first)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of 1 GiB (to scale HBM byte counters)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the sketching step "
              "shards by user with no exchange in the forward; multi-GPU runs are not part "
              "of this build.", file=sys.stderr)
        return 2

    import torch

    from paper_2609_08443_amd import sa_sketch as sa

    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = 1 << 28  # 2^28 fp32 = 1 GiB read + 1 GiB written per copy
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "copies": 3}))
        return 0
    w = wl.config(WORKLOADS[args.workload])
    dev = wl.device_tensors(w, "cuda")
    code = sa.SA_BF16 if w.dtype == "bf16" else sa.SA_FP32
    B, T, H, M, d, R = w.B, w.T, w.H, w.M, w.d, w.R
    sketch = torch.empty((B, H, M, d), dtype=torch.float32, device="cuda")
    lse = torch.empty((T, H), dtype=torch.float32, device="cuda")
    ws_f = torch.empty(max(sa.fwd_workspace_size(B, T, H, M, d, code), 1), dtype=torch.uint8,
                       device="cuda")
    if w.bwd:
        dK = torch.empty((T, H, d), dtype=torch.float32, device="cuda")
        dV = torch.empty((T, H, d), dtype=torch.float32, device="cuda")
        dP = torch.empty((H, M, d), dtype=torch.float32, device="cuda")
        ws_b = torch.empty(max(sa.bwd_workspace_size(B, T, H, M, d, code, R), 1),
                           dtype=torch.uint8, device="cuda")

    def step():
        sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale, sketch=sketch,
                      lse=lse, workspace=ws_f)
        if w.bwd:
            sa.sketch_bwd(dev["K"], dev["V"], dev["P"], dev["offsets"], dev["dsketch"], lse,
                          w.scale, dK=dK, dV=dV, dP=dP, workspace=ws_b)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: outer events for the step, library events for each kernel
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    sa.kernel_times()  # clear
    sa.profile_enable(True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    sa.profile_enable(False)
    kt = sa.kernel_times()
    ms_step = e0.elapsed_time(e1) / args.steps

    # fwd-only rate from the per-kernel events of the forward's launches
    fwd_names = ("worklist", "fused_fwd", "splitL_merge", "plain_fwd")
    fwd_ms = sum(kt[n][1] for n in fwd_names if n in kt) / args.steps
    kernels = {n: {"launches": c, "avg_ms": tot / c} for n, (c, tot) in kt.items()}

    flops_step = fwd_algorithmic_flops(w) + (bwd_algorithmic_flops(w) if w.bwd else 0.0)
    known = {n: v for n, v in kt.items() if kernel_work(n, w) is not None}
    dom = max(known.items(), key=lambda kv: kv[1][1])[0] if known else None
    roof = None
    if dom is not None:
        fl, fl_exec, by, bound = kernel_work(dom, w)
        avg_ms = kt[dom][1] / kt[dom][0]
        if bound == "mfma" and by / (PEAK_HBM_GBS * 1e9) > fl / (PEAK_BF16_TFLOPS * 1e12):
            # the matrix-core kernel's algorithmic intensity is below the ridge
            # point: its roofline ceiling is the HBM roof
            bound = "hbm"
        if bound == "mfma":
            ach, peak, unit = fl / (avg_ms * 1e-3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
        elif bound == "hbm":
            ach, peak, unit = by / (avg_ms * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
        else:  # plain fp32 vector arithmetic: fp32 vector peak
            ach, peak, unit = fl / (avg_ms * 1e-3) / 1e12, 157.3, "TFLOP/s"
        roof = {"kernel": dom, "bound": bound, "achieved": ach, "peak": peak, "unit": unit,
                "frac": ach / peak, "traffic": measured_traffic(dom, args.workload),
                "avg_ms": avg_ms,
                "algorithmic_flops_per_launch": fl, "algorithmic_bytes_per_launch": by,
                "executed_mfma_tflops": fl_exec / (avg_ms * 1e-3) / 1e12 if fl_exec else None,
                "algorithmic_intensity_flop_per_byte": fl / by,
                "mfma_frac": fl / (avg_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}

    def timed(fn):
        """ms per call of fn over the timed steps, and the library's per-kernel times."""
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        sa.kernel_times()
        sa.profile_enable(True)
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(args.steps):
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        sa.profile_enable(False)
        return t0.elapsed_time(t1) / args.steps, sa.kernel_times()

    def kernel_dict(kd):
        return {n: {"launches": c, "avg_ms": tot / c} for n, (c, tot) in kd.items()}

    # token-wise normalised variant (the paper's comparison normalisation), timed on
    # the same batch after the step; not part of the step
    tokenwise = None
    if w.dtype == "bf16" and not args.no_variants:
        sk_tw = torch.empty((B, H, M, d), dtype=torch.float32, device="cuda")
        lse_tw = torch.empty((B, H, M), dtype=torch.float32, device="cuda")
        ws_tw = torch.empty(max(sa.tokenwise_workspace_size(B, T, H, M, d, code), 1), dtype=torch.uint8,
                            device="cuda")

        def tw():
            sa.sketch_fwd_tokenwise(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale, sketch=sk_tw,
                                    lse_m=lse_tw, workspace=ws_tw)
        tw_ms, ktw = timed(tw)
        del sk_tw, lse_tw, ws_tw
        main_ms = ktw["tokenwise_fwd"][1] / ktw["tokenwise_fwd"][0] if "tokenwise_fwd" in ktw else None
        tokenwise = {"tokens_per_s": T / (tw_ms * 1e-3), "ms": tw_ms, "kernels": kernel_dict(ktw),
                     "mfma_util": fwd_algorithmic_flops(w) / (tw_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                     "kernel_mfma_frac": (fwd_algorithmic_flops(w) / (main_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
                                          if main_ms else None)}

    # SA layer with its projections (K = X W_K, Q = P W_Q, X aggregated) on the same
    # batch, X = the V tensor: fwd (+ bwd) per step; not part of the step
    layer = None
    if not args.no_variants:
        proj = wl.device_projections(w, "cuda")
        X = dev["V"]
        ws_lf = torch.empty(max(sa.layer_fwd_workspace_size(B, T, H, M, d, code), 1), dtype=torch.uint8,
                            device="cuda")
        if w.bwd:
            ws_lb = torch.empty(max(sa.layer_bwd_workspace_size(B, T, H, M, d, code, R), 1),
                                dtype=torch.uint8, device="cuda")

        def lay():
            sa.layer_fwd(X, dev["P"], proj["Wq"], proj["Wk"], dev["offsets"], w.scale, sketch=sketch,
                         lse=lse, workspace=ws_lf)
            if w.bwd:
                sa.layer_bwd(X, dev["P"], proj["Wq"], proj["Wk"], dev["offsets"], dev["dsketch"], lse,
                             w.scale, workspace=ws_lb)
        ly_ms, kly = timed(lay)
        layer = {"tokens_per_s": T / (ly_ms * 1e-3), "ms": ly_ms, "kernels": kernel_dict(kly),
                 "step": "sa_layer_fwd + sa_layer_bwd" if w.bwd else "sa_layer_fwd",
                 "mfma_util": flops_step / (ly_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}

    # stacked SA (N_sa = 2 layers, the paper's deployed depth) on the same batch,
    # X = the V tensor: the forward alone, then a training step (forward keeping
    # its intermediates + backward); not part of the step
    block = None
    if not args.no_variants:
        n_layers = 2
        bp = wl.device_block_params(w, n_layers, "cuda")
        ws_bl = torch.empty(max(sa.block_fwd_workspace_size(B, T, H, M, d, n_layers, code), 1),
                            dtype=torch.uint8, device="cuda")
        out_bl = torch.empty((B, H, M, d), dtype=torch.float32, device="cuda")

        def blk():
            sa.block_fwd(dev["V"], dev["P"], bp["Wq"], bp["Wk"], bp["ln"], bp["W1"], bp["W3"], bp["W2"],
                         dev["offsets"], w.scale, out=out_bl, workspace=ws_bl)
        bl_ms, kbl = timed(blk)
        block = {"tokens_per_s": T / (bl_ms * 1e-3), "ms": bl_ms, "n_layers": n_layers,
                 "kernels": kernel_dict(kbl), "step": "sa_block_fwd"}
        if w.bwd:
            del ws_bl
            # training: the forward keeps its intermediates in `saved`, the
            # backward reads them instead of replaying the forward
            ws_bb = torch.empty(max(sa.block_bwd_workspace_size(B, T, H, M, d, n_layers, code, True),
                                    sa.block_fwd_workspace_size(B, T, H, M, d, n_layers, code), 1),
                                dtype=torch.uint8, device="cuda")
            saved = sa.block_saved_buffer(dev["V"], dev["P"], bp["Wq"], dev["offsets"])
            dout = dev["dsketch"][:, 0].contiguous()

            def blk_train():
                sa.block_fwd(dev["V"], dev["P"], bp["Wq"], bp["Wk"], bp["ln"], bp["W1"], bp["W3"], bp["W2"],
                             dev["offsets"], w.scale, out=out_bl, saved=saved, workspace=ws_bb)
                sa.block_bwd(dev["V"], dev["P"], bp["Wq"], bp["Wk"], bp["ln"], bp["W1"], bp["W3"], bp["W2"],
                             dev["offsets"], dout, w.scale, saved=saved, workspace=ws_bb)
            bt_ms, kbt = timed(blk_train)
            block["train_step"] = {"tokens_per_s": T / (bt_ms * 1e-3), "ms": bt_ms, "kernels": kernel_dict(kbt),
                                   "step": "sa_block_fwd (saved) + sa_block_bwd",
                                   "workspace_bytes": ws_bb.numel(), "saved_bytes": saved.numel()}
            del ws_bb, saved

    # reordered single-query STCA over the sketch (the sketch's consumer): the
    # batch's users, R = 40 targets each (the training-side MRLB group), k = M
    # sketch rows adapted to D = 1024 with h = 16 heads of 64; not part of the step
    stca = None
    if w.dtype == "bf16" and not args.no_variants:
        Rs, Ds, hs = 40, 1024, 16
        st = wl.device_stca(w.seed, B, Rs, M, Ds, "bf16")
        sargs = [st[n] for n in ("Xs", "q", "Wq", "Wk", "Wv")]
        ws_sf = torch.empty(sa.stca_fwd_workspace_size(B, Rs, M, Ds, hs, code), dtype=torch.uint8, device="cuda")
        ws_sb = torch.empty(sa.stca_bwd_workspace_size(B, Rs, M, Ds, hs, code), dtype=torch.uint8, device="cuda")
        out_s = torch.empty((B, Rs, Ds), dtype=torch.float32, device="cuda")

        def stf():
            sa.stca_fwd(*sargs, h=hs, out=out_s, workspace=ws_sf)

        def stfb():
            sa.stca_fwd(*sargs, h=hs, out=out_s, workspace=ws_sf)
            sa.stca_bwd(*sargs, h=hs, dout=st["dout"], workspace=ws_sb)
        sf_ms, ksf = timed(stf)
        sb_ms, ksb = timed(stfb)
        # Appendix G.2: 4 k D h + 6 D^2 per target and layer (forward); the backward
        # has two products per forward product
        fl_f = float(B) * Rs * (4.0 * M * Ds * hs + 6.0 * Ds * Ds)
        stca = {"config": {"B": B, "R": Rs, "k": M, "D": Ds, "h": hs},
                "fwd_ms": sf_ms, "fwd_bwd_ms": sb_ms,
                "targets_per_s_fwd": B * Rs / (sf_ms * 1e-3), "targets_per_s_fwd_bwd": B * Rs / (sb_ms * 1e-3),
                "fwd_tflops": fl_f / (sf_ms * 1e-3) / 1e12,
                "fwd_bwd_tflops": 3 * fl_f / (sb_ms * 1e-3) / 1e12,
                "fwd_mfma_util": fl_f / (sf_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                "fwd_bwd_mfma_util": 3 * fl_f / (sb_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                "kernels_fwd": kernel_dict(ksf), "kernels_fwd_bwd": kernel_dict(ksb)}
        del st, sargs, ws_sf, ws_sb, out_s

    out = {
        "metric": METRIC,
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) K/V/dSketch, N(0,1/d) P; paper-shaped lengths)",
        "config": {"workload": w.name, "B": B, "T": T, "H": H, "M": M, "d": d, "R": R,
                   "step": "sa_sketch_fwd + sa_sketch_bwd" if w.bwd else "sa_sketch_fwd"},
        "fwd_tokens_per_s": T / (fwd_ms * 1e-3) if fwd_ms > 0 else None,
        "token_heads_per_s": T * H / (ms_step * 1e-3),
        "mfma_util_step": flops_step / (ms_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "mfma_util_fwd": (fwd_algorithmic_flops(w) / (fwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
                          if fwd_ms > 0 else None),
        "wall_s_timed": wall,
        "kernels": kernels,
        "roofline": roof,
        "tokenwise_fwd": tokenwise,
        "layer": layer,
        "block_fwd": block,
        "stca": stca,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, dev, args.cpu_tokens)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

"""Benchmark of the SA sketching step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c5] [--no-cpu-baseline]
                    [--no-configs] [--no-variants]

A step is one pass of the whole hot path over one batch: sa_sketch_fwd
(work list, fused forward, split-L merge) then sa_sketch_bwd (MRLB target sum,
backward kernels).  The default workload is the ragged 100K batch trained with
4 target instances per user (32 users, log-uniform lengths in [1e3, 1e5],
H = 4, d = 128, M = 512, bf16, R = 4).  Inputs are synthetic, drawn on the
device with fixed seeds, resident in HBM before timing starts.

Prints one JSON line.  ``value`` is history tokens per second of the whole
step, timed over K steps with nothing but the library's launches inside the
timed region; ``fwd_tokens_per_s`` times the forward alone the same way.  The
per-kernel figures come from a separate pass of K steps with the library's
per-launch HIP events switched on.  ``roofline`` describes the kernel with the
largest share of the step against the roof that binds at its algorithmic FLOPs
(GEMM convention of Appendix G: 4 M d per (token, head) in the forward, 8 M d
in the backward) and algorithmic bytes: the one with the larger ideal time, so
a kernel below the ridge point is measured in bytes per second over its live
HIP-event time; ``kernel_roofline`` does the same for every kernel of the
step.  ``configs`` times the forward of the other paper-shaped batches (the
single-user fp32 case, the uniform 16 x 10K batch with its inputs rotated
through copies larger than the 256 MB Infinity Cache, and the 64 x 100K
batch).  ``cpu_baseline`` times the CPU oracle on a bounded sample of the
same batch.
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

# HBM bytes per launch of the step's kernels on the default workload, from
# rocprofv3's request counters (128 RDREQ_128B + 64 RDREQ_64B + 32 RDREQ_32B read,
# 64 WRREQ_64B + 32 (WRREQ - WRREQ_64B) written; exact on a plain 1 GiB copy),
# taken with --no-configs --no-variants so that only the step's launches are
# averaged, keyed by the sha256 of the kernel's source file at the time: a
# changed kernel reports traffic = null.
# Source: profiles/hbm_bytes_c5_ragged100k_fwd_bwd.md
MEASURED_TRAFFIC = {
    "fused_fwd": ("paper_2609_08443_amd/csrc/fwd_fused.hip",
                  "d95d57d9a73986256ac7444c7b95b5d25f6e592308de1aca4d0b37338b5712e8",
                  1.115e9 + 0.145e9),
    "bwd_token": ("paper_2609_08443_amd/csrc/bwd_fused.hip",
                  "04c2f979ec2709a93a48939f23c469eddc2e712161f692aa703e9002acbfd291",
                  1.362e9 + 2.250e9),
    "bwd_proto": ("paper_2609_08443_amd/csrc/bwd_fused.hip",
                  "04c2f979ec2709a93a48939f23c469eddc2e712161f692aa703e9002acbfd291",
                  1.220e9 + 0.100e9),
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
# counts the recomputation of S (and of dA) that the backward kernels do instead of storing:
# the token side computes S once when its first sweep's weights fit in registers (M <= 512).
def kernel_work(name: str, w: wl.Workload):
    th = float(w.T) * w.H
    md = float(w.M) * w.d
    el = 2 if w.dtype == "bf16" else 4
    if name == "fused_fwd":
        return 4 * md * th, 4 * md * th, fwd_algorithmic_bytes(w), "mfma"
    if name == "bwd_token":   # dA, dV, dK (+ S; for M > 512 S again in the second sweep)
        return 6 * md * th, (8 if w.M <= 512 else 10) * md * th, th * w.d * (2 * el + 8) + 4 * th, "mfma"
    if name == "bwd_proto":   # dP (+ S and dA)
        return 2 * md * th, 6 * md * th, th * w.d * 2 * el + 8 * th, "mfma"
    if name == "plain_fwd":
        return 4 * md * th, 0.0, fwd_algorithmic_bytes(w), "alu"
    if name == "plain_bwd":
        return 8 * md * th, 0.0, bwd_algorithmic_bytes(w), "alu"
    return None


# ---------------------------------------------------------------- CPU baseline
def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w: wl.Workload, dev: dict, budget_tokens: int) -> dict:
    """The fp64 oracle (fwd, plus bwd when the step has it) on the shortest users of the
    batch whose total length reaches budget_tokens, on every host thread; then on one
    thread over the first 2000 tokens of the shortest user.  Reported in tokens/s."""
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
    dS = dev["dsketch"][users].cpu().numpy() if w.bwd else None

    def run(K_, V_, o_, dS_, nthreads):
        t0 = time.perf_counter()
        oracle.fwd(K_, V_, P, o_, w.scale, nthreads=nthreads)
        if w.bwd:
            oracle.bwd(K_, V_, P, o_, dS_, w.scale, nthreads=nthreads)
        return time.perf_counter() - t0

    dt = run(K, V, o, dS, 0)
    ntok = int(lens.sum())
    # one thread: the first n1 tokens of the shortest user (its upstream gradient as is)
    b0 = int(order[0])
    n1 = int(min(2000, w.lengths[b0]))
    s0 = int(off[b0])
    K1 = dev["K"][s0:s0 + n1].float().cpu().numpy()
    V1 = dev["V"][s0:s0 + n1].float().cpu().numpy()
    dS1 = dev["dsketch"][b0:b0 + 1].cpu().numpy() if w.bwd else None
    dt1 = run(K1, V1, np.array([0, n1], np.int64), dS1, 1)
    kind = "fwd+bwd" if w.bwd else "fwd"
    return {"value": ntok / dt, "unit": "tokens/s", "cores": min(threads, len(users) * w.H),
            "kind": "oracle",
            "sample": f"{len(users)} shortest users ({ntok} tokens, all {w.H} heads, {kind}) of the "
                      f"same batch, fp64, {dt:.1f} s",
            "cpu_model": cpu_model(), "host_threads": threads,
            "single_thread": {"value": n1 / dt1, "unit": "tokens/s",
                              "sample": f"first {n1} tokens of user {b0} (all {w.H} heads, {kind}), "
                                        f"fp64, one thread, {dt1:.1f} s"}}


# ---------------------------------------------------------------- main
def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the timings of the token-wise variant, the SA layer, the block and STCA")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the forward timings of the other paper-shaped batches")
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

    stream = torch.cuda.current_stream()

    def plain_loop(fn, reps):
        """ms per call of fn over reps calls: two stream events around the calls,
        nothing else inside the timed region."""
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / reps

    # headline: the step alone, no per-launch events
    wall0 = time.perf_counter()
    ms_step = plain_loop(step, args.steps)
    wall = time.perf_counter() - wall0

    # the forward alone, timed the same way
    def fwd_only():
        sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale, sketch=sketch, lse=lse,
                      workspace=ws_f)
    for _ in range(args.warmup):
        fwd_only()
    fwd_ms = plain_loop(fwd_only, args.steps)

    # per-kernel times: a separate pass of the same steps with the library's
    # per-launch events on the launch stream
    sa.kernel_times()  # clear
    sa.profile_enable(True)
    plain_loop(step, args.steps)
    sa.profile_enable(False)
    kt = sa.kernel_times()
    kernels = {n: {"launches": c, "avg_ms": tot / c} for n, (c, tot) in kt.items()}

    flops_step = fwd_algorithmic_flops(w) + (bwd_algorithmic_flops(w) if w.bwd else 0.0)

    def kernel_roof(name, wk, avg_ms, workload_key):
        fl, fl_exec, by, bound = kernel_work(name, wk)
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
        return {"kernel": name, "bound": bound, "achieved": ach, "peak": peak, "unit": unit,
                "frac": ach / peak, "traffic": measured_traffic(name, workload_key),
                "avg_ms": avg_ms,
                "algorithmic_flops_per_launch": fl, "algorithmic_bytes_per_launch": by,
                "executed_mfma_tflops": fl_exec / (avg_ms * 1e-3) / 1e12 if fl_exec else None,
                "algorithmic_intensity_flop_per_byte": fl / by,
                "mfma_frac": fl / (avg_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}

    known = {n: v for n, v in kt.items() if kernel_work(n, w) is not None}
    kernel_roofline = {n: kernel_roof(n, w, tot / c, args.workload) for n, (c, tot) in known.items()}
    dom = max(known.items(), key=lambda kv: kv[1][1])[0] if known else None
    roof = kernel_roofline[dom] if dom is not None else None

    # the forward of the other paper-shaped batches: the 2048-token fp32 case
    # (time only), the 16 x 10K batch with its K and V rotated through copies that
    # together exceed the 256 MB Infinity Cache (so every call reads HBM), and the
    # 64 x 100K batch
    configs = None
    if not args.no_configs and args.workload == "c5":
        configs = {}
        for key in ("c1", "c2", "c4"):
            wc = wl.config(WORKLOADS[key])
            dc = wl.device_tensors(wc, "cuda")
            cc = sa.SA_BF16 if wc.dtype == "bf16" else sa.SA_FP32
            skc = torch.empty((wc.B, wc.H, wc.M, wc.d), dtype=torch.float32, device="cuda")
            lsc = torch.empty((wc.T, wc.H), dtype=torch.float32, device="cuda")
            wsc = torch.empty(max(sa.fwd_workspace_size(wc.B, wc.T, wc.H, wc.M, wc.d, cc), 1),
                              dtype=torch.uint8, device="cuda")
            kv_bytes = 2 * dc["K"].numel() * dc["K"].element_size()
            n_copies = int(math.ceil(512e6 / kv_bytes)) + 1 if key == "c2" else 1
            copies = [(dc["K"], dc["V"])] + [(dc["K"].clone(), dc["V"].clone()) for _ in range(n_copies - 1)]
            it = [0]

            def fc():
                Kc, Vc = copies[it[0] % n_copies]
                it[0] += 1
                sa.sketch_fwd(Kc, Vc, dc["P"], dc["offsets"], wc.scale, sketch=skc, lse=lsc, workspace=wsc)
            reps = 5 if key == "c4" else args.steps
            for _ in range(max(args.warmup, n_copies)):
                fc()
            ms = plain_loop(fc, reps)
            sa.kernel_times()
            sa.profile_enable(True)
            plain_loop(fc, reps)
            sa.profile_enable(False)
            kc = sa.kernel_times()
            main_k = "fused_fwd" if "fused_fwd" in kc else "plain_fwd"
            entry = {"workload": wc.name, "T": wc.T, "ms": ms, "tokens_per_s": wc.T / (ms * 1e-3),
                     "reps": reps,
                     "kernels": {n: {"launches": c, "avg_ms": tot / c} for n, (c, tot) in kc.items()}}
            if key == "c2":
                entry["input_copies"] = n_copies
                entry["input_copy_bytes"] = kv_bytes
            if key != "c1" and main_k in kc:
                entry["roofline"] = kernel_roof(main_k, wc, kc[main_k][1] / kc[main_k][0], key)
                entry["mfma_util"] = fwd_algorithmic_flops(wc) / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
            configs[key] = entry
            del dc, copies, skc, lsc, wsc
            torch.cuda.empty_cache()

    def timed(fn):
        """ms per call of fn over the timed steps (no per-launch events), and the
        library's per-kernel times from a second pass."""
        for _ in range(args.warmup):
            fn()
        ms = plain_loop(fn, args.steps)
        sa.kernel_times()
        sa.profile_enable(True)
        plain_loop(fn, args.steps)
        sa.profile_enable(False)
        return ms, sa.kernel_times()

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
        "kernels_note": "per-launch HIP events, from a separate pass of the same steps",
        "roofline": roof,
        "kernel_roofline": kernel_roofline,
        "configs": configs,
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

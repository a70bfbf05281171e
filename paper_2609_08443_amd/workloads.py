"""Seeded synthetic workloads for the Sketch Attention (SA) sketching step.

This module only draws inputs: it holds none of the method's arithmetic.  It is
the one piece shared by the CPU oracle (``oracle/``), the GPU tests and the
benchmark, so both sides of every parity check see the same bytes.

The paper's workloads are proprietary user histories (Douyin); what stands in
for them here are tensors with the paper's shapes: histories of up to 100K
tokens (section 2.1, n_max), a 10K recent suffix (section 2.2, L_r), k = 512 to
2K prototypes and d = 64 or 128 (Table 2 ablations, Appendix G.4), ragged
across users.  Values: K, V ~ N(0, 1), prototypes P ~ N(0, 1/d), upstream
gradients dSketch ~ N(0, 1); bf16 tensors are drawn in fp32 and rounded to
nearest-even.

Two generators with the same distributions:

* ``host_tensors``  -- numpy PCG64, one stream per (seed, tensor, user), so any
  single user can be regenerated alone.  Exact and platform independent; used
  for every size the CPU can draw in seconds.
* ``device_tensors`` -- torch's on-device Philox generator, one seed per
  (seed, tensor, user).  Used for the multi-GB full-size batches; sampled users
  are copied back to the host for the oracle.

Tensor layouts (token-major, packed, no padding):
  K, V     [T, H, d]     T = sum of the user lengths
  P        [H, M, d]     shared by all users
  offsets  [B + 1] int64 CSR offsets, offsets[0] = 0, offsets[B] = T
  dsketch  [B, R, H, M, d] fp32

For the SA layer with its projections the history X is the V stream and the
projections W_Q, W_K [H, d, d] ~ N(0, 1/d), so that K = X W_K and Q = P W_Q have
the statistics of the K and P above.

For the STCA over the sketch (``host_stca`` / ``device_stca``): adapted sketches
Xs [B, k, D] ~ N(0, 1), target queries q [B, R, D] ~ N(0, 1), W_Q, W_K, W_V
[D, D] ~ N(0, 1/D) (so that each head's logits have unit scale at
scale = 1/sqrt(D/h)) and upstream gradients dout [B, R, D] ~ N(0, 1).
"""

from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional, Sequence

import numpy as np

# tensor ids of the per-(seed, tensor, user) streams
TID_LENGTHS, TID_K, TID_V, TID_P, TID_DSKETCH = 0, 1, 2, 3, 4
TID_WQ, TID_WK = 5, 6
TID_BLOCK = 7   # stacked-block parameters: 7 + kind
TID_STCA = 100  # STCA over the sketch: 100 + kind

BASE_SEED = 8443


@dataclasses.dataclass
class Workload:
    """Shape and seed of one synthetic batch."""

    name: str
    lengths: np.ndarray  # int64 [B]
    H: int
    M: int
    d: int
    dtype: str  # "bf16" or "fp32"
    seed: int
    R: int = 1  # target instances that reuse each user's sketch (backward input)
    bwd: bool = False

    @property
    def B(self) -> int:
        return int(self.lengths.shape[0])

    @property
    def T(self) -> int:
        return int(self.lengths.sum())

    @property
    def offsets(self) -> np.ndarray:
        off = np.zeros(self.B + 1, dtype=np.int64)
        np.cumsum(self.lengths, out=off[1:])
        return off

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "B": self.B,
            "T": self.T,
            "H": self.H,
            "M": self.M,
            "d": self.d,
            "dtype": self.dtype,
            "R": self.R,
            "bwd": self.bwd,
            "seed": self.seed,
            "L_min": int(self.lengths.min()) if self.B else 0,
            "L_max": int(self.lengths.max()) if self.B else 0,
        }


def loguniform_lengths(seed: int, B: int, lo: int, hi: int) -> np.ndarray:
    """L_b = clamp(rint(exp(U(ln lo, ln hi))), lo, hi), one seeded stream."""
    rng = np.random.default_rng([seed, TID_LENGTHS, 0])
    u = rng.uniform(math.log(lo), math.log(hi), size=B)
    return np.clip(np.rint(np.exp(u)), lo, hi).astype(np.int64)


def config(cfg: int) -> Workload:
    """The five paper-shaped configurations (1-based ids)."""
    seed = BASE_SEED + cfg
    if cfg == 1:
        return Workload("single_user_L2048_H1_d64_M64_fp32",
                        np.full(1, 2048, np.int64), 1, 64, 64, "fp32", seed)
    if cfg == 2:
        return Workload("uniform_16x10k_H4_d64_M256_bf16",
                        np.full(16, 10_000, np.int64), 4, 256, 64, "bf16", seed)
    if cfg == 3:
        return Workload("ragged_32x[1k,100k]_H4_d128_M512_bf16",
                        loguniform_lengths(seed, 32, 1_000, 100_000), 4, 512, 128,
                        "bf16", seed)
    if cfg == 4:
        return Workload("full_64x100k_H8_d64_M1024_bf16",
                        np.full(64, 100_000, np.int64), 8, 1024, 64, "bf16", seed)
    if cfg == 5:
        w = config(3)
        # same ragged batch as config 3 (same lengths and token values), plus bwd
        return Workload("ragged_32x[1k,100k]_H4_d128_M512_bf16_fwd+bwd_R4",
                        w.lengths, 4, 512, 128, "bf16", w.seed, R=4, bwd=True)
    raise ValueError(f"unknown config {cfg}")


def custom(lengths: Sequence[int], H: int, M: int, d: int, dtype: str = "bf16",
           seed: int = 1234, R: int = 1, bwd: bool = False,
           name: Optional[str] = None) -> Workload:
    lengths = np.asarray(lengths, dtype=np.int64)
    if name is None:
        name = f"custom_B{len(lengths)}_H{H}_M{M}_d{d}_{dtype}_s{seed}"
    return Workload(name, lengths, H, M, d, dtype, seed, R=R, bwd=bwd)


# --------------------------------------------------------------------------
# bf16 bit helpers (storage format only)
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact upcast of bf16 bits to fp32."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# host (numpy) generator
# --------------------------------------------------------------------------

def _normal(seed: int, tid: int, b: int, shape, std: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng([seed, tid, b])
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def _finish(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp32 stays fp32; bf16 is returned as the fp32 value of the rounded bf16."""
    if dtype == "fp32":
        return x
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


def host_user(w: Workload, b: int) -> dict:
    """K, V of user b (fp32 arrays holding exact bf16 values in bf16 mode)."""
    L = int(w.lengths[b])
    K = _finish(_normal(w.seed, TID_K, b, (L, w.H, w.d)), w.dtype)
    V = _finish(_normal(w.seed, TID_V, b, (L, w.H, w.d)), w.dtype)
    return {"K": K, "V": V}


def host_prototypes(w: Workload) -> np.ndarray:
    return _finish(_normal(w.seed, TID_P, 0, (w.H, w.M, w.d), 1.0 / math.sqrt(w.d)),
                   w.dtype)


def host_projections(w: Workload) -> dict:
    """W_Q, W_K [H, d, d] of the SA layer (exact bf16 values in bf16 mode)."""
    sd = 1.0 / math.sqrt(w.d)
    return {"Wq": _finish(_normal(w.seed, TID_WQ, 0, (w.H, w.d, w.d), sd), w.dtype),
            "Wk": _finish(_normal(w.seed, TID_WK, 0, (w.H, w.d, w.d), sd), w.dtype)}


def device_projections(w: Workload, device="cuda") -> dict:
    """W_Q, W_K on the device (torch Philox, as device_tensors)."""
    import torch

    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    g = torch.Generator(device=device)
    out = {}
    for name, tid in (("Wq", TID_WQ), ("Wk", TID_WK)):
        g.manual_seed(_torch_seed(w.seed, tid, 0))
        out[name] = (torch.randn((w.H, w.d, w.d), generator=g, device=device, dtype=torch.float32)
                     / math.sqrt(w.d)).to(tdt)
    return out


def _block_shapes(w: Workload, L: int):
    d = w.d
    return {"Wq": ((L, w.H, d, d), 1.0 / math.sqrt(d)), "Wk": ((L, w.H, d, d), 1.0 / math.sqrt(d)),
            "W1": ((L, w.H, d, 2 * d), 1.0 / math.sqrt(d)), "W3": ((L, w.H, d, 2 * d), 1.0 / math.sqrt(d)),
            "W2": ((L, w.H, 2 * d, d), 1.0 / math.sqrt(2 * d)), "ln": ((L, 4, w.H, d), 0.1)}


def _ln_from_noise(x: np.ndarray) -> np.ndarray:
    """Gains 1 + noise (slots 0, 2), biases = noise (slots 1, 3)."""
    x = x.copy()
    x[:, 0] += 1.0
    x[:, 2] += 1.0
    return x


def host_block_params(w: Workload, L: int) -> dict:
    """Stacked-block parameters for L layers (exact bf16 values in bf16 mode):
    projections ~ N(0, 1/fan_in), norm gains 1 + N(0, 0.01), biases N(0, 0.01)."""
    out = {}
    for k, (name, (shape, sd)) in enumerate(_block_shapes(w, L).items()):
        x = _normal(w.seed, TID_BLOCK + k, 0, shape, sd)
        if name == "ln":
            x = _ln_from_noise(x)
        out[name] = _finish(x, w.dtype)
    return out


def device_block_params(w: Workload, L: int, device="cuda") -> dict:
    """host_block_params' distributions, drawn on the device (torch Philox)."""
    import torch

    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    g = torch.Generator(device=device)
    out = {}
    for k, (name, (shape, sd)) in enumerate(_block_shapes(w, L).items()):
        g.manual_seed(_torch_seed(w.seed, TID_BLOCK + k, 0))
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * sd
        if name == "ln":
            x[:, 0] += 1.0
            x[:, 2] += 1.0
        out[name] = x.to(tdt)
    return out


_STCA_KINDS = ("Xs", "q", "Wq", "Wk", "Wv", "dout")


def _stca_shapes(B: int, R: int, k: int, D: int):
    sd = 1.0 / math.sqrt(D)
    return {"Xs": ((B, k, D), 1.0), "q": ((B, R, D), 1.0), "Wq": ((D, D), sd), "Wk": ((D, D), sd),
            "Wv": ((D, D), sd), "dout": ((B, R, D), 1.0)}


def host_stca(seed: int, B: int, R: int, k: int, D: int, dtype: str = "bf16") -> dict:
    """STCA inputs on the host (exact bf16 values in bf16 mode; dout stays fp32)."""
    out = {}
    for i, (name, (shape, sd)) in enumerate(_stca_shapes(B, R, k, D).items()):
        x = _normal(seed, TID_STCA + i, 0, shape, sd)
        out[name] = x if name == "dout" else _finish(x, dtype)
    return out


def device_stca(seed: int, B: int, R: int, k: int, D: int, dtype: str = "bf16", device="cuda") -> dict:
    """host_stca's distributions drawn on the device (torch Philox)."""
    import torch

    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device=device)
    out = {}
    for i, (name, (shape, sd)) in enumerate(_stca_shapes(B, R, k, D).items()):
        g.manual_seed(_torch_seed(seed, TID_STCA + i, 0))
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * sd
        out[name] = x if name == "dout" else x.to(tdt)
    return out


def host_dsketch_user(w: Workload, b: int) -> np.ndarray:
    return _normal(w.seed, TID_DSKETCH, b, (w.R, w.H, w.M, w.d))


def host_tensors(w: Workload, users: Optional[Sequence[int]] = None) -> dict:
    """Whole batch (or the listed users, packed in that order) on the host.

    Returns fp32 arrays; in bf16 mode every value is exactly representable in
    bf16 and ``to_bf16_bits`` gives the storage bits.
    """
    if users is None:
        users = range(w.B)
    users = list(users)
    Ks, Vs, dS = [], [], []
    for b in users:
        u = host_user(w, b)
        Ks.append(u["K"])
        Vs.append(u["V"])
        if w.bwd:
            dS.append(host_dsketch_user(w, b))
    lengths = w.lengths[users] if len(users) else np.zeros(0, np.int64)
    off = np.zeros(len(users) + 1, np.int64)
    np.cumsum(lengths, out=off[1:])
    empty = np.zeros((0, w.H, w.d), np.float32)
    out = {
        "K": np.concatenate(Ks) if Ks else empty,
        "V": np.concatenate(Vs) if Vs else empty.copy(),
        "P": host_prototypes(w),
        "offsets": off,
    }
    if w.bwd:
        out["dsketch"] = (np.stack(dS) if dS else
                          np.zeros((0, w.R, w.H, w.M, w.d), np.float32))
    return out


# --------------------------------------------------------------------------
# device (torch Philox) generator, for the multi-GB batches
# --------------------------------------------------------------------------

def _torch_seed(seed: int, tid: int, b: int) -> int:
    h = hashlib.sha256(f"sa-sketch:{seed}:{tid}:{b}".encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def device_tensors(w: Workload, device="cuda", with_dsketch: Optional[bool] = None) -> dict:
    """Whole batch generated on the device (torch tensors).

    bf16 mode: K, V, P are torch.bfloat16 (fp32 draws rounded to nearest-even);
    fp32 mode: torch.float32.  offsets is int64 on the device.
    """
    import torch

    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    T = w.T
    K = torch.empty((T, w.H, w.d), dtype=tdt, device=device)
    V = torch.empty((T, w.H, w.d), dtype=tdt, device=device)
    off = w.offsets
    g = torch.Generator(device=device)
    for b in range(w.B):
        s, e = int(off[b]), int(off[b + 1])
        if e == s:
            continue
        g.manual_seed(_torch_seed(w.seed, TID_K, b))
        K[s:e] = torch.randn((e - s, w.H, w.d), generator=g, device=device,
                             dtype=torch.float32).to(tdt)
        g.manual_seed(_torch_seed(w.seed, TID_V, b))
        V[s:e] = torch.randn((e - s, w.H, w.d), generator=g, device=device,
                             dtype=torch.float32).to(tdt)
    g.manual_seed(_torch_seed(w.seed, TID_P, 0))
    P = (torch.randn((w.H, w.M, w.d), generator=g, device=device, dtype=torch.float32)
         / math.sqrt(w.d)).to(tdt)
    out = {"K": K, "V": V, "P": P,
           "offsets": torch.from_numpy(off).to(device)}
    if with_dsketch is None:
        with_dsketch = w.bwd
    if with_dsketch:
        dS = torch.empty((w.B, w.R, w.H, w.M, w.d), dtype=torch.float32, device=device)
        for b in range(w.B):
            g.manual_seed(_torch_seed(w.seed, TID_DSKETCH, b))
            dS[b] = torch.randn((w.R, w.H, w.M, w.d), generator=g, device=device,
                                dtype=torch.float32)
        out["dsketch"] = dS
    return out


def to_device(host: dict, dtype: str, device="cuda") -> dict:
    """Upload ``host_tensors`` output; bf16 tensors keep their exact bits."""
    import torch

    out = {}
    for k, v in host.items():
        if k in ("K", "V", "X", "P", "Wq", "Wk", "Wv", "W1", "W2", "W3", "ln", "Xs", "q") and dtype == "bf16":
            bits = f32_to_bf16_bits(v).view(np.int16)
            out[k] = torch.from_numpy(bits.copy()).to(device).view(torch.bfloat16)
        else:
            out[k] = torch.from_numpy(np.ascontiguousarray(v)).to(device)
    return out

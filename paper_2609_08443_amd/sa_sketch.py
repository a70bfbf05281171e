"""Python binding of the SA sketching library (include/sa_sketch.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of libsa_sketch.so.  torch provides device memory and the stream.
There is no fallback: if the library is missing, or a call fails, an
``SAError`` is raised.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsa_sketch.so")

SA_BF16, SA_FP32 = 0, 1
_STATUS = {0: "SA_OK", 1: "SA_ERR_INVALID_ARG", 2: "SA_ERR_UNSUPPORTED", 3: "SA_ERR_WORKSPACE",
           4: "SA_ERR_BAD_OFFSETS", 5: "SA_ERR_HIP"}
ITEM_WORDS = 8

EXPORTS = ("sa_sketch_fwd_workspace_size", "sa_sketch_fwd", "sa_sketch_fwd_noalloc", "sa_sketch_bwd_workspace_size",
           "sa_sketch_bwd", "sa_build_worklist", "sa_sketch_fwd_chunk_tokens",
           "sa_sketch_fwd_tokenwise_workspace_size", "sa_sketch_fwd_tokenwise",
           "sa_layer_fwd_workspace_size", "sa_layer_fwd", "sa_layer_bwd_workspace_size",
           "sa_layer_bwd", "sa_block_fwd_workspace_size", "sa_block_fwd",
           "sa_block_saved_size", "sa_block_saved_offset", "sa_block_bwd_workspace_size", "sa_block_bwd",
           "sa_stca_fwd_workspace_size", "sa_stca_fwd",
           "sa_stca_bwd_workspace_size", "sa_stca_bwd", "sa_gemm_tile_shapes", "sa_gemm_bf16",
           "sa_profile_enable", "sa_kernel_times", "sa_status_string", "sa_last_error")


class SAError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.status_name = _STATUS.get(status, str(status))
        super().__init__(f"{self.status_name}: {detail}")


_lib = None


def lib() -> ctypes.CDLL:
    """Load the in-tree library (built by ``paper_2609_08443_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise SAError(-1, f"{LIB_PATH} is missing; run python -m paper_2609_08443_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    c = ctypes
    i64, i32, sz, vp, f32 = c.c_int64, c.c_int32, c.c_size_t, c.c_void_p, c.c_float
    L.sa_sketch_fwd_workspace_size.argtypes = [i64, i64, i32, i32, i32, c.c_int]
    L.sa_sketch_fwd_workspace_size.restype = sz
    L.sa_sketch_bwd_workspace_size.argtypes = [i64, i64, i32, i32, i32, c.c_int, i32]
    L.sa_sketch_bwd_workspace_size.restype = sz
    L.sa_sketch_fwd_chunk_tokens.argtypes = [i64, i64, i32, i32, i32, c.c_int]
    L.sa_sketch_fwd_chunk_tokens.restype = i64
    L.sa_sketch_fwd.argtypes = [vp, vp, vp, vp, i64, i64, i32, i32, i32, f32, c.c_int, vp, vp,
                                vp, sz, vp]
    L.sa_sketch_fwd.restype = c.c_int
    L.sa_sketch_bwd.argtypes = [vp, vp, vp, vp, i64, i64, i32, i32, i32, f32, c.c_int, vp, i32,
                                vp, vp, vp, vp, vp, sz, vp]
    L.sa_sketch_bwd.restype = c.c_int
    L.sa_gemm_tile_shapes.argtypes = []
    L.sa_gemm_tile_shapes.restype = i32
    L.sa_gemm_bf16.argtypes = [vp, i64, i64, i64, vp, i64, i64, i64, i64, vp, i32, i64, i64, i32, i32, i32, i32,
                               f32, i32, i32, vp]
    L.sa_gemm_bf16.restype = c.c_int
    L.sa_sketch_fwd_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i32, i32, i32, f32, c.c_int, vp, vp, vp]
    L.sa_sketch_fwd_noalloc.restype = c.c_int
    L.sa_sketch_fwd_tokenwise_workspace_size.argtypes = [i64, i64, i32, i32, i32, c.c_int]
    L.sa_sketch_fwd_tokenwise_workspace_size.restype = sz
    L.sa_sketch_fwd_tokenwise.argtypes = [vp, vp, vp, vp, i64, i64, i32, i32, i32, f32, c.c_int,
                                          vp, vp, vp, sz, vp]
    L.sa_sketch_fwd_tokenwise.restype = c.c_int
    L.sa_layer_fwd_workspace_size.argtypes = [i64, i64, i32, i32, i32, c.c_int]
    L.sa_layer_fwd_workspace_size.restype = sz
    L.sa_layer_fwd.argtypes = [vp, vp, vp, vp, vp, i64, i64, i32, i32, i32, f32, c.c_int, vp, vp,
                               vp, sz, vp]
    L.sa_layer_fwd.restype = c.c_int
    L.sa_layer_bwd_workspace_size.argtypes = [i64, i64, i32, i32, i32, c.c_int, i32]
    L.sa_layer_bwd_workspace_size.restype = sz
    L.sa_layer_bwd.argtypes = [vp, vp, vp, vp, vp, i64, i64, i32, i32, i32, f32, c.c_int, vp, i32,
                               vp, vp, vp, vp, vp, vp, sz, vp]
    L.sa_layer_bwd.restype = c.c_int
    L.sa_block_fwd_workspace_size.argtypes = [i64, i64, i32, i32, i32, i32, c.c_int]
    L.sa_block_fwd_workspace_size.restype = sz
    L.sa_block_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i32, i32, i32, i32, f32, f32,
                               c.c_int, vp, vp, vp, sz, vp, sz, vp]
    L.sa_block_fwd.restype = c.c_int
    L.sa_block_saved_size.argtypes = [i64, i64, i32, i32, i32, i32, c.c_int]
    L.sa_block_saved_size.restype = sz
    L.sa_block_saved_offset.argtypes = [i64, i64, i32, i32, i32, i32, c.c_int, i32, i32]
    L.sa_block_saved_offset.restype = sz
    L.sa_block_bwd_workspace_size.argtypes = [i64, i64, i32, i32, i32, i32, c.c_int, i32]
    L.sa_block_bwd_workspace_size.restype = sz
    L.sa_block_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i32, i32, i32, i32, f32, f32,
                               c.c_int, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp, sz, vp]
    L.sa_block_bwd.restype = c.c_int
    for nm in ("sa_stca_fwd_workspace_size", "sa_stca_bwd_workspace_size"):
        getattr(L, nm).argtypes = [i64, i32, i32, i32, i32, c.c_int]
        getattr(L, nm).restype = sz
    L.sa_stca_fwd.argtypes = [vp, vp, vp, vp, vp, i64, i32, i32, i32, i32, f32, c.c_int, vp, vp, vp, sz, vp]
    L.sa_stca_fwd.restype = c.c_int
    L.sa_stca_bwd.argtypes = [vp, vp, vp, vp, vp, i64, i32, i32, i32, i32, f32, c.c_int, vp, vp, vp, vp, vp, vp,
                              vp, sz, vp]
    L.sa_stca_bwd.restype = c.c_int
    L.sa_build_worklist.argtypes = [vp, i64, i64, i32, i64, vp, i64, vp, vp]
    L.sa_build_worklist.restype = c.c_int
    L.sa_status_string.argtypes = [c.c_int]
    L.sa_status_string.restype = c.c_char_p
    L.sa_last_error.argtypes = []
    L.sa_last_error.restype = c.c_char_p
    L.sa_profile_enable.argtypes = [i32]
    L.sa_profile_enable.restype = None
    L.sa_kernel_times.argtypes = [i32, vp, vp, vp]
    L.sa_kernel_times.restype = i32
    _lib = L
    return L


def _check(rc: int):
    if rc != 0:
        raise SAError(rc, lib().sa_last_error().decode())


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return SA_BF16
    if t.dtype == torch.float32:
        return SA_FP32
    raise SAError(1, f"unsupported tensor dtype {t.dtype}")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


def _require(t, name, shape, dtype, device):
    if t.shape != tuple(shape):
        raise SAError(1, f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise SAError(1, f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise SAError(1, f"{name} must be contiguous")
    if t.device != device:
        raise SAError(1, f"{name} is on {t.device}, expected {device}")


def fwd_workspace_size(B, T, H, M, d, dtype_code) -> int:
    return int(lib().sa_sketch_fwd_workspace_size(B, T, H, M, d, dtype_code))


def bwd_workspace_size(B, T, H, M, d, dtype_code, R) -> int:
    return int(lib().sa_sketch_bwd_workspace_size(B, T, H, M, d, dtype_code, R))


def fwd_chunk_tokens(B, T, H, M, d, dtype_code) -> int:
    return int(lib().sa_sketch_fwd_chunk_tokens(B, T, H, M, d, dtype_code))


def _workspace(nbytes, device, workspace):
    import torch
    if nbytes == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
    elif workspace.numel() * workspace.element_size() < nbytes:
        raise SAError(3, f"workspace of {nbytes} bytes needed")
    return workspace, workspace.numel() * workspace.element_size()


def sketch_fwd(K, V, P, offsets, scale: Optional[float] = None, sketch=None, lse=None,
               want_lse: bool = True, workspace=None, stream=None):
    """sa_sketch_fwd on torch tensors.  Returns (sketch [B,H,M,d] fp32, lse [T,H] or None)."""
    import torch
    T, H, d = K.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    dev = K.device
    code = _dtype_code(K)
    _require(K, "K", (T, H, d), K.dtype, dev)
    _require(V, "V", (T, H, d), K.dtype, dev)
    _require(P, "P", (H, M, d), K.dtype, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if sketch is None:
        sketch = torch.empty((B, H, M, d), dtype=torch.float32, device=dev)
    _require(sketch, "sketch", (B, H, M, d), torch.float32, dev)
    if lse is None and want_lse:
        lse = torch.empty((T, H), dtype=torch.float32, device=dev)
    if lse is not None:
        _require(lse, "lse", (T, H), torch.float32, dev)
    ws, nbytes = _workspace(fwd_workspace_size(B, T, H, M, d, code), dev, workspace)
    rc = lib().sa_sketch_fwd(_ptr(K), _ptr(V), _ptr(P), _ptr(offsets), B, T, H, M, d,
                             float(scale), code, _ptr(sketch), _ptr(lse), _ptr(ws), nbytes,
                             _stream_handle(stream))
    _check(rc)
    return sketch, lse


NOALLOC_SCRATCH_BYTES = 128 << 20


def sketch_fwd_noalloc(K, V, P, offsets, scale: Optional[float] = None, sketch=None, lse=None,
                       want_lse: bool = True, stream=None):
    """sa_sketch_fwd_noalloc on torch tensors: the library's own device scratch
    array instead of a workspace.  The caller passes (or this allocates, before the
    call) the outputs.  Returns (sketch, lse or None)."""
    import torch
    T, H, d = K.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    dev = K.device
    code = _dtype_code(K)
    _require(K, "K", (T, H, d), K.dtype, dev)
    _require(V, "V", (T, H, d), K.dtype, dev)
    _require(P, "P", (H, M, d), K.dtype, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if sketch is None:
        sketch = torch.empty((B, H, M, d), dtype=torch.float32, device=dev)
    _require(sketch, "sketch", (B, H, M, d), torch.float32, dev)
    if lse is None and want_lse:
        lse = torch.empty((T, H), dtype=torch.float32, device=dev)
    if lse is not None:
        _require(lse, "lse", (T, H), torch.float32, dev)
    rc = lib().sa_sketch_fwd_noalloc(_ptr(K), _ptr(V), _ptr(P), _ptr(offsets), B, T, H, M, d,
                                     float(scale), code, _ptr(sketch), _ptr(lse), _stream_handle(stream))
    _check(rc)
    return sketch, lse


def tokenwise_workspace_size(B, T, H, M, d, dtype_code) -> int:
    return int(lib().sa_sketch_fwd_tokenwise_workspace_size(B, T, H, M, d, dtype_code))


def sketch_fwd_tokenwise(K, V, P, offsets, scale: Optional[float] = None, sketch=None, lse_m=None,
                         want_lse: bool = True, workspace=None, stream=None):
    """sa_sketch_fwd_tokenwise on torch tensors (weights normalised over each user's
    tokens per prototype).  Returns (sketch [B,H,M,d] fp32, lse_m [B,H,M] or None)."""
    import torch
    T, H, d = K.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    dev = K.device
    code = _dtype_code(K)
    _require(K, "K", (T, H, d), K.dtype, dev)
    _require(V, "V", (T, H, d), K.dtype, dev)
    _require(P, "P", (H, M, d), K.dtype, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if sketch is None:
        sketch = torch.empty((B, H, M, d), dtype=torch.float32, device=dev)
    _require(sketch, "sketch", (B, H, M, d), torch.float32, dev)
    if lse_m is None and want_lse:
        lse_m = torch.empty((B, H, M), dtype=torch.float32, device=dev)
    if lse_m is not None:
        _require(lse_m, "lse_m", (B, H, M), torch.float32, dev)
    ws, nbytes = _workspace(tokenwise_workspace_size(B, T, H, M, d, code), dev, workspace)
    rc = lib().sa_sketch_fwd_tokenwise(_ptr(K), _ptr(V), _ptr(P), _ptr(offsets), B, T, H, M, d,
                                       float(scale), code, _ptr(sketch), _ptr(lse_m), _ptr(ws),
                                       nbytes, _stream_handle(stream))
    _check(rc)
    return sketch, lse_m


def sketch_bwd(K, V, P, offsets, dsketch, lse, scale: Optional[float] = None, dK=None,
               dV=None, dP=None, workspace=None, stream=None) -> Tuple:
    """sa_sketch_bwd on torch tensors.  dsketch: [B,R,H,M,d].  Returns (dK, dV, dP)."""
    import torch
    T, H, d = K.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    R = dsketch.shape[1]
    dev = K.device
    code = _dtype_code(K)
    _require(K, "K", (T, H, d), K.dtype, dev)
    _require(V, "V", (T, H, d), K.dtype, dev)
    _require(P, "P", (H, M, d), K.dtype, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    _require(dsketch, "dsketch", (B, R, H, M, d), torch.float32, dev)
    _require(lse, "lse", (T, H), torch.float32, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if dK is None:
        dK = torch.empty((T, H, d), dtype=torch.float32, device=dev)
    if dV is None:
        dV = torch.empty((T, H, d), dtype=torch.float32, device=dev)
    if dP is None:
        dP = torch.empty((H, M, d), dtype=torch.float32, device=dev)
    ws, nbytes = _workspace(bwd_workspace_size(B, T, H, M, d, code, R), dev, workspace)
    rc = lib().sa_sketch_bwd(_ptr(K), _ptr(V), _ptr(P), _ptr(offsets), B, T, H, M, d,
                             float(scale), code, _ptr(dsketch), R, _ptr(lse), _ptr(dK), _ptr(dV),
                             _ptr(dP), _ptr(ws), nbytes, _stream_handle(stream))
    _check(rc)
    return dK, dV, dP


def layer_fwd_workspace_size(B, T, H, M, d, dtype_code) -> int:
    return int(lib().sa_layer_fwd_workspace_size(B, T, H, M, d, dtype_code))


def layer_bwd_workspace_size(B, T, H, M, d, dtype_code, R) -> int:
    return int(lib().sa_layer_bwd_workspace_size(B, T, H, M, d, dtype_code, R))


def _layer_inputs(X, P, Wq, Wk, offsets):
    import torch
    T, H, d = X.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    dev = X.device
    _require(X, "X", (T, H, d), X.dtype, dev)
    _require(P, "P", (H, M, d), X.dtype, dev)
    _require(Wq, "Wq", (H, d, d), X.dtype, dev)
    _require(Wk, "Wk", (H, d, d), X.dtype, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    return B, T, H, M, d, dev, _dtype_code(X)


def layer_fwd(X, P, Wq, Wk, offsets, scale: Optional[float] = None, sketch=None, lse=None,
              want_lse: bool = True, workspace=None, stream=None):
    """sa_layer_fwd on torch tensors: one SA layer with its projections (K = X W_K,
    Q = P W_Q, the history X aggregated).  Returns (sketch [B,H,M,d] fp32, lse [T,H] or None)."""
    import torch
    B, T, H, M, d, dev, code = _layer_inputs(X, P, Wq, Wk, offsets)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if sketch is None:
        sketch = torch.empty((B, H, M, d), dtype=torch.float32, device=dev)
    _require(sketch, "sketch", (B, H, M, d), torch.float32, dev)
    if lse is None and want_lse:
        lse = torch.empty((T, H), dtype=torch.float32, device=dev)
    if lse is not None:
        _require(lse, "lse", (T, H), torch.float32, dev)
    ws, nbytes = _workspace(layer_fwd_workspace_size(B, T, H, M, d, code), dev, workspace)
    rc = lib().sa_layer_fwd(_ptr(X), _ptr(P), _ptr(Wq), _ptr(Wk), _ptr(offsets), B, T, H, M, d,
                            float(scale), code, _ptr(sketch), _ptr(lse), _ptr(ws), nbytes,
                            _stream_handle(stream))
    _check(rc)
    return sketch, lse


def layer_bwd(X, P, Wq, Wk, offsets, dsketch, lse, scale: Optional[float] = None, workspace=None,
              stream=None) -> Tuple:
    """sa_layer_bwd on torch tensors.  dsketch: [B,R,H,M,d].  Returns (dX, dP, dWq, dWk), fp32."""
    import torch
    B, T, H, M, d, dev, code = _layer_inputs(X, P, Wq, Wk, offsets)
    R = dsketch.shape[1]
    _require(dsketch, "dsketch", (B, R, H, M, d), torch.float32, dev)
    _require(lse, "lse", (T, H), torch.float32, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    dX = torch.empty((T, H, d), dtype=torch.float32, device=dev)
    dP = torch.empty((H, M, d), dtype=torch.float32, device=dev)
    dWq = torch.empty((H, d, d), dtype=torch.float32, device=dev)
    dWk = torch.empty((H, d, d), dtype=torch.float32, device=dev)
    ws, nbytes = _workspace(layer_bwd_workspace_size(B, T, H, M, d, code, R), dev, workspace)
    rc = lib().sa_layer_bwd(_ptr(X), _ptr(P), _ptr(Wq), _ptr(Wk), _ptr(offsets), B, T, H, M, d,
                            float(scale), code, _ptr(dsketch), R, _ptr(lse), _ptr(dX), _ptr(dP),
                            _ptr(dWq), _ptr(dWk), _ptr(ws), nbytes, _stream_handle(stream))
    _check(rc)
    return dX, dP, dWq, dWk


def block_fwd_workspace_size(B, T, H, M, d, n_layers, dtype_code) -> int:
    return int(lib().sa_block_fwd_workspace_size(B, T, H, M, d, n_layers, dtype_code))


def block_saved_size(B, T, H, M, d, n_layers, dtype_code) -> int:
    return int(lib().sa_block_saved_size(B, T, H, M, d, n_layers, dtype_code))


def block_saved_buffer(X, P, Wq, offsets):
    """A device buffer for the training forward's intermediates (sa_block_fwd's
    `saved`), sized for these inputs."""
    import torch
    T, H, d = X.shape
    n = block_saved_size(offsets.shape[0] - 1, T, H, P.shape[1], d, Wq.shape[0], _dtype_code(X))
    return torch.empty(max(n, 1), dtype=torch.uint8, device=X.device)


SAVED_ITEMS = {"state": 0, "Q": 1, "Pp": 2, "lse": 3}


def block_saved_views(saved, B, T, H, M, d, n_layers, dtype_code) -> list:
    """Views of the intermediates that a training block_fwd kept in `saved`, one
    dict per layer: "Q" and "Pp" [B,H,M,d] (fp32, and the input dtype for P'),
    "lse" [T,H], and "state" [B,H,M,d] for layers after the first.  The first
    layer's Q and P' are [H,M,d] (the shared prototypes' queries)."""
    import torch
    out = []
    el_dt = torch.bfloat16 if dtype_code == SA_BF16 else torch.float32
    for l in range(n_layers):
        views = {}
        for name, item in SAVED_ITEMS.items():
            off = int(lib().sa_block_saved_offset(B, T, H, M, d, n_layers, dtype_code, l, item))
            if off == (1 << 64) - 1:
                continue
            rows = (H * M if l == 0 else B * H * M) if name in ("Q", "Pp") else None
            dt = el_dt if name == "Pp" else torch.float32
            n = T * H if name == "lse" else (rows if rows is not None else B * H * M) * d
            nbytes = n * (2 if dt == torch.bfloat16 else 4)
            v = saved[off:off + nbytes].view(dt)
            if name == "lse":
                v = v.view(T, H)
            elif l == 0:
                v = v.view(H, M, d)
            else:
                v = v.view(B, H, M, d)
            views[name] = v
        out.append(views)
    return out


def _saved_arg(saved, nbytes):
    if saved is None:
        return None, 0
    have = saved.numel() * saved.element_size()
    if have < nbytes:
        raise SAError(3, f"saved buffer of {nbytes} bytes needed, {have} given")
    return saved, have


def block_fwd(X, P, Wq, Wk, ln, W1, W3, W2, offsets, scale: Optional[float] = None, eps: float = 1e-5,
              out=None, want_lse: bool = False, saved=None, workspace=None, stream=None):
    """sa_block_fwd on torch tensors: stacked SA with len(Wq) layers.
    With `saved` (from block_saved_buffer) the intermediates are kept there for
    block_bwd.  Returns (out [B,H,M,d] fp32, lse [n_layers,T,H] or None)."""
    import torch
    T, H, d = X.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    L = Wq.shape[0]
    dev = X.device
    code = _dtype_code(X)
    dt = X.dtype
    _require(X, "X", (T, H, d), dt, dev)
    _require(P, "P", (H, M, d), dt, dev)
    _require(Wq, "Wq", (L, H, d, d), dt, dev)
    _require(Wk, "Wk", (L, H, d, d), dt, dev)
    _require(ln, "ln", (L, 4, H, d), dt, dev)
    _require(W1, "W1", (L, H, d, 2 * d), dt, dev)
    _require(W3, "W3", (L, H, d, 2 * d), dt, dev)
    _require(W2, "W2", (L, H, 2 * d, d), dt, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty((B, H, M, d), dtype=torch.float32, device=dev)
    _require(out, "out", (B, H, M, d), torch.float32, dev)
    lse = torch.empty((L, T, H), dtype=torch.float32, device=dev) if want_lse else None
    ws, nbytes = _workspace(block_fwd_workspace_size(B, T, H, M, d, L, code), dev, workspace)
    sv, sbytes = _saved_arg(saved, block_saved_size(B, T, H, M, d, L, code))
    rc = lib().sa_block_fwd(_ptr(X), _ptr(P), _ptr(Wq), _ptr(Wk), _ptr(ln), _ptr(W1), _ptr(W3), _ptr(W2),
                            _ptr(offsets), B, T, H, M, d, L, float(scale), float(eps), code, _ptr(out),
                            _ptr(lse), _ptr(sv), sbytes, _ptr(ws), nbytes, _stream_handle(stream))
    _check(rc)
    return out, lse


def block_bwd_workspace_size(B, T, H, M, d, n_layers, dtype_code, with_saved: bool = False) -> int:
    return int(lib().sa_block_bwd_workspace_size(B, T, H, M, d, n_layers, dtype_code, int(bool(with_saved))))


def block_bwd(X, P, Wq, Wk, ln, W1, W3, W2, offsets, dout, scale: Optional[float] = None, eps: float = 1e-5,
              saved=None, workspace=None, stream=None):
    """sa_block_bwd on torch tensors: gradients of <dout, block_fwd(...)>.
    `saved`: the buffer a training block_fwd with the same inputs filled (the
    forward is then not replayed), or None.
    Returns a dict of fp32 tensors dX, dP, dWq, dWk, dln, dW1, dW3, dW2 (shapes of
    the inputs)."""
    import torch
    T, H, d = X.shape
    M = P.shape[1]
    B = offsets.shape[0] - 1
    L = Wq.shape[0]
    dev = X.device
    code = _dtype_code(X)
    dt = X.dtype
    _require(X, "X", (T, H, d), dt, dev)
    _require(P, "P", (H, M, d), dt, dev)
    _require(Wq, "Wq", (L, H, d, d), dt, dev)
    _require(Wk, "Wk", (L, H, d, d), dt, dev)
    _require(ln, "ln", (L, 4, H, d), dt, dev)
    _require(W1, "W1", (L, H, d, 2 * d), dt, dev)
    _require(W3, "W3", (L, H, d, 2 * d), dt, dev)
    _require(W2, "W2", (L, H, 2 * d, d), dt, dev)
    _require(offsets, "offsets", (B + 1,), torch.int64, dev)
    _require(dout, "dout", (B, H, M, d), torch.float32, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    f32 = dict(dtype=torch.float32, device=dev)
    g = {"dX": torch.empty((T, H, d), **f32), "dP": torch.empty((H, M, d), **f32),
         "dWq": torch.empty((L, H, d, d), **f32), "dWk": torch.empty((L, H, d, d), **f32),
         "dln": torch.empty((L, 4, H, d), **f32), "dW1": torch.empty((L, H, d, 2 * d), **f32),
         "dW3": torch.empty((L, H, d, 2 * d), **f32), "dW2": torch.empty((L, H, 2 * d, d), **f32)}
    ws, nbytes = _workspace(block_bwd_workspace_size(B, T, H, M, d, L, code, saved is not None), dev, workspace)
    sv, sbytes = _saved_arg(saved, block_saved_size(B, T, H, M, d, L, code))
    rc = lib().sa_block_bwd(_ptr(X), _ptr(P), _ptr(Wq), _ptr(Wk), _ptr(ln), _ptr(W1), _ptr(W3), _ptr(W2),
                            _ptr(offsets), B, T, H, M, d, L, float(scale), float(eps), code, _ptr(dout),
                            _ptr(g["dX"]), _ptr(g["dP"]), _ptr(g["dWq"]), _ptr(g["dWk"]), _ptr(g["dln"]),
                            _ptr(g["dW1"]), _ptr(g["dW3"]), _ptr(g["dW2"]), _ptr(sv), sbytes, _ptr(ws), nbytes,
                            _stream_handle(stream))
    _check(rc)
    return g


def stca_fwd_workspace_size(B, R, k, D, h, dtype_code) -> int:
    return int(lib().sa_stca_fwd_workspace_size(B, R, k, D, h, dtype_code))


def stca_bwd_workspace_size(B, R, k, D, h, dtype_code) -> int:
    return int(lib().sa_stca_bwd_workspace_size(B, R, k, D, h, dtype_code))


def _stca_check(Xs, q, Wq, Wk, Wv):
    import torch
    B, k, D = Xs.shape
    R = q.shape[1]
    dev, dt = Xs.device, Xs.dtype
    _require(Xs, "Xs", (B, k, D), dt, dev)
    _require(q, "q", (B, R, D), dt, dev)
    for name, W in (("Wq", Wq), ("Wk", Wk), ("Wv", Wv)):
        _require(W, name, (D, D), dt, dev)
    return B, R, k, D, dev, _dtype_code(Xs), torch


def stca_fwd(Xs, q, Wq, Wk, Wv, h: int, scale: Optional[float] = None, out=None, want_lse: bool = False,
             workspace=None, stream=None):
    """sa_stca_fwd on torch tensors: reordered single-query STCA of R targets per user
    over the user's sketch.  Returns (out [B,R,D] fp32, lse [B,R,h] or None)."""
    B, R, k, D, dev, code, torch = _stca_check(Xs, q, Wq, Wk, Wv)
    if scale is None:
        scale = 1.0 / math.sqrt(D // h)
    if out is None:
        out = torch.empty((B, R, D), dtype=torch.float32, device=dev)
    _require(out, "out", (B, R, D), torch.float32, dev)
    lse = torch.empty((B, R, h), dtype=torch.float32, device=dev) if want_lse else None
    ws, nbytes = _workspace(stca_fwd_workspace_size(B, R, k, D, h, code), dev, workspace)
    rc = lib().sa_stca_fwd(_ptr(Xs), _ptr(q), _ptr(Wq), _ptr(Wk), _ptr(Wv), B, R, k, D, h, float(scale), code,
                           _ptr(out), _ptr(lse), _ptr(ws), nbytes, _stream_handle(stream))
    _check(rc)
    return out, lse


def stca_bwd(Xs, q, Wq, Wk, Wv, h: int, dout, scale: Optional[float] = None, workspace=None, stream=None):
    """sa_stca_bwd on torch tensors: dict of fp32 gradients dXs, dq, dWq, dWk, dWv."""
    B, R, k, D, dev, code, torch = _stca_check(Xs, q, Wq, Wk, Wv)
    _require(dout, "dout", (B, R, D), torch.float32, dev)
    if scale is None:
        scale = 1.0 / math.sqrt(D // h)
    f32 = dict(dtype=torch.float32, device=dev)
    g = {"dXs": torch.empty((B, k, D), **f32), "dq": torch.empty((B, R, D), **f32),
         "dWq": torch.empty((D, D), **f32), "dWk": torch.empty((D, D), **f32), "dWv": torch.empty((D, D), **f32)}
    ws, nbytes = _workspace(stca_bwd_workspace_size(B, R, k, D, h, code), dev, workspace)
    rc = lib().sa_stca_bwd(_ptr(Xs), _ptr(q), _ptr(Wq), _ptr(Wk), _ptr(Wv), B, R, k, D, h, float(scale), code,
                           _ptr(dout), _ptr(g["dXs"]), _ptr(g["dq"]), _ptr(g["dWq"]), _ptr(g["dWk"]),
                           _ptr(g["dWv"]), _ptr(ws), nbytes, _stream_handle(stream))
    _check(rc)
    return g


def gemm_tile_shapes() -> int:
    return int(lib().sa_gemm_tile_shapes())


def gemm_bf16(A, a_strides, B, b_strides, C, c_strides, M, N, K, batch, alpha=1.0, accumulate=False, b_mod=0,
              tile_shape=-1, stream=None):
    """sa_gemm_bf16 on torch tensors: A, B bf16 and C (fp32 or bf16) device
    tensors addressed by (z, row, col) element strides a_strides = (a_z, a_m, a_k),
    b_strides = (b_z, b_k, b_n), c_strides = (c_z, c_m).  Returns C."""
    import torch
    for name, t in (("A", A), ("B", B)):
        if t.dtype != torch.bfloat16 or not t.is_cuda:
            raise SAError(1, f"{name} must be a bf16 device tensor")
    if C.dtype not in (torch.float32, torch.bfloat16) or not C.is_cuda:
        raise SAError(1, "C must be a fp32 or bf16 device tensor")
    rc = lib().sa_gemm_bf16(_ptr(A), *a_strides, _ptr(B), *b_strides, b_mod, _ptr(C),
                            1 if C.dtype == torch.bfloat16 else 0, *c_strides, M, N, K, batch, float(alpha),
                            1 if accumulate else 0, tile_shape, _stream_handle(stream))
    _check(rc)
    return C


def profile_enable(on: bool = True) -> None:
    """Bracket every library launch of this thread with HIP events (benchmarks)."""
    lib().sa_profile_enable(1 if on else 0)


def kernel_times(max_kernels: int = 32) -> dict:
    """{kernel name: (launches, total ms)} since the previous call (waits for the events)."""
    names = ctypes.create_string_buffer(48 * max_kernels)
    n_l = (ctypes.c_int64 * max_kernels)()
    ms = (ctypes.c_double * max_kernels)()
    n = lib().sa_kernel_times(max_kernels, ctypes.addressof(names), ctypes.addressof(n_l),
                              ctypes.addressof(ms))
    if n < 0:
        raise SAError(5, "collecting kernel times failed")
    out = {}
    for i in range(n):
        nm = names.raw[48 * i: 48 * (i + 1)].split(b"\0", 1)[0].decode()
        out[nm] = (int(n_l[i]), float(ms[i]))
    return out


def build_worklist(offsets, T: int, H: int, chunk_tokens: int, max_items: Optional[int] = None,
                   stream=None):
    """sa_build_worklist: returns the items as an int32 tensor [n_items, 8] on the device."""
    import torch
    B = offsets.shape[0] - 1
    if max_items is None:
        max_items = (H * T + chunk_tokens - 1) // chunk_tokens + H * B
    items = torch.empty((max(max_items, 1), ITEM_WORDS), dtype=torch.int32, device=offsets.device)
    n = torch.zeros(1, dtype=torch.int64, device=offsets.device)
    rc = lib().sa_build_worklist(_ptr(offsets), B, T, H, chunk_tokens, _ptr(items), max_items,
                                 _ptr(n), _stream_handle(stream))
    _check(rc)
    return items[: int(n.item())]

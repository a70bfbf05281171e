"""CPU oracle of the SA sketching step (fp64).  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU library
and never imports it.  The arithmetic lives in ``sa_oracle.c``; this module
only marshals numpy arrays.

Functions follow SequenceO1 section 3.1 (affinities S, prototype-wise softmax
A, sketch A X), Appendix B steps 1-3, and the chain-rule backward stated in the
header of ``sa_oracle.c``; ``fwd_tokenwise`` is the token-wise normalised
alternative of the appendix on prototype-wise normalisation.  ``oracle.layer``
holds the SA layer with its projections (Appendix G.3: Q = P W_Q, K = X W_K,
V = X) in fp64 numpy; ``oracle.block`` the stacked SA block (section 3.3) and
``oracle.stca`` the reordered single-query STCA over the sketch (Appendix G.2).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsa_oracle.so")
_lib = None

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(os.path.join(_HERE, "sa_oracle.c"))):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    c = ctypes
    lib.sa_oracle_fwd.argtypes = [_f32p, _f32p, _f32p, _i64p, c.c_int64, c.c_int32,
                                  c.c_int32, c.c_int32, c.c_double, _f64p,
                                  c.c_void_p, c.c_int32]
    lib.sa_oracle_fwd.restype = c.c_int
    lib.sa_oracle_bwd.argtypes = [_f32p, _f32p, _f32p, _i64p, c.c_int64, c.c_int32,
                                  c.c_int32, c.c_int32, c.c_double, _f32p, c.c_int32,
                                  _f64p, _f64p, _f64p, c.c_int32]
    lib.sa_oracle_bwd.restype = c.c_int
    lib.sa_oracle_weights.argtypes = [_f32p, _f32p, c.c_int64, c.c_int32, c.c_int32,
                                      c.c_int32, c.c_double, _f64p, c.c_void_p]
    lib.sa_oracle_weights.restype = c.c_int
    lib.sa_oracle_fwd_tokenwise.argtypes = [_f32p, _f32p, _f32p, _i64p, c.c_int64, c.c_int32,
                                            c.c_int32, c.c_int32, c.c_double, _f64p,
                                            c.c_void_p, c.c_int32]
    lib.sa_oracle_fwd_tokenwise.restype = c.c_int
    lib.sa_oracle_max_threads.argtypes = []
    lib.sa_oracle_max_threads.restype = c.c_int
    _lib = lib
    return lib


def _f32(x):
    return np.ascontiguousarray(x, dtype=np.float32)


def _dims(K, P):
    K = np.asarray(K)
    P = np.asarray(P)
    if K.ndim != 3 or P.ndim != 3 or K.shape[1] != P.shape[0] or K.shape[2] != P.shape[2]:
        raise ValueError(f"shape mismatch K{K.shape} P{P.shape}")
    return K.shape[0], P.shape[0], P.shape[1], P.shape[2]


def max_threads() -> int:
    return int(_load().sa_oracle_max_threads())


def fwd(K, V, P, offsets, scale=None, nthreads: int = 0, want_lse: bool = True):
    """Forward oracle.

    K, V: [T,H,d]; P: [H,M,d]; offsets: int64 [B+1].
    Returns (sketch [B,H,M,d] fp64, lse [T,H] fp64 or None).
    """
    lib = _load()
    T, H, M, d = _dims(K, P)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    B = offsets.shape[0] - 1
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    sketch = np.empty((B, H, M, d), np.float64)
    lse = np.full((T, H), np.nan, np.float64) if want_lse else None
    rc = lib.sa_oracle_fwd(_f32(K), _f32(V), _f32(P), offsets, B, H, M, d, float(scale),
                           sketch, lse.ctypes.data if want_lse else None, int(nthreads))
    if rc != 0:
        raise ValueError(f"sa_oracle_fwd failed ({rc})")
    return sketch, lse


def bwd(K, V, P, offsets, dsketch, scale=None, nthreads: int = 0):
    """Backward oracle.  dsketch: [B,R,H,M,d].  Returns (dK, dV, dP) in fp64."""
    lib = _load()
    T, H, M, d = _dims(K, P)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    B = offsets.shape[0] - 1
    dsketch = _f32(dsketch)
    if dsketch.shape[0] != B or dsketch.shape[2:] != (H, M, d):
        raise ValueError(f"dsketch shape {dsketch.shape}")
    R = dsketch.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    dK = np.zeros((T, H, d), np.float64)
    dV = np.zeros((T, H, d), np.float64)
    dP = np.zeros((H, M, d), np.float64)
    rc = lib.sa_oracle_bwd(_f32(K), _f32(V), _f32(P), offsets, B, H, M, d, float(scale),
                           dsketch, R, dK, dV, dP, int(nthreads))
    if rc != 0:
        raise ValueError(f"sa_oracle_bwd failed ({rc})")
    return dK, dV, dP


def weights(K, P, scale=None):
    """Allocation weights A[t,h,m] (softmax over prototypes) and lse[t,h]."""
    lib = _load()
    T, H, M, d = _dims(K, P)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    A = np.empty((T, H, M), np.float64)
    lse = np.empty((T, H), np.float64)
    rc = lib.sa_oracle_weights(_f32(K), _f32(P), T, H, M, d, float(scale), A, lse.ctypes.data)
    if rc != 0:
        raise ValueError(f"sa_oracle_weights failed ({rc})")
    return A, lse


def fwd_tokenwise(K, V, P, offsets, scale=None, nthreads: int = 0, want_lse: bool = True):
    """Token-wise normalised forward (softmax over each user's tokens per prototype).

    Returns (sketch [B,H,M,d] fp64, lse_m [B,H,M] fp64 or None; -inf for empty users).
    """
    lib = _load()
    T, H, M, d = _dims(K, P)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    B = offsets.shape[0] - 1
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    sketch = np.empty((B, H, M, d), np.float64)
    lse = np.full((B, H, M), np.nan, np.float64) if want_lse else None
    rc = lib.sa_oracle_fwd_tokenwise(_f32(K), _f32(V), _f32(P), offsets, B, H, M, d, float(scale),
                                     sketch, lse.ctypes.data if want_lse else None, int(nthreads))
    if rc != 0:
        raise ValueError(f"sa_oracle_fwd_tokenwise failed ({rc})")
    return sketch, lse

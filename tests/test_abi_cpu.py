"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every entry point include/sa_sketch.h declares, and rejects bad arguments
before anything is enqueued."""
import ctypes
import os
import re

import pytest

from oracle import worklist as wlref
from paper_2609_08443_amd import sa_sketch as sa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sa_sketch.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sa_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = sa.lib()
    names = declared_functions()
    assert len(names) >= 8, names
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(sa.EXPORTS)


def test_status_strings():
    L = sa.lib()
    for code, name in sa._STATUS.items():
        assert L.sa_status_string(code).decode() == name


NULL = None


def call_fwd(B=2, T=10, H=1, M=128, d=64, scale=0.125, dtype=sa.SA_BF16, K=1 << 12, V=1 << 12,
             P=1 << 12, off=1 << 12, sketch=1 << 12, lse=NULL, ws=NULL, wsb=0):
    return sa.lib().sa_sketch_fwd(K, V, P, off, B, T, H, M, d, scale, dtype, sketch, lse, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), 1), (dict(H=0), 1), (dict(M=0), 1), (dict(d=0), 1), (dict(T=-5), 1),
    (dict(d=96), 2), (dict(d=32), 2), (dict(M=5000), 2), (dict(T=1 << 31), 2),
    (dict(scale=float("nan")), 1), (dict(scale=-1.0), 1), (dict(scale=float("inf")), 1),
    (dict(dtype=7), 2),
    (dict(K=NULL), 1), (dict(V=NULL), 1), (dict(P=NULL), 1), (dict(off=NULL), 1),
    (dict(sketch=NULL), 1),
    (dict(K=(1 << 12) + 4), 1), (dict(sketch=(1 << 12) + 8), 1), (dict(lse=(1 << 12) + 2), 1),
])
def test_fwd_rejects_bad_arguments(kw, code):
    assert call_fwd(**kw) == code
    assert sa.lib().sa_last_error().decode() != ""


def test_fwd_zero_users_is_noop():
    # B = 0 returns before touching any pointer
    assert call_fwd(B=0, K=NULL, V=NULL, P=NULL, off=NULL, sketch=NULL) == 0


def test_fwd_workspace_too_small():
    need = sa.fwd_workspace_size(2, 10, 1, 128, 64, sa.SA_BF16)
    assert need > 0
    assert call_fwd(ws=NULL, wsb=0) == 3
    assert call_fwd(ws=1 << 20, wsb=need - 1) == 3


def test_bwd_rejects_bad_arguments():
    L = sa.lib()
    p = 1 << 12
    args = dict(K=p, V=p, P=p, off=p, B=2, T=10, H=1, M=128, d=64, scale=0.125, dtype=0, ds=p,
                R=1, lse=p, dK=p, dV=p, dP=p, ws=NULL, wsb=0)

    def call(**kw):
        a = dict(args, **kw)
        return L.sa_sketch_bwd(a["K"], a["V"], a["P"], a["off"], a["B"], a["T"], a["H"], a["M"],
                               a["d"], a["scale"], a["dtype"], a["ds"], a["R"], a["lse"], a["dK"],
                               a["dV"], a["dP"], a["ws"], a["wsb"], None)
    assert call(R=0) == 1
    assert call(lse=NULL) == 1
    assert call(ds=NULL) == 1
    assert call(dP=NULL) == 1
    assert call(d=80) == 2
    assert call() == 3  # no workspace
    assert sa.bwd_workspace_size(2, 10, 1, 128, 64, 0, 1) > 0


def test_worklist_rejects_bad_arguments():
    L = sa.lib()
    assert L.sa_build_worklist(1 << 12, 2, 10, 1, 0, 1 << 12, 4, 1 << 12, None) == 1
    assert L.sa_build_worklist(None, 2, 10, 1, 4, 1 << 12, 4, 1 << 12, None) == 1
    assert L.sa_build_worklist(1 << 12, 2, 10, 1, 4, 1 << 12, 4, None, None) == 1


@pytest.mark.parametrize("offsets,T,H,C", [
    ([0, 5, 5, 17, 18], 18, 2, 4), ([0, 100], 100, 3, 32), ([0, 0, 0], 0, 2, 7),
    ([0, 1, 2, 3], 3, 1, 1), ([0, 64, 64, 200], 200, 2, 64)])
def test_reference_worklist_covers_every_token_once(offsets, T, H, C):
    items = wlref.worklist(offsets, T, H, C)
    assert wlref.coverage_ok(items, offsets, H)
    n_ranges = (H * T + C - 1) // C
    assert len(items) <= n_ranges + H * (len(offsets) - 1)
    for (b, h, t0, t1, r, split, first, _) in items:
        assert t1 > t0 and r * C <= h * T + t0 and h * T + t1 <= (r + 1) * C


def test_layer_fwd_rejects_bad_arguments():
    L = sa.lib()
    p = 1 << 12
    args = dict(X=p, P=p, Wq=p, Wk=p, off=p, B=2, T=10, H=1, M=128, d=64, scale=0.125, dtype=0,
                sketch=p, lse=NULL, ws=NULL, wsb=0)

    def call(**kw):
        a = dict(args, **kw)
        return L.sa_layer_fwd(a["X"], a["P"], a["Wq"], a["Wk"], a["off"], a["B"], a["T"], a["H"],
                              a["M"], a["d"], a["scale"], a["dtype"], a["sketch"], a["lse"], a["ws"],
                              a["wsb"], None)
    for name in ("X", "P", "Wq", "Wk", "off", "sketch"):
        assert call(**{name: NULL}) == 1, name
    assert call(Wk=p + 2) == 1
    assert call(d=96) == 2
    assert call(B=0, X=NULL, P=NULL) == 0
    need = sa.layer_fwd_workspace_size(2, 10, 1, 128, 64, 0)
    # at least Q (fp32) and P' (bf16) on top of the sketching workspace
    assert need >= sa.fwd_workspace_size(2, 10, 1, 128, 64, 0) + 128 * 64 * 6
    assert call() == 3
    assert call(ws=1 << 20, wsb=need - 1) == 3


def test_layer_bwd_rejects_bad_arguments():
    L = sa.lib()
    p = 1 << 12
    args = dict(X=p, P=p, Wq=p, Wk=p, off=p, B=2, T=10, H=1, M=128, d=64, scale=0.125, dtype=0,
                ds=p, R=1, lse=p, dX=p, dP=p, dWq=p, dWk=p, ws=NULL, wsb=0)

    def call(**kw):
        a = dict(args, **kw)
        return L.sa_layer_bwd(a["X"], a["P"], a["Wq"], a["Wk"], a["off"], a["B"], a["T"], a["H"],
                              a["M"], a["d"], a["scale"], a["dtype"], a["ds"], a["R"], a["lse"],
                              a["dX"], a["dP"], a["dWq"], a["dWk"], a["ws"], a["wsb"], None)
    assert call(R=0) == 1
    for name in ("X", "P", "Wq", "Wk", "ds", "lse", "dX", "dP", "dWq", "dWk"):
        assert call(**{name: NULL}) == 1, name
    assert call(dWq=p + 4) == 1
    assert call(d=80) == 2
    assert call() == 3
    assert sa.layer_bwd_workspace_size(2, 10, 1, 128, 64, 0, 1) > sa.bwd_workspace_size(2, 10, 1, 128, 64, 0, 1)


def test_block_fwd_rejects_bad_arguments():
    L = sa.lib()
    p = 1 << 12
    args = dict(X=p, P=p, Wq=p, Wk=p, ln=p, W1=p, W3=p, W2=p, off=p, B=2, T=10, H=1, M=128, d=64, n=2,
                scale=0.125, eps=1e-5, dtype=0, out=p, lse=NULL, sv=NULL, svb=0, ws=NULL, wsb=0)

    def call(**kw):
        a = dict(args, **kw)
        return L.sa_block_fwd(a["X"], a["P"], a["Wq"], a["Wk"], a["ln"], a["W1"], a["W3"], a["W2"], a["off"],
                              a["B"], a["T"], a["H"], a["M"], a["d"], a["n"], a["scale"], a["eps"], a["dtype"],
                              a["out"], a["lse"], a["sv"], a["svb"], a["ws"], a["wsb"], None)
    for name in ("X", "P", "Wq", "Wk", "ln", "W1", "W3", "W2", "off", "out"):
        assert call(**{name: NULL}) == 1, name
    assert call(n=0) == 1
    assert call(eps=0.0) == 1 and call(eps=float("nan")) == 1
    assert call(W2=p + 2) == 1
    assert call(d=96) == 2
    assert call() == 3
    # a saved buffer too small or misaligned is rejected before any launch
    need = sa.block_saved_size(2, 10, 1, 128, 64, 2, 0)
    assert need > 0 and sa.block_saved_size(2, 10, 1, 128, 64, 0, 0) == 0
    assert call(ws=p, wsb=1 << 40, sv=p, svb=need - 1) == 3
    assert call(ws=p, wsb=1 << 40, sv=p + 4, svb=need) == 3
    assert sa.block_fwd_workspace_size(2, 10, 1, 128, 64, 2, 0) > sa.fwd_workspace_size(2, 10, 1, 128, 64, 0)


def test_block_bwd_rejects_bad_arguments():
    L = sa.lib()
    p = 1 << 12
    args = dict(X=p, P=p, Wq=p, Wk=p, ln=p, W1=p, W3=p, W2=p, off=p, B=2, T=10, H=1, M=128, d=64, n=2,
                scale=0.125, eps=1e-5, dtype=0, dout=p, dX=p, dP=p, dWq=p, dWk=p, dln=p, dW1=p, dW3=p, dW2=p,
                sv=NULL, svb=0, ws=NULL, wsb=0)

    def call(**kw):
        a = dict(args, **kw)
        return L.sa_block_bwd(a["X"], a["P"], a["Wq"], a["Wk"], a["ln"], a["W1"], a["W3"], a["W2"], a["off"],
                              a["B"], a["T"], a["H"], a["M"], a["d"], a["n"], a["scale"], a["eps"], a["dtype"],
                              a["dout"], a["dX"], a["dP"], a["dWq"], a["dWk"], a["dln"], a["dW1"], a["dW3"],
                              a["dW2"], a["sv"], a["svb"], a["ws"], a["wsb"], None)
    for name in ("X", "P", "Wq", "Wk", "ln", "W1", "W3", "W2", "off", "dout", "dX", "dP", "dWq", "dWk", "dln",
                 "dW1", "dW3", "dW2"):
        assert call(**{name: NULL}) == 1, name
    assert call(n=0) == 1 and call(B=0) == 1
    assert call(eps=-1.0) == 1
    assert call(dW3=p + 8) == 1
    assert call(d=96) == 2
    assert call() == 3
    need = sa.block_saved_size(2, 10, 1, 128, 64, 2, 0)
    assert call(ws=p, wsb=1 << 40, sv=p, svb=need - 1) == 3
    assert call(ws=p, wsb=1 << 40, sv=p + 4, svb=need) == 3
    assert sa.block_bwd_workspace_size(2, 10, 1, 128, 64, 2, 0) > sa.block_fwd_workspace_size(2, 10, 1, 128, 64, 2, 0)
    # with a saved buffer the replay's per-layer region is left out of the workspace
    assert (sa.block_bwd_workspace_size(2, 10, 1, 128, 64, 2, 0)
            - sa.block_bwd_workspace_size(2, 10, 1, 128, 64, 2, 0, True)) == need


def test_stca_rejects_bad_arguments():
    L = sa.lib()
    p = 1 << 12
    fargs = dict(X=p, q=p, Wq=p, Wk=p, Wv=p, B=2, R=4, k=64, D=128, h=2, scale=0.125, dtype=0, out=p, lse=NULL,
                 ws=NULL, wsb=0)

    def fwd(**kw):
        a = dict(fargs, **kw)
        return L.sa_stca_fwd(a["X"], a["q"], a["Wq"], a["Wk"], a["Wv"], a["B"], a["R"], a["k"], a["D"], a["h"],
                             a["scale"], a["dtype"], a["out"], a["lse"], a["ws"], a["wsb"], None)
    for name in ("X", "q", "Wq", "Wk", "Wv", "out"):
        assert fwd(**{name: NULL}) == 1, name
    assert fwd(h=3) == 1 and fwd(R=0) == 1 and fwd(k=0) == 1 and fwd(scale=0.0) == 1 and fwd(dtype=7) == 1
    assert fwd(q=p + 4) == 1
    assert fwd(B=0) == 0
    assert fwd() == 3
    bargs = dict(fargs, dout=p, dX=p, dq=p, dWq=p, dWk=p, dWv=p)

    def bwd(**kw):
        a = dict(bargs, **kw)
        return L.sa_stca_bwd(a["X"], a["q"], a["Wq"], a["Wk"], a["Wv"], a["B"], a["R"], a["k"], a["D"], a["h"],
                             a["scale"], a["dtype"], a["dout"], a["dX"], a["dq"], a["dWq"], a["dWk"], a["dWv"],
                             a["ws"], a["wsb"], None)
    for name in ("X", "q", "Wq", "Wk", "Wv", "dout", "dX", "dq", "dWq", "dWk", "dWv"):
        assert bwd(**{name: NULL}) == 1, name
    assert bwd(B=0) == 1 and bwd(D=100, h=3) == 1
    assert bwd() == 3
    assert sa.stca_bwd_workspace_size(2, 4, 64, 128, 2, 0) > sa.stca_fwd_workspace_size(2, 4, 64, 128, 2, 0) > 0


def test_block_saved_offsets():
    """Offsets of the saved intermediates: inside the buffer, 256-byte aligned,
    per layer at a fixed stride; invalid requests give (size_t)-1."""
    L = sa.lib()
    B, T, H, M, d, n = 3, 700, 2, 128, 64, 2
    bad = (1 << 64) - 1
    total = L.sa_block_saved_size(B, T, H, M, d, n, sa.SA_BF16)
    offs = {}
    for l in range(n):
        for item in range(4):
            o = L.sa_block_saved_offset(B, T, H, M, d, n, sa.SA_BF16, l, item)
            if l == 0 and item == 0:
                assert o == bad
                continue
            assert o % 256 == 0 and o < total
            offs[l, item] = o
    stride = total // n
    for item in range(1, 4):
        assert offs[1, item] - offs[0, item] == stride
    assert offs[0, 2] - offs[0, 1] >= 4 * B * H * M * d       # Q (fp32) before P'
    assert offs[0, 3] - offs[0, 2] >= 2 * B * H * M * d       # P' (bf16) before lse
    for args in ((n, sa.SA_BF16, n, 1), (n, sa.SA_BF16, -1, 1), (n, sa.SA_BF16, 0, 4), (0, sa.SA_BF16, 0, 1)):
        assert L.sa_block_saved_offset(B, T, H, M, d, *args) == bad

"""sa_sketch_fwd_noalloc (the forward for callers that cannot allocate: the
library's own device scratch array instead of a workspace) against
sa_sketch_fwd, through the C ABI: two calls in a row, the second on a smaller
input, each bit-identical to the workspace entry point (same kernels, same
plan) and within the oracle's bounds; a shape beyond the scratch size is
rejected before any launch."""
import numpy as np
import pytest

import oracle
from paper_2609_08443_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sa():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_08443_amd import sa_sketch
    sa_sketch.lib()
    return sa_sketch


def normwise(gpu, ref, axes):
    err = np.abs(gpu.astype(np.float64) - ref).max(axis=axes)
    return err / np.maximum(np.abs(ref).max(axis=axes), 1e-30)


CASES = [  # (lengths, H, M, d, dtype): a long split user, then a smaller batch
    ([3000, 0, 47, 1200, 5], 2, 512, 128, "bf16"),
    ([70, 0, 33], 1, 256, 64, "bf16"),
    ([40, 0, 77], 2, 64, 64, "fp32"),
]


def test_noalloc_matches_workspace_entry_point(sa):
    for i, (lengths, H, M, d, dtype) in enumerate(CASES):
        w = wl.custom(lengths, H, M, d, dtype, seed=500 + i)
        host = wl.host_tensors(w)
        dev = wl.to_device(host, dtype)
        print(f"no-alloc call {i}: lengths={lengths} H={H} M={M} d={d} {dtype}", flush=True)
        sk0, lse0 = sa.sketch_fwd(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
        sk1, lse1 = sa.sketch_fwd_noalloc(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale)
        torch.cuda.synchronize()
        assert torch.equal(sk0, sk1) and torch.equal(lse0, lse1)
        ref, rlse = oracle.fwd(host["K"], host["V"], host["P"], host["offsets"], w.scale)
        e = normwise(sk1.cpu().numpy(), ref, (2, 3))
        nonempty = np.asarray(w.lengths) > 0
        assert np.all(e[nonempty] <= (2e-2 if dtype == "bf16" else 1e-4)), e.max()
        assert np.abs(lse1.cpu().numpy() - rlse).max() <= (1e-3 if dtype == "bf16" else 1e-5)
    # the plain path without lse uses the scratch for its lse
    sk2, none = sa.sketch_fwd_noalloc(dev["K"], dev["V"], dev["P"], dev["offsets"], w.scale, want_lse=False)
    torch.cuda.synchronize()
    assert none is None and torch.equal(sk2, sk0)


def test_noalloc_rejects_shapes_beyond_its_scratch(sa):
    B, T, H, M, d = 64, 6_400_000, 8, 1024, 64
    need = sa.fwd_workspace_size(B, T, H, M, d, sa.SA_BF16)
    assert need > sa.NOALLOC_SCRATCH_BYTES
    # host-side rejection: no tensor is touched (null pointers would be refused
    # anyway, so small stand-ins of the right alignment are passed)
    K = torch.empty(8, dtype=torch.bfloat16, device="cuda")
    off = torch.zeros(B + 1, dtype=torch.int64, device="cuda")
    sk = torch.empty(8, dtype=torch.float32, device="cuda")
    rc = sa.lib().sa_sketch_fwd_noalloc(sa._ptr(K), sa._ptr(K), sa._ptr(K), sa._ptr(off), B, T, H, M, d,
                                        0.125, sa.SA_BF16, sa._ptr(sk), None, None)
    assert rc == 3
    assert b"no-allocation" in sa.lib().sa_last_error()

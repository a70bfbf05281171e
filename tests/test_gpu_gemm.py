"""GPU parity of the library's batched matrix-core product (sa_gemm_bf16), the
kernel under the STCA step and the layer and block gradients, on every tile
shape and operand layout, against a float64 numpy product of the same bf16
operands.

Each case is ragged (M and N one partial tile past a whole one) with a batch of
two, K = 192 (three slabs; 64 for the one-slab shapes).  fp32 results: max
|C - ref| <= 2e-5 max |ref| (fp32 accumulation of exact bf16 x bf16 products).  bf16 results: |C - ref| <= 2^-8 |ref| +
2e-5 max |ref| per element (one rounding to bf16)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# (rows, columns, one 64-deep slab only): the library's tile shapes in order
SHAPES = [(160, 256, False), (128, 256, False), (256, 128, False), (128, 128, False), (64, 128, False),
          (128, 64, False), (64, 64, False), (160, 256, True), (128, 128, True), (128, 64, True), (64, 64, True)]


@pytest.fixture(scope="module")
def sa():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_08443_amd import sa_sketch
    sa_sketch.lib()
    return sa_sketch


def operands(seed, M, N, K, batch, a_kc, b_kc, b_mod):
    g = torch.Generator().manual_seed(seed)
    zb = b_mod if b_mod > 0 else batch
    a = torch.randn((batch, M, K), generator=g).to(torch.bfloat16)   # A[z](m, k)
    b = torch.randn((zb, K, N), generator=g).to(torch.bfloat16)      # B[z](k, n)
    if a_kc:
        a_dev, a_str = a.contiguous().cuda(), (M * K, K, 1)
    else:
        a_dev, a_str = a.transpose(1, 2).contiguous().cuda(), (M * K, 1, M)
    if b_kc:
        b_dev, b_str = b.transpose(1, 2).contiguous().cuda(), (N * K, 1, K)
    else:
        b_dev, b_str = b.contiguous().cuda(), (N * K, N, 1)
    return a, b, a_dev, a_str, b_dev, b_str


def reference(a, b, batch, b_mod, alpha, c0):
    A = a.double().numpy()
    B = b.double().numpy()
    out = np.stack([A[z] @ B[z % b_mod if b_mod > 0 else z] for z in range(batch)]) * alpha
    return out + c0 if c0 is not None else out


def check(c, ref, c_bf16):
    got = c.float().cpu().double().numpy()
    scale = np.abs(ref).max()
    err = np.abs(got - ref)
    if c_bf16:
        assert np.all(err <= 2.0 ** -8 * np.abs(ref) + 2e-5 * scale), err.max()
    else:
        assert err.max() <= 2e-5 * scale, (err.max(), scale)


@pytest.mark.parametrize("shape", range(len(SHAPES)))
@pytest.mark.parametrize("a_kc,b_kc", [(True, True), (True, False), (False, True), (False, False)])
@pytest.mark.parametrize("c_bf16", [False, True])
def test_tile_shape_matches_numpy(sa, shape, a_kc, b_kc, c_bf16):
    assert sa.gemm_tile_shapes() == len(SHAPES)
    bm, bn, one = SHAPES[shape]
    M, N, K, batch = bm + 24, bn + 40, 64 if one else 192, 2
    print(f"gemm shape {shape} ({bm}x{bn}) a_kc={a_kc} b_kc={b_kc} c_bf16={c_bf16}", flush=True)
    a, b, a_dev, a_str, b_dev, b_str = operands(100 + shape, M, N, K, batch, a_kc, b_kc, 0)
    c = torch.zeros((batch, M, N), dtype=torch.bfloat16 if c_bf16 else torch.float32, device="cuda")
    if bm == 160 and not a_kc:
        # 160 rows do not split into whole loads of an m-contiguous operand
        with pytest.raises(sa.SAError):
            sa.gemm_bf16(a_dev, a_str, b_dev, b_str, c, (M * N, N), M, N, K, batch, tile_shape=shape)
        return
    sa.gemm_bf16(a_dev, a_str, b_dev, b_str, c, (M * N, N), M, N, K, batch, alpha=0.5, tile_shape=shape)
    torch.cuda.synchronize()
    check(c, reference(a, b, batch, 0, 0.5, None), c_bf16)


@pytest.mark.parametrize("shape", range(len(SHAPES)))
@pytest.mark.parametrize("c_bf16", [False, True])
def test_accumulate_shared_weights_single_slab(sa, shape, c_bf16):
    """C += alpha A B with B shared by the batch (b_mod = 1) and one 64-deep slab."""
    bm, bn, _ = SHAPES[shape]
    M, N, K, batch = 2 * bm - 8, bn + 8, 64, 3
    print(f"gemm accumulate shape {shape} M={M} N={N} K={K} c_bf16={c_bf16}", flush=True)
    a, b, a_dev, a_str, b_dev, b_str = operands(200 + shape, M, N, K, batch, True, shape % 2 == 0, 1)
    g = torch.Generator().manual_seed(300 + shape)
    c0 = torch.randn((batch, M, N), generator=g)
    if c_bf16:
        c0 = c0.to(torch.bfloat16)
    c = c0.cuda()
    sa.gemm_bf16(a_dev, a_str, b_dev, b_str, c, (M * N, N), M, N, K, batch, alpha=-1.5, accumulate=True,
                 b_mod=1, tile_shape=shape)
    torch.cuda.synchronize()
    check(c, reference(a, b, batch, 1, -1.5, c0.double().numpy()), c_bf16)


def test_automatic_choice_and_fallback(sa):
    """tile_shape = -1: the library's own choice, on a product that fills the chip
    and on one whose contraction length (100) the matrix cores do not take."""
    for (M, N, K, batch) in ((640, 512, 256, 8), (640, 1024, 64, 4), (72, 40, 100, 2)):
        print(f"gemm automatic M={M} N={N} K={K} batch={batch}", flush=True)
        a, b, a_dev, a_str, b_dev, b_str = operands(7 + K, M, N, K, batch, True, False, 0)
        c = torch.zeros((batch, M, N), dtype=torch.float32, device="cuda")
        sa.gemm_bf16(a_dev, a_str, b_dev, b_str, c, (M * N, N), M, N, K, batch)
        torch.cuda.synchronize()
        check(c, reference(a, b, batch, 0, 1.0, None), False)
    with pytest.raises(sa.SAError):   # a forced shape needs K a multiple of 64
        sa.gemm_bf16(a_dev, a_str, b_dev, b_str, c, (M * N, N), M, N, K, batch, tile_shape=3)

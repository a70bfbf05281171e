// Batched dense products on the matrix cores:
//
//   C[z](m, n) = alpha sum_k A[z](m, k) B[z](k, n)   (+ C[z](m, n) when accumulating)
//
// with A[z](m, k) = A[z a_z + m a_m + k a_k], B[z](k, n) = B[z b_z + k b_k + n b_n],
// C[z](m, n) = C[z c_z + m c_m + n].  Each operand is contiguous either along k
// (a_k = 1, b_k = 1) or along its other index (a_m = 1, b_n = 1), so transposed
// operands cost nothing at the call site.
//
// Tile 128 x 128 x 64 per workgroup of four waves, each wave a 64 x 64 block of
// 2 x 2 v_mfma_f32_32x32x16_bf16 tiles.  Both operands are staged in LDS as
// [row][64 k] bf16 (16-byte chunks XOR-swizzled so that operand reads of 32
// rows are conflict free) in two buffers; global loads run two k slabs ahead
// through two register sets, so a load has two slabs of products to land.  A
// k-contiguous tile is loaded as 16-byte row pieces; an m- (n-) contiguous tile
// as 4 k rows x 8 columns per thread, transposed in registers into 8 column
// pieces of 4 k values (written so that each store instruction meets every
// LDS bank twice, its minimum).  Tiles of one batch run on one XCD so that its operands share that
// L2.  An fp32 operand (allowed when the caller accepts bf16 rounding of its
// inputs) is loaded as the same pieces of fp32 values and rounded to bf16 when
// its slab is staged.  Products whose shapes or strides do not fit (k not a
// multiple of 64, unaligned strides, fp32 operands without that permission) run
// on the register-tiled fp32 product of layer.hip.
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

using namespace tile;

constexpr int GBM = 128, GBN = 128, GBK = 64;

struct MgArgs {
    const void* A;
    int64_t a_z, a_m, a_k;
    const void* B;
    int64_t b_z, b_k, b_n, b_mod;
    void* C;
    int64_t c_z, c_m;
    int32_t M, N, K, tm, tn;
    float alpha;
    int32_t accumulate;
};

// One thread's share of a [128 rows][64 k] slab: four 16-byte pieces of 8 bf16,
// named so that they stay in registers.
struct Slab {
    uint4 p0, p1, p2, p3;
};
// The same share of an fp32 operand: each piece as two 16-byte halves.
struct Slab32 {
    uint4 p0a, p0b, p1a, p1b, p2a, p2b, p3a, p3b;
};

__device__ inline uint4 round8(const uint4& a, const uint4& b) {
    return make_uint4(pack_bf16x2(__uint_as_float(a.x), __uint_as_float(a.y)),
                      pack_bf16x2(__uint_as_float(a.z), __uint_as_float(a.w)),
                      pack_bf16x2(__uint_as_float(b.x), __uint_as_float(b.y)),
                      pack_bf16x2(__uint_as_float(b.z), __uint_as_float(b.w)));
}
__device__ inline Slab cook(const Slab& s) { return s; }
__device__ inline Slab cook(const Slab32& s) {
    return Slab{round8(s.p0a, s.p0b), round8(s.p1a, s.p1b), round8(s.p2a, s.p2b), round8(s.p3a, s.p3b)};
}

// Per-thread sources of the four pieces of an operand's slabs: element (row, k)
// sits at base[row s_row + k s_k].  KC: s_k = 1 (rows are k runs), piece i is
// row (tid + 256 i) / 8, 16-byte chunk tid % 8; rows at or past nrows read row
// nrows - 1.  Otherwise s_row = 1: piece i is k row 4 (tid % 16) + i, columns
// 8 (tid / 16) .. + 7 (nrows is a multiple of 8; columns past it read zeros).
// Slab kt is the pieces at offset kt * step.
template <typename T>
struct Src {
    const T *p0, *p1, *p2, *p3;
    int64_t step;
    bool ok;
};

template <bool KC, typename T>
__device__ inline Src<T> make_src(const T* base, int64_t s_row, int64_t s_k, int row0, int nrows, int tid) {
    Src<T> s;
    if constexpr (KC) {
        const T* b = base + 8 * (tid & 7);
        auto at = [&](int i) {
            const int row = row0 + ((tid + 256 * i) >> 3);
            return b + (int64_t)(row < nrows ? row : nrows - 1) * s_row;
        };
        s.p0 = at(0);
        s.p1 = at(1);
        s.p2 = at(2);
        s.p3 = at(3);
        s.step = GBK;
        s.ok = true;
    } else {
        const int row = row0 + 8 * (tid >> 4);
        s.ok = row < nrows;
        s.p0 = base + (int64_t)(4 * (tid & 15)) * s_k + (s.ok ? row : 0);
        s.p1 = s.p0 + s_k;
        s.p2 = s.p1 + s_k;
        s.p3 = s.p2 + s_k;
        s.step = GBK * s_k;
    }
    return s;
}

__device__ inline Slab load_slab(const Src<uint16_t>& s, int kt) {
    const int64_t o = kt * s.step;
    Slab r;
    if (s.ok) {
        r.p0 = *reinterpret_cast<const uint4*>(s.p0 + o);
        r.p1 = *reinterpret_cast<const uint4*>(s.p1 + o);
        r.p2 = *reinterpret_cast<const uint4*>(s.p2 + o);
        r.p3 = *reinterpret_cast<const uint4*>(s.p3 + o);
    } else {
        r.p0 = r.p1 = r.p2 = r.p3 = make_uint4(0, 0, 0, 0);
    }
    return r;
}
__device__ inline Slab32 load_slab(const Src<float>& s, int kt) {
    const int64_t o = kt * s.step;
    Slab32 r;
    if (s.ok) {
        r.p0a = *reinterpret_cast<const uint4*>(s.p0 + o);
        r.p0b = *reinterpret_cast<const uint4*>(s.p0 + o + 4);
        r.p1a = *reinterpret_cast<const uint4*>(s.p1 + o);
        r.p1b = *reinterpret_cast<const uint4*>(s.p1 + o + 4);
        r.p2a = *reinterpret_cast<const uint4*>(s.p2 + o);
        r.p2b = *reinterpret_cast<const uint4*>(s.p2 + o + 4);
        r.p3a = *reinterpret_cast<const uint4*>(s.p3 + o);
        r.p3b = *reinterpret_cast<const uint4*>(s.p3 + o + 4);
    } else {
        r.p0a = r.p0b = r.p1a = r.p1b = r.p2a = r.p2b = r.p3a = r.p3b = make_uint4(0, 0, 0, 0);
    }
    return r;
}

// registers -> LDS slab [128 rows][64 k], swizzled (layout swz<64>)
template <bool KC>
__device__ inline void store_slab(uint16_t* lds, const Slab& s, int tid) {
    if constexpr (KC) {
        const int kc = tid & 7;
        *reinterpret_cast<uint4*>(lds + swz<64>(tid >> 3, kc)) = s.p0;
        *reinterpret_cast<uint4*>(lds + swz<64>((tid + 256) >> 3, kc)) = s.p1;
        *reinterpret_cast<uint4*>(lds + swz<64>((tid + 512) >> 3, kc)) = s.p2;
        *reinterpret_cast<uint4*>(lds + swz<64>((tid + 768) >> 3, kc)) = s.p3;
    } else {
        // piece i holds columns 8 mb .. 8 mb + 7 of k row 4 kb + i; column j gets the
        // thread's four k values as one 8-byte piece.  The 16 k groups of a
        // half-wave cover every chunk of a row, and the upper half-wave writes
        // columns in the order j ^ 1 (rows of the other parity), so each write
        // instruction spreads over all 64 banks.
        const int kb = tid & 15, mb = tid >> 4, flip = (tid >> 5) & 1;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int sh = 16 * ((j & 1) ^ flip);   // column j ^ flip: same dword, other half
            auto el = [&](const uint4& v) {
                const uint32_t w = (j >> 1) == 0 ? v.x : (j >> 1) == 1 ? v.y : (j >> 1) == 2 ? v.z : v.w;
                return (w >> sh) & 0xffffu;
            };
            const uint32_t lo = el(s.p0) | (el(s.p1) << 16);
            const uint32_t hi = el(s.p2) | (el(s.p3) << 16);
            *reinterpret_cast<uint2*>(lds + swz<64>(8 * mb + (j ^ flip), kb >> 1) + 4 * (kb & 1)) =
                make_uint2(lo, hi);
        }
    }
}

template <bool A_KC, bool B_KC, bool C_BF16, typename TA, typename TB>
__global__ __launch_bounds__(256, 2) void mfma_gemm_kernel(MgArgs g) {
    __shared__ __attribute__((aligned(16))) uint16_t As[2][GBM * GBK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][GBN * GBK];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hl = lane >> 5;
    const int64_t tiles = (int64_t)g.tm * g.tn;
    const int64_t id = xcd_range(blockIdx.x, gridDim.x);
    const int64_t z = id / tiles;
    const int tt = (int)(id % tiles);
    const int m0 = (tt / g.tn) * GBM, n0 = (tt % g.tn) * GBN;
    const TA* Ab = reinterpret_cast<const TA*>(g.A) + z * g.a_z;
    const TB* Bb = reinterpret_cast<const TB*>(g.B) + (g.b_mod > 0 ? z % g.b_mod : z) * g.b_z;
    const int nk = g.K / GBK;
    const Src<TA> sa_ = make_src<A_KC>(Ab, g.a_m, g.a_k, m0, g.M, tid);
    const Src<TB> sb_ = make_src<B_KC>(Bb, g.b_n, g.b_k, n0, g.N, tid);
    auto lda = [&](int kt) { return load_slab(sa_, kt); };
    auto ldb = [&](int kt) { return load_slab(sb_, kt); };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const int wm = w & 1, wn = w >> 1;
    auto mul = [&](int buf) __attribute__((always_inline)) {
        const uint16_t* Ac = As[buf];
        const uint16_t* Bc = Bs[buf];
#pragma unroll
        for (int ks = 0; ks < GBK / 16; ++ks) {
            const bf16x8 a0 = lds_b128(Ac, swz<64>(wm * 64 + l32, 2 * ks + hl));
            const bf16x8 a1 = lds_b128(Ac, swz<64>(wm * 64 + 32 + l32, 2 * ks + hl));
            const bf16x8 b0 = lds_b128(Bc, swz<64>(wn * 64 + l32, 2 * ks + hl));
            const bf16x8 b1 = lds_b128(Bc, swz<64>(wn * 64 + 32 + l32, 2 * ks + hl));
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        }
    };
    // Slab kt + 1 waits in registers while slab kt is multiplied out of LDS buffer
    // kt % 2 and slab kt + 2 is loaded: a load has two slabs of products to land.
    // The buffer a slab is stored into was last read before the previous barrier;
    // the barriers wait for LDS traffic only, so the loads stay in flight.
    auto an = lda(0);
    auto bn = ldb(0);
    store_slab<A_KC>(As[0], cook(an), tid);
    store_slab<B_KC>(Bs[0], cook(bn), tid);
    if (nk > 1) {
        an = lda(1);
        bn = ldb(1);
    }
    lds_barrier();
#pragma unroll 2
    for (int kt = 0; kt < nk; ++kt) {
        decltype(an) af;
        decltype(bn) bf;
        if (kt + 2 < nk) {
            af = lda(kt + 2);
            bf = ldb(kt + 2);
        }
        mul(kt & 1);
        if (kt + 1 < nk) {
            store_slab<A_KC>(As[(kt + 1) & 1], cook(an), tid);
            store_slab<B_KC>(Bs[(kt + 1) & 1], cook(bn), tid);
        }
        lds_barrier();
        an = af;
        bn = bf;
    }

    // C layout of a 32 x 32 tile: lane = column, register r = row srow(r, hl)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = n0 + wn * 64 + 32 * j + l32;
            if (n >= g.N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wm * 64 + 32 * i + srow(r, hl);
                if (m >= g.M) continue;
                const int64_t o = z * g.c_z + (int64_t)m * g.c_m + n;
                float v = g.alpha * acc[i][j][r];
                if constexpr (C_BF16) {
                    uint16_t* Cp = reinterpret_cast<uint16_t*>(g.C);
                    if (g.accumulate) v += __uint_as_float((uint32_t)Cp[o] << 16);
                    Cp[o] = to_bf16(v);
                } else {
                    float* Cp = reinterpret_cast<float*>(g.C);
                    if (g.accumulate) v += Cp[o];
                    Cp[o] = v;
                }
            }
        }
}

template <bool A_KC, bool B_KC, typename TA, typename TB>
hipError_t mgemm_launch_t(const MgArgs& g, bool c_bf16, int64_t batch, hipStream_t stream) {
    const int64_t blocks = (int64_t)g.tm * g.tn * batch;
    if (c_bf16)
        hipLaunchKernelGGL((mfma_gemm_kernel<A_KC, B_KC, true, TA, TB>), dim3((unsigned)blocks), dim3(256), 0, stream,
                           g);
    else
        hipLaunchKernelGGL((mfma_gemm_kernel<A_KC, B_KC, false, TA, TB>), dim3((unsigned)blocks), dim3(256), 0,
                           stream, g);
    return hipGetLastError();
}

template <bool A_KC, bool B_KC>
hipError_t mgemm_launch(const MgArgs& g, bool a_bf16, bool b_bf16, bool c_bf16, int64_t batch, hipStream_t stream) {
    if (a_bf16 && b_bf16) return mgemm_launch_t<A_KC, B_KC, uint16_t, uint16_t>(g, c_bf16, batch, stream);
    if (a_bf16) return mgemm_launch_t<A_KC, B_KC, uint16_t, float>(g, c_bf16, batch, stream);
    if (b_bf16) return mgemm_launch_t<A_KC, B_KC, float, uint16_t>(g, c_bf16, batch, stream);
    return mgemm_launch_t<A_KC, B_KC, float, float>(g, c_bf16, batch, stream);
}

bool al8(int64_t v) { return v % 8 == 0; }
bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

bool gemm_on_matrix_cores(const GemmDesc& d) {
    if (!(d.a_bf16 || d.round_bf16) || !(d.b_bf16 || d.round_bf16)) return false;
    if (d.K <= 0 || d.K % GBK != 0 || d.M <= 0 || d.N <= 0 || d.b_mod < 0) return false;
    const bool a_kc = d.a_k == 1, b_kc = d.b_k == 1;
    if (!a_kc && d.a_m != 1) return false;
    if (!b_kc && d.b_n != 1) return false;
    // 16-byte pieces: every stride and base on 8 bf16
    if (!al16(d.A) || !al16(d.B) || !al8(d.a_z) || !al8(d.b_z)) return false;
    if (!al8(a_kc ? d.a_m : d.a_k) || !al8(b_kc ? d.b_n : d.b_k)) return false;
    if (!a_kc && d.M % 8 != 0) return false;
    if (!b_kc && d.N % 8 != 0) return false;
    const int64_t blocks = (int64_t)((d.M + GBM - 1) / GBM) * ((d.N + GBN - 1) / GBN) * d.batch;
    return blocks < (int64_t(1) << 31);
}

hipError_t launch_gemm(const GemmDesc& d, hipStream_t stream) {
    if (d.batch <= 0 || d.M <= 0 || d.N <= 0) return hipSuccess;
    if (!gemm_on_matrix_cores(d)) return launch_small_gemm_general(d, stream);
    MgArgs g;
    g.A = d.A;
    g.a_z = d.a_z; g.a_m = d.a_m; g.a_k = d.a_k;
    g.B = d.B;
    g.b_z = d.b_z; g.b_k = d.b_k; g.b_n = d.b_n; g.b_mod = d.b_mod;
    g.C = d.C;
    g.c_z = d.c_z; g.c_m = d.c_m;
    g.M = d.M; g.N = d.N; g.K = d.K;
    g.tm = (d.M + GBM - 1) / GBM;
    g.tn = (d.N + GBN - 1) / GBN;
    g.alpha = d.alpha;
    g.accumulate = d.accumulate ? 1 : 0;
    const bool a_kc = d.a_k == 1, b_kc = d.b_k == 1;
    if (a_kc && b_kc) return mgemm_launch<true, true>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
    if (a_kc) return mgemm_launch<true, false>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
    if (b_kc) return mgemm_launch<false, true>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
    return mgemm_launch<false, false>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
}

}  // namespace sa

// Batched dense products on the matrix cores:
//
//   C[z](m, n) = alpha sum_k A[z](m, k) B[z](k, n)   (+ C[z](m, n) when accumulating)
//
// with A[z](m, k) = A[z a_z + m a_m + k a_k], B[z](k, n) = B[z b_z + k b_k + n b_n],
// C[z](m, n) = C[z c_z + m c_m + n].  Each operand is contiguous either along k
// (a_k = 1, b_k = 1) or along its other index (a_m = 1, b_n = 1), so transposed
// operands cost nothing at the call site.
//
// Two kernels.  Products with bf16 operands run mfma_gemm_lt_kernel (tile shape
// chosen per product, operands loaded straight into LDS; see below).  Products
// with an fp32 operand the caller allows rounding to bf16 run mfma_gemm_kernel:
// tile 128 x 128 x 64 per workgroup of four waves, each wave a 64 x 64 block of
// 2 x 2 v_mfma_f32_32x32x16_bf16 tiles; both operands staged in LDS as [row][64 k]
// bf16 (16-byte chunks XOR-swizzled so that operand reads of 32 rows are conflict
// free) in two buffers, global loads running two k slabs ahead through two
// register sets; a k-contiguous tile loaded as 16-byte row pieces, an m- (n-)
// contiguous tile as 4 k rows x 8 columns per thread transposed in registers into
// 8 column pieces of 4 k values (written so that each store instruction meets
// every LDS bank twice, its minimum); fp32 pieces rounded to bf16 as the slab is
// staged.  In both, the tiles of one batch run on one XCD so that its operands
// share that L2.  Products whose shapes or strides do not fit (k not a multiple of
// 64, unaligned strides, fp32 operands without that permission) run on the
// register-tiled fp32 product of layer.hip.
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
    int32_t c_rows16;   // N, c_m, c_z multiples of 8 and C 16-byte aligned
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

// ---------------------------------------------------------------------------
// Tiles for bf16 operands: BM x BN = (32 FM PM) x (32 FN PN) per workgroup of four
// waves in a PM x PN grid, each wave FM x FN v_mfma_f32_32x32x16_bf16 tiles; as many
// workgroups per CU as the shape's LDS and registers allow.  Three LDS stages of
// one 64-deep k slab each, loaded two slabs ahead (one stage for one-slab
// products).  Both operands go straight from global memory into LDS by direct
// loads (global_load_lds, lane l of a load writing the 16-byte chunk that belongs
// at LDS position l), so they take neither registers nor LDS store instructions:
// a k-contiguous operand into a swizzled [rows][64 k] layout read with
// ds_read_b128, an m- (n-) contiguous one as it lies in memory, [64 k][R], read
// with the transposing ds_read_b64_tr_b16.  Every slab issues the same number of
// loads per thread ((BM + BN) / 32: rows and columns past the matrix read its
// last ones), so the wait for slab kt + 1 at the end of slab kt is a fixed count
// and the loads of slab kt + 2 stay in flight across the barrier.  Results pass
// through a wave-private LDS area so that a lane stores 8 consecutive outputs.
template <int FM, int FN, int PM, int PN, int NS_ = 3>
struct LtCfg {
    static constexpr int BM = 32 * FM * PM, BN = 32 * FN * PN;
    static constexpr int A_BYTES = BM * GBK * 2, B_BYTES = BN * GBK * 2;
    // NS = 3: three stages, loaded two slabs ahead; NS = 1: one slab (K = 64), so
    // that several workgroups share a CU and one's loads overlap another's stores
    static constexpr int NS = NS_, STAGE = A_BYTES + B_BYTES;
    static constexpr int STAGING = 4 * 32 * (32 * FN + 8) * 4;   // the epilogue's areas
    static constexpr int LDS = NS * STAGE > STAGING ? NS * STAGE : STAGING;
    static constexpr int LOADS = (BM + BN) / 32;
    // workgroups per CU that the LDS and (estimated) registers allow
    static constexpr int REGS = 16 * FM * FN + 8 * (FM + FN) + 32;
    static constexpr int OCC_LDS = (160 * 1024) / LDS, OCC_REG = 512 / REGS;
    static constexpr int OCC1 = OCC_LDS < OCC_REG ? OCC_LDS : OCC_REG;
    static constexpr int OCC = OCC1 > 4 ? 4 : (OCC1 < 1 ? 1 : OCC1);
    static_assert(NS == 1 || NS == 3, "stages");
    static_assert(PM * PN == 4, "four waves");
    static_assert(LDS <= 160 * 1024, "LDS");
    static_assert(LOADS < 64, "vmcnt range");
};

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4) from
// base + off (base wave-uniform) to LDS bytes [lds + 16 lane, + 16), written as
// inline assembly: the compiler cannot tell which LDS bytes such a load writes,
// so for the builtin it makes the transposing LDS reads wait for every load in
// flight, the next slabs' included.  Completion is awaited by the explicit
// vmcnt waits of lt_barrier (and the vmcnt(0) before the epilogue).
// M0 (which holds the load's LDS address) is a reserved register, so the block
// saves and restores it instead of declaring it clobbered.
__device__ __forceinline__ void lt_dma16(const char* base, uint32_t off, const uint8_t* lds) {
    const uint32_t l = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)lds;
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(off), "s"(base), "s"(l)
        : "memory");
}

template <int N>
__device__ __forceinline__ void lt_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

template <int R, bool KC>
struct LtOperand;

// k-contiguous operand, R rows: load q = w + 4 i (i < R / 32) of a slab fills LDS
// rows 8 q .. 8 q + 7; lane l takes row 8 q + l / 8 and the chunk whose swizzled
// position is l % 8.  Offsets are 32-bit byte offsets from the batch's base.
template <int R>
struct LtOperand<R, true> {
    static constexpr int Q = R / 32;
    const char* base;
    int64_t step;   // bytes from one slab to the next
    uint32_t off[Q];
    __device__ __forceinline__ void init(const uint16_t* b, int64_t s_row, int64_t /*s_k*/, int row0, int nrows,
                                         int w, int lane) {
        base = reinterpret_cast<const char*>(b);
        step = GBK * 2;
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            const int row = 8 * (w + 4 * i) + (lane >> 3);
            const int c = (lane & 7) ^ swz_x<64>(row);
            const int gr = min(row0 + row, nrows - 1);
            off[i] = (uint32_t)(((int64_t)gr * s_row + 8 * c) * 2);
        }
    }
    __device__ __forceinline__ void issue(int kt, uint8_t* lds, int w) {
        const char* p = base + kt * step;
#pragma unroll
        for (int i = 0; i < Q; ++i) lt_dma16(p, off[i], lds + (w + 4 * i) * 1024);
    }
};

// 16-byte chunk swizzle of an m- (n-) contiguous slab ([64 k][R] bf16, LPR = R / 8
// chunks per row): the eight k rows one transposing read touches (64 bytes of rows
// k0 + 0..3 and k0 + 8..11) fall in four different 64-byte windows of the 256
// bytes of banks instead of one.  Rows of 256 bytes or more start on the same
// bank, so row k moves by (k mod 4) windows; 128-byte rows alternate between the
// two halves, so row k moves by one window when bit 1 of k is set.  Measured: 8%
// less time on a product with both operands transposed, 2% on one.
__device__ __forceinline__ int tr_swizzle(int k, int lpr) {
    return lpr >= 16 ? (k & 3) << 2 : ((k >> 1) & 1) << 2;
}

// m- (n-) contiguous operand: the slab is kept as it lies in memory, [64 k][R] (rows
// of R bf16), its 16-byte chunks permuted within each row by tr_swizzle.  Lane l of
// load q = w + 4 i fills LDS chunk p = 64 q + l, at row k = p / LPR and position
// p mod LPR, with the global chunk at that position XOR tr_swizzle(k) (columns
// past the matrix read its last eight).  Its fragments are read with the
// transposing ds_read_b64_tr_b16 (lt_frag).
template <int R>
struct LtOperand<R, false> {
    static_assert(R % 64 == 0 && R <= 512, "transposed operand tile");   // LPR >= 8
    static constexpr int Q = R / 32, LPR = R / 8;   // loads per thread, lanes per row
    static_assert(64 % LPR == 0, "whole rows per load");
    static constexpr int RPL = 64 / LPR;            // rows per load
    const char* base;
    int64_t step;
    uint32_t off[Q];
    __device__ __forceinline__ void init(const uint16_t* b, int64_t /*s_row*/, int64_t s_k, int row0, int nrows,
                                         int w, int lane) {
        base = reinterpret_cast<const char*>(b);
        step = GBK * s_k * 2;
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            const int idx = (w + 4 * i) * 64 + lane;        // chunk index in the slab
            const int k = idx / LPR, col = min(row0 + 8 * ((idx % LPR) ^ tr_swizzle(k, LPR)), nrows - 8);
            off[i] = (uint32_t)(((int64_t)k * s_k + col) * 2);
        }
    }
    __device__ __forceinline__ void issue(int kt, uint8_t* lds, int w) {
        const char* p = base + kt * step;
#pragma unroll
        for (int i = 0; i < Q; ++i) lt_dma16(p, off[i], lds + (w + 4 * i) * 1024);
    }
};

// fragment (32 rows or columns from `first`, k step ks) of an operand slab in LDS:
// k-contiguous: ds_read_b128 of the swizzled rows; otherwise two transposing
// reads: inside each 16-lane group, lane i receives element i % 4 of the 8-byte
// pieces addressed by lanes 4 e + i / 4 (e < 4), so lane 4 e + j addresses k row
// e (then e + 4) and columns 4 j .. 4 j + 3 of its group's 16 columns.
template <int R, bool KC>
__device__ __forceinline__ bf16x8 lt_frag(const uint8_t* lds, int first, int ks, int lane) {
    const int l32 = lane & 31, hl = lane >> 5;
    if constexpr (KC) {
        return lds_b128(reinterpret_cast<const uint16_t*>(lds), swz<64>(first + l32, 2 * ks + hl));
    } else {
        typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
        const int s = lane & 15, g = (lane >> 4) & 1;
        const int k = 16 * ks + 8 * hl + (s >> 2), col = first + 16 * g + 4 * (s & 3);
        typedef __attribute__((address_space(3))) short lds_short;
        constexpr int LPR = R / 8;
        lds_short* base = (lds_short*)(const_cast<uint8_t*>(lds));
        lds_short* p = base + k * R + 8 * ((col >> 3) ^ tr_swizzle(k, LPR)) + (col & 7);
        lds_short* q = base + (k + 4) * R + 8 * ((col >> 3) ^ tr_swizzle(k + 4, LPR)) + (col & 7);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)q);
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
}

template <int FM, int FN, int PM, int PN, bool A_KC, bool B_KC, bool C_BF16, int NS>
__global__ __launch_bounds__(256, (LtCfg<FM, FN, PM, PN, NS>::OCC)) void mfma_gemm_lt_kernel(MgArgs g) {
    using C = LtCfg<FM, FN, PM, PN, NS>;
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];
    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hl = lane >> 5;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t tiles = (int64_t)g.tm * g.tn;
    const int64_t id = xcd_range(blockIdx.x, gridDim.x);
    const int64_t z = id / tiles;
    const int tt = (int)(id % tiles);
    const int m0 = (tt / g.tn) * C::BM, n0 = (tt % g.tn) * C::BN;
    const uint16_t* Ab = reinterpret_cast<const uint16_t*>(g.A) + z * g.a_z;
    const uint16_t* Bb = reinterpret_cast<const uint16_t*>(g.B) + (g.b_mod > 0 ? z % g.b_mod : z) * g.b_z;
    const int nk = g.K / GBK;
    LtOperand<C::BM, A_KC> opa;
    LtOperand<C::BN, B_KC> opb;
    opa.init(Ab, g.a_m, g.a_k, m0, g.M, w, lane);
    opb.init(Bb, g.b_n, g.b_k, n0, g.N, w, lane);
    auto stage = [&](int s) { return smem + (s % C::NS) * C::STAGE; };
    // slab kt into the stage of slab position pos
    auto issue = [&](int kt, int pos) __attribute__((always_inline)) {
        uint8_t* st = stage(pos);
        opa.issue(kt, st, w);
        opb.issue(kt, st + C::A_BYTES, w);
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const int wm = w % PM, wn = w / PM;
    // operand reads of step ks + 1 are issued before the products of step ks
    auto mul = [&](int kt) __attribute__((always_inline)) {
        const uint8_t* As = stage(kt);
        const uint8_t* Bs = stage(kt) + C::A_BYTES;
        bf16x8 a[2][FM], b[2][FN];
        auto rd = [&](int ks, bf16x8 (&ao)[FM], bf16x8 (&bo)[FN]) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < FM; ++i) ao[i] = lt_frag<C::BM, A_KC>(As, 32 * (FM * wm + i), ks, lane);
#pragma unroll
            for (int j = 0; j < FN; ++j) bo[j] = lt_frag<C::BN, B_KC>(Bs, 32 * (FN * wn + j), ks, lane);
        };
        rd(0, a[0], b[0]);
#pragma unroll
        for (int ks = 0; ks < GBK / 16; ++ks) {
            if (ks + 1 < GBK / 16) rd(ks + 1, a[(ks + 1) & 1], b[(ks + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of the products
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks & 1][i], b[ks & 1][j], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // slab kt: slab kt + 2 is loaded, slab kt is multiplied, slab kt + 1's loads are
    // awaited (the loads of slab kt + 2, if any, stay in flight)
    if constexpr (C::NS == 1) {   // the host launches it for K = 64 only
        issue(0, 0);
        lt_barrier<0>();
        mul(0);
    } else {
        issue(0, 0);
        if (nk > 1) issue(1, 1);
        if (nk > 1) lt_barrier<C::LOADS>();
        else lt_barrier<0>();
        for (int kt = 0; kt < nk; ++kt) {
            const bool ahead = kt + 2 < nk;
            if (ahead) issue(kt + 2, kt + 2);
            mul(kt);
            if (ahead) lt_barrier<C::LOADS>();
            else if (kt + 1 < nk) lt_barrier<0>();
        }
    }

    // Epilogue.  With 16-byte aligned rows of C, each wave passes its results
    // through its own LDS area ([32 rows][32 FN + 8] fp32, one row of tiles at a
    // time) so that a lane stores 8 consecutive outputs; otherwise one element per
    // lane and register.
    const bool rows16 = g.c_rows16 != 0;
    __syncthreads();   // every wave is done with the operand stages
    constexpr int P = 32 * FN + 8, LPR = 4 * FN, RPP = 64 / LPR;
    float* stg = reinterpret_cast<float*>(smem) + w * 32 * P;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int mt = m0 + 32 * (FM * wm + i);
        if (rows16) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) stg[srow(r, hl) * P + 32 * j + l32] = g.alpha * acc[i][j][r];
            wave_lds_order();
#pragma unroll
            for (int ps = 0; ps < 32 / RPP; ++ps) {
                const int rr = ps * RPP + lane / LPR, cc = 8 * (lane % LPR);
                const float4 v0 = *reinterpret_cast<const float4*>(stg + rr * P + cc);
                const float4 v1 = *reinterpret_cast<const float4*>(stg + rr * P + cc + 4);
                const int m = mt + rr, n = n0 + 32 * FN * wn + cc;
                if (m < g.M && n < g.N) {
                    const int64_t o = z * g.c_z + (int64_t)m * g.c_m + n;
                    float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
                    if constexpr (C_BF16) {
                        uint4* Cp = reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(g.C) + o);
                        if (g.accumulate) {
                            const uint4 c = *Cp;
                            const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
                            for (int e = 0; e < 8; ++e)
                                v[e] += __uint_as_float((e & 1) ? (cw[e >> 1] & 0xffff0000u) : (cw[e >> 1] << 16));
                        }
                        *Cp = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                                         pack_bf16x2(v[6], v[7]));
                    } else {
                        float4* Cp = reinterpret_cast<float4*>(reinterpret_cast<float*>(g.C) + o);
                        if (g.accumulate) {
                            const float4 c0 = Cp[0], c1 = Cp[1];
                            v[0] += c0.x; v[1] += c0.y; v[2] += c0.z; v[3] += c0.w;
                            v[4] += c1.x; v[5] += c1.y; v[6] += c1.z; v[7] += c1.w;
                        }
                        Cp[0] = make_float4(v[0], v[1], v[2], v[3]);
                        Cp[1] = make_float4(v[4], v[5], v[6], v[7]);
                    }
                }
            }
            wave_lds_order();
        } else {
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int n = n0 + 32 * (FN * wn + j) + l32;
                if (n >= g.N) continue;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = mt + srow(r, hl);
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
    }
}

template <int FM, int FN, int PM, int PN, int NS, bool A_KC, bool B_KC>
hipError_t lt_launch(MgArgs g, bool c_bf16, int64_t batch, hipStream_t stream) {
    using C = LtCfg<FM, FN, PM, PN, NS>;
    g.tm = (g.M + C::BM - 1) / C::BM;
    g.tn = (g.N + C::BN - 1) / C::BN;
    const int64_t blocks = (int64_t)g.tm * g.tn * batch;
    if (c_bf16)
        hipLaunchKernelGGL((mfma_gemm_lt_kernel<FM, FN, PM, PN, A_KC, B_KC, true, NS>), dim3((unsigned)blocks),
                           dim3(256), 0, stream, g);
    else
        hipLaunchKernelGGL((mfma_gemm_lt_kernel<FM, FN, PM, PN, A_KC, B_KC, false, NS>), dim3((unsigned)blocks),
                           dim3(256), 0, stream, g);
    return hipGetLastError();
}

template <int FM, int FN, int PM, int PN, int NS>
hipError_t lt_dispatch(const MgArgs& g, bool a_kc, bool b_kc, bool c_bf16, int64_t batch, hipStream_t stream) {
    if (a_kc && b_kc) return lt_launch<FM, FN, PM, PN, NS, true, true>(g, c_bf16, batch, stream);
    if (a_kc) return lt_launch<FM, FN, PM, PN, NS, true, false>(g, c_bf16, batch, stream);
    if constexpr (LtCfg<FM, FN, PM, PN, NS>::BM % 64 == 0) {
        if (b_kc) return lt_launch<FM, FN, PM, PN, NS, false, true>(g, c_bf16, batch, stream);
        return lt_launch<FM, FN, PM, PN, NS, false, false>(g, c_bf16, batch, stream);
    }
    return hipErrorInvalidValue;
}

// Tile shapes: rows, columns, relative speed per tile element (fewer LDS and L2
// bytes per product for bigger tiles), workgroups per CU, whether the A operand
// may be m-contiguous (160 rows do not split into whole loads of rows), and
// whether the shape is a one-slab (K = 64) variant.
struct LtShape {
    int bm, bn;
    double eff;
    int occ;
    bool a_mc_ok;
    bool one_slab;   // K = 64 only
};
constexpr LtShape kLtShapes[] = {
    {160, 256, 1.0, 1, false, false}, {128, 256, 0.85, 1, true, false}, {256, 128, 0.85, 1, true, false},
    {128, 128, 0.7, 1, true, false},  {64, 128, 0.55, 2, true, false},  {128, 64, 0.6, 2, true, false},
    {64, 64, 0.62, 3, true, false},   {160, 256, 1.0, 2, false, true},  {128, 128, 0.7, 4, true, true},
    {128, 64, 0.6, 4, true, true},    {64, 64, 0.5, 4, true, true}};

// The per-lane load offsets of an operand are 32-bit byte offsets from the slab's
// base: a k-contiguous operand's reach over its rows and K, an m- (n-)
// contiguous one's over one slab's 64 k rows and its columns.
bool lt_offsets_fit(const GemmDesc& d, bool a_kc, bool b_kc) {
    auto fits = [&](bool kc, int64_t rows, int64_t s_row, int64_t s_k) {
        const int64_t reach = kc ? (rows - 1) * s_row + d.K : (GBK - 1) * s_k + rows;
        return reach * 2 < (int64_t(1) << 32);
    };
    return fits(a_kc, d.M, d.a_m, d.a_k) && fits(b_kc, d.N, d.b_n, d.b_k);
}

// The shape with the least estimated time: rounds of `occ` tiles per compute unit,
// each round the tile's work over its speed times the tiles that share a CU (two
// resident workgroups split its matrix cores); small tiles win where big ones
// leave compute units idle.  -1 if none applies (byte offsets of a k-contiguous
// operand beyond 32 bits).
int choose_lt(const GemmDesc& d, bool a_kc, bool b_kc) {
    if (!lt_offsets_fit(d, a_kc, b_kc)) return -1;
    const int64_t cus = device_cus();
    int best = -1;
    double best_cost = 0;
    for (int i = 0; i < (int)(sizeof(kLtShapes) / sizeof(kLtShapes[0])); ++i) {
        const LtShape& t = kLtShapes[i];
        // one-slab products take the one-slab shapes (same tiles, more of them per CU)
        if ((!a_kc && !t.a_mc_ok) || t.one_slab != (d.K == GBK)) continue;
        const int64_t tiles = (int64_t)((d.M + t.bm - 1) / t.bm) * ((d.N + t.bn - 1) / t.bn) * d.batch;
        if (tiles >= (int64_t(1) << 31)) continue;
        const int64_t rounds = (tiles + cus * t.occ - 1) / (cus * t.occ);
        const int64_t share = std::min<int64_t>(t.occ, (tiles + cus - 1) / cus);
        const double cost = (double)rounds * share * t.bm * t.bn / t.eff;
        if (best < 0 || cost < best_cost) {
            best = i;
            best_cost = cost;
        }
    }
    return best;
}

hipError_t lt_run(int shape, const MgArgs& g, bool a_kc, bool b_kc, bool c_bf16, int64_t batch,
                  hipStream_t stream) {
    switch (shape) {
        case 0: return lt_dispatch<5, 2, 1, 4, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 1: return lt_dispatch<4, 2, 1, 4, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 2: return lt_dispatch<4, 2, 2, 2, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 3: return lt_dispatch<2, 2, 2, 2, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 4: return lt_dispatch<1, 2, 2, 2, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 5: return lt_dispatch<2, 1, 2, 2, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 6: return lt_dispatch<1, 1, 2, 2, 3>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 7: return lt_dispatch<5, 2, 1, 4, 1>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 8: return lt_dispatch<2, 2, 2, 2, 1>(g, a_kc, b_kc, c_bf16, batch, stream);
        case 9: return lt_dispatch<2, 1, 2, 2, 1>(g, a_kc, b_kc, c_bf16, batch, stream);
        default: return lt_dispatch<1, 1, 2, 2, 1>(g, a_kc, b_kc, c_bf16, batch, stream);
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

namespace {

MgArgs make_args(const GemmDesc& d) {
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
    g.c_rows16 = (d.N % 8 == 0 && d.c_m % 8 == 0 && d.c_z % 8 == 0 && al16(d.C)) ? 1 : 0;
    return g;
}

}  // namespace

hipError_t launch_gemm(const GemmDesc& d, hipStream_t stream) {
    if (d.batch <= 0 || d.M <= 0 || d.N <= 0) return hipSuccess;
    if (!gemm_on_matrix_cores(d)) return launch_small_gemm_general(d, stream);
    const MgArgs g = make_args(d);
    const bool a_kc = d.a_k == 1, b_kc = d.b_k == 1;
    if (d.a_bf16 && d.b_bf16) {
        const int shape = choose_lt(d, a_kc, b_kc);
        if (shape >= 0) return lt_run(shape, g, a_kc, b_kc, d.c_bf16, d.batch, stream);
    }
    if (a_kc && b_kc) return mgemm_launch<true, true>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
    if (a_kc) return mgemm_launch<true, false>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
    if (b_kc) return mgemm_launch<false, true>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
    return mgemm_launch<false, false>(g, d.a_bf16, d.b_bf16, d.c_bf16, d.batch, stream);
}

int gemm_tile_shapes() { return (int)(sizeof(kLtShapes) / sizeof(kLtShapes[0])); }

hipError_t launch_gemm_tile_shape(const GemmDesc& d, int shape, hipStream_t stream) {
    if (shape < 0) return launch_gemm(d, stream);
    if (shape >= gemm_tile_shapes() || !d.a_bf16 || !d.b_bf16 || !gemm_on_matrix_cores(d))
        return hipErrorInvalidValue;
    const bool a_kc = d.a_k == 1, b_kc = d.b_k == 1;
    const LtShape& t = kLtShapes[shape];
    if ((!a_kc && !t.a_mc_ok) || (t.one_slab && d.K != GBK) || !lt_offsets_fit(d, a_kc, b_kc))
        return hipErrorInvalidValue;
    if ((int64_t)((d.M + t.bm - 1) / t.bm) * ((d.N + t.bn - 1) / t.bn) * d.batch >= (int64_t(1) << 31))
        return hipErrorInvalidValue;
    if (d.batch <= 0 || d.M <= 0 || d.N <= 0) return hipSuccess;
    return lt_run(shape, make_args(d), a_kc, b_kc, d.c_bf16, d.batch, stream);
}

}  // namespace sa

// Backward of the SA sketching step on gfx950 matrix cores (bf16 inputs,
// fp32 gradients).
//
// Chain rule of the forward (section 3.1: S = scale K P^T, A = softmax over
// prototypes, sketch = A^T V), with the MRLB sum of section 4.2 done first
// (dY = sum over the R target instances that reuse a user's sketch):
//
//   A[t,m]  = exp(scale * S[t,m] - lse[t])        (recomputed from the saved lse)
//   dV_t    = sum_m A[t,m] dY_m
//   D_t     = sum_m A[t,m] <V_t, dY_m>  =  <V_t, dV_t>
//   dS[t,m] = A[t,m] (<V_t, dY_m> - D_t)
//   dK_t    = scale sum_m dS[t,m] P_m
//   dP_m    = scale sum_t dS[t,m] K_t             (over every user and token)
//
// Three device passes:
//   prep   dY (fp32, R summed) -> bf16 in two layouts; P -> bf16 transposed.
//   token  per token tile: dV (first sweep over the prototypes), D_t = <V_t, dV_t>,
//          then dK (second sweep).  Works in the transposed orientation S^T (rows =
//          prototypes, lanes = tokens) so that the reductions over prototypes are
//          matrix-core contractions whose k slots are the register index of S^T.
//          Prototype blocks of 32 are streamed through LDS and shared by the
//          waves (each wave owns 32 tokens).  For M <= 512 the first sweep's
//          weights are held in registers for the second (bwd_token_held_kernel,
//          four waves); otherwise the second sweep recomputes them
//          (bwd_token_kernel, eight waves).
//   proto  dP for a slice of the prototypes, in the forward's orientation (lanes =
//          prototypes): the prototype slice and the user's dY slice stay in LDS
//          (or in registers with one 32-prototype tile per wave), dS^T . K
//          accumulates in registers with K^T read by the transposing LDS load;
//          one partial per work-list segment, summed per head in segment order
//          (deterministic).
#include <type_traits>
#include <utility>

#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

using namespace tile;

// A wave raises its issue priority for the length of a matrix-core chain and
// drops it for its exponential / elementwise phase, so that the two waves of a
// SIMD drift into opposite phases (one feeds the matrix core while the other
// runs VALU and LDS work) instead of contending for the same unit in lockstep.
// The changes take registers of the chain as operands, which orders the raise
// before the chain's first MFMA and the drop after its results.
__device__ inline void prio_up(const bf16x8& a) { asm volatile("s_setprio 1" :: "v"(a)); }
__device__ inline void prio_down(f32x16& a) { asm volatile("s_setprio 0" : "+v"(a)); }

// Scheduling groups (sched_group_barrier masks: 0x008 MFMA, 0x002 VALU, 0x100
// LDS read).  N copies of {one MFMA, R LDS reads, V VALU instructions}: the
// MFMAs of one chain alternate with the independent VALU work of the previous
// block, and the operand reads run ahead of the MFMAs that take them.
template <int N, int R, int V>
__device__ inline void sched_mfma_ds_valu() {
    if constexpr (N > 0) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (R > 0) __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
        if constexpr (V > 0) __builtin_amdgcn_sched_group_barrier(0x002, V, 0);
        sched_mfma_ds_valu<N - 1, R, V>();
    }
}
template <int R>
__device__ inline void sched_ds() {
    __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
}

__device__ inline float xhalf_sum(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// f(integral_constant<int, I>) for I = 0 .. N-1, each I a compile-time constant
// (so that arrays indexed by it stay in registers)
template <typename F, int... I>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// s_waitcnt for vector memory only: at most N of this wave's vector-memory
// operations still outstanding (the other counters are not waited for)
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// A workgroup barrier after at most N outstanding vector-memory operations and
// none of LDS.  The wait is the compiler's own instruction, so it knows that
// every earlier LDS read has landed (an inline-assembly wait would leave it
// waiting again, after the barrier, behind newer reads); the scheduling fences
// keep each side's instructions on its side.
template <int N>
__device__ __forceinline__ void stage_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Token blocks of a token-side workgroup: segment k of the work list (user b,
// head h, tokens up to t1) and its tokens [tb, te); the blocks of a segment
// start at its first token.
struct TokBlk {
    int64_t k;
    int b, h, t1, tb, te;
};
template <int TB>
struct TokSeq {
    const int32_t* items;
    int64_t k1, T;
    int B, H;
    // the first block of the first valid segment at or after k
    __device__ bool first_from(int64_t k, TokBlk& o) const {
        // the item list is read through the constant address space, so that
        // these wave-uniform reads are scalar loads (no vector-memory wait)
        typedef const __attribute__((address_space(4))) int32_t cint;
        for (; k < k1; ++k) {
            cint* it = (cint*)items + k * IT_WORDS;
            const int b = it[IT_B], h = it[IT_H], t0 = it[IT_T0], t1 = it[IT_T1];
            if (b < 0 || b >= B || h < 0 || h >= H || t0 < 0 || t1 <= t0 || t1 > T) continue;
            o.k = k; o.b = b; o.h = h; o.t1 = t1; o.tb = t0;
            o.te = t0 + TB < t1 ? t0 + TB : t1;
            return true;
        }
        return false;
    }
    // the block `steps` blocks after c
    __device__ bool advance(TokBlk c, int64_t steps, TokBlk& o) const {
        while (true) {
            const int64_t left = (c.t1 - c.tb + TB - 1) / TB;   // c and the blocks after it
            if (steps < left) {
                o = c;
                o.tb = c.tb + (int)steps * TB;
                o.te = o.tb + TB < c.t1 ? o.tb + TB : c.t1;
                return true;
            }
            steps -= left;
            if (!first_from(c.k + 1, c)) return false;
        }
    }
};

typedef float f32x4 __attribute__((ext_vector_type(4)));

// A 16-byte LDS store written as inline assembly.  The compiler orders every
// LDS access it knows of behind all outstanding direct global->LDS loads (it
// cannot tell their target areas apart), which would drain the prototype-block
// stream before each row-staging store; callers of this store keep it to an
// area no direct load writes, and order its later reads with lgkmcnt.
__device__ __forceinline__ void lds_store16_asm(float* p, f32x4 v) {
    const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float*)p;
    asm volatile("ds_write_b128 %0, %1" ::"v"(a), "v"(v) : "memory");
}
// Four 16-byte LDS loads at p + q * stride bytes (q < 4), in one inline-assembly
// block that waits for them, for the same reason.
__device__ __forceinline__ void lds_load16x4_asm(f32x4 (&o)[4], const float* p, int stride) {
    const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)p;
    asm volatile(
        "ds_read_b128 %0, %4\n"
        "ds_read_b128 %1, %4 offset:%5\n"
        "ds_read_b128 %2, %4 offset:%6\n"
        "ds_read_b128 %3, %4 offset:%7\n"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3])
        : "v"(a), "i"(stride), "i"(2 * stride), "i"(3 * stride)
        : "memory");
}

// f * acc (a wave's 32 tokens tok0 + 0..31, lane = token, rows j = 32 jt +
// srow(r, hl)) into the rows of out [T, H, D], only tokens below te.  The C
// layout holds 16-byte pieces of 32 token rows per store; each 32-column slice
// goes through the wave's LDS area stg ([32][ROWF] fp32) so that every store
// instruction writes whole 128-byte lines of 8 tokens.
//
// CLAMP: lanes past te store to row te - 1 instead of being masked off, so that
// every wave issues the same number of store instructions; only for callers
// whose lanes past the end computed exactly the last token's values (their
// inputs are copies of its rows), and never with add.
template <int D, int ROWF, bool CLAMP = false>
__device__ __forceinline__ void store_token_rows(const f32x16 (&acc)[D / 32], float* stg, float* out, float f,
                                                 int tok0, int te, int H, int h, bool add, int lane) {
    const int l32 = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int jt = 0; jt < D / 32; ++jt) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
            lds_store16_asm(stg + l32 * ROWF + 8 * g + 4 * hl,
                            (f32x4){f * acc[jt][4 * g], f * acc[jt][4 * g + 1], f * acc[jt][4 * g + 2],
                                    f * acc[jt][4 * g + 3]});
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's own area
        f32x4 rows[4];
        lds_load16x4_asm(rows, stg + (lane >> 3) * ROWF + 4 * (lane & 7), 8 * ROWF * 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int t = 8 * q + (lane >> 3), cc = 4 * (lane & 7);
            const float4 v = make_float4(rows[q][0], rows[q][1], rows[q][2], rows[q][3]);
            const int tk = CLAMP ? min(tok0 + t, te - 1) : tok0 + t;
            if (CLAMP || tk < te) {
                float4* o = reinterpret_cast<float4*>(out + ((int64_t)tk * H + h) * D + jt * 32 + cc);
                if (!CLAMP && add) {
                    const float4 u = *o;
                    *o = make_float4(u.x + v.x, u.y + v.y, u.z + v.z, u.w + v.w);
                } else {
                    *o = v;
                }
            }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // reads done before the next slice
    }
}

// D_t = <V_t, dV_t> for the lane's token.  The lane holds dV[t, j] for j = 32 jt +
// 8 g + 4 hl + e (e < 4, C layout of dV^T) and V[t, j] for j = 16 kk + 8 hl +
// 0..7 (B operand layout).  Swapping dwords 0-1 of the upper half with dwords
// 2-3 of the lower half gives both halves V at j = 16 kk + 4 hl + 0..3 (dwords
// 0-1) and 16 kk + 8 + 4 hl + 0..3 (dwords 2-3): with kk = 2 jt + g / 2, the
// columns of dV registers 4 g .. 4 g + 3.  Each half holds half the sum.
template <int D>
__device__ __forceinline__ float dot_v_dv(const bf16x8 (&vb)[D / 16], const f32x16 (&dvt)[D / 32]) {
    float Dt = 0.f;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
        const u32x4 v = __builtin_bit_cast(u32x4, vb[kk]);
        const auto p0 = __builtin_amdgcn_permlane32_swap(v[0], v[2], false, false);
        const auto p1 = __builtin_amdgcn_permlane32_swap(v[1], v[3], false, false);
        const uint32_t q[2][2] = {{p0[0], p1[0]}, {p0[1], p1[1]}};
#pragma unroll
        for (int sh = 0; sh < 2; ++sh) {
            const int jt = kk >> 1, g = 2 * (kk & 1) + sh;
            Dt = __builtin_fmaf(bf16_lo(q[sh][0]), dvt[jt][4 * g + 0], Dt);
            Dt = __builtin_fmaf(bf16_hi(q[sh][0]), dvt[jt][4 * g + 1], Dt);
            Dt = __builtin_fmaf(bf16_lo(q[sh][1]), dvt[jt][4 * g + 2], Dt);
            Dt = __builtin_fmaf(bf16_hi(q[sh][1]), dvt[jt][4 * g + 3], Dt);
        }
    }
    return Dt;
}

// ------------------------------------------------------------------ prep
// dY[b,h] = sum_r dsketch[b,r,h] (fp32) written as bf16 row-major Ymj[b,h,m,j]
// and transposed Yjm[b,h,j,p] with p = perm16(m); P -> Pjm[h,j,p] likewise.
// One workgroup per 32-prototype block: the rows are summed and converted with
// 16-byte accesses, staged in LDS, and the transposed block is written as 64-byte
// rows.  Workgroups [0, B*H*M/32) take dY blocks, the next n_p*M/32 take P blocks
// (n_p = H shared prototype blocks, or B*H with one block per user and head).
template <int D>
__global__ __launch_bounds__(256) void prep_kernel(const float* __restrict__ ds, int64_t B, int32_t R,
                                                   int32_t H, int32_t M, int64_t n_p,
                                                   const uint16_t* __restrict__ P,
                                                   uint16_t* __restrict__ Ymj,
                                                   uint16_t* __restrict__ Yjm,
                                                   uint16_t* __restrict__ Pjm) {
    constexpr int KCH = D / 8;                       // 16-byte bf16 chunks per row
    constexpr int NCH = 32 * KCH;                    // chunks per block
    __shared__ __attribute__((aligned(16))) uint16_t tile[32 * D];
    const int tid = threadIdx.x;
    const int64_t MD = (int64_t)M * D;
    const int64_t nb = M / 32;
    const int64_t blk = blockIdx.x;
    const bool is_y = blk < B * H * nb;
    const int64_t pair = is_y ? blk / nb : (blk - B * H * nb) / nb;   // b*H + h, or h
    const int mb = (int)((is_y ? blk : blk - B * H * nb) % nb);
    if (!is_y && pair >= n_p) return;
    uint16_t* rowdst = is_y ? Ymj + pair * MD : nullptr;
    uint16_t* trdst = (is_y ? Yjm : Pjm) + pair * MD;
    // (unrolled so that the loads of both chunks and several targets are in flight)
#pragma unroll
    for (int i = tid; i < NCH; i += 256) {
        const int r = i / KCH, c = i % KCH;
        const int64_t off = (int64_t)(mb * 32 + r) * D + c * 8;
        u32x4 v;
        if (is_y) {
            const int64_t b = pair / H, h = pair % H;
            float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
            for (int rr = 0; rr < R; ++rr) {
                const float4* src = reinterpret_cast<const float4*>(ds + ((b * R + rr) * H + h) * MD + off);
                const float4 x0 = src[0], x1 = src[1];
                acc[0] += x0.x; acc[1] += x0.y; acc[2] += x0.z; acc[3] += x0.w;
                acc[4] += x1.x; acc[5] += x1.y; acc[6] += x1.z; acc[7] += x1.w;
            }
            v = (u32x4){pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                        pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7])};
            *reinterpret_cast<u32x4*>(rowdst + off) = v;
        } else {
            v = *reinterpret_cast<const u32x4*>(P + pair * MD + off);
        }
        *reinterpret_cast<u32x4*>(tile + r * D + c * 8) = v;
    }
    __syncthreads();
    // transposed: row j, columns p = 0..31 of this block, p = perm16(m)
    for (int i = tid; i < NCH; i += 256) {
        const int j = i / 4, c = i % 4;
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int m0 = perm16(8 * c + 2 * e), m1 = perm16(8 * c + 2 * e + 1);
            w[e] = (uint32_t)tile[m0 * D + j] | ((uint32_t)tile[m1 * D + j] << 16);
        }
        *reinterpret_cast<u32x4*>(trdst + (int64_t)j * M + mb * 32 + c * 8) = (u32x4){w[0], w[1], w[2], w[3]};
    }
}

// ------------------------------------------------------------------ token side
constexpr int kTokWaves = 8;   // waves of the token-side kernel: two per SIMD

template <int D, int NW_>
struct TokCfg {
    static constexpr int NW = NW_;
    static constexpr int THREADS = NW * 64;
    static constexpr int TB = 32 * NW;                 // tokens per block (32 per wave)
    static constexpr int KS = D / 16;
    static constexpr int JT = D / 32;
    static constexpr int KCH = D / 8;                  // 16-byte chunks per row
    static constexpr int BLK = 32 * D;                 // bf16 elements of one 32-row block
    // LDS: three stages of {Pmj, Pjm, Ymj, Yjm} prototype blocks (block mb + 1 is
    // resident while mb is consumed and mb + 2 is in flight)
    static constexpr int BUF = 4 * BLK;
    static constexpr int STAGES = 3;
    // per wave: one [32 tokens][32 columns] fp32 slice of an output, rows padded
    static constexpr int ROWF = 36;
    static constexpr int STG_FLOATS = 32 * ROWF;
    static constexpr int OFF_STG = STAGES * BUF * 2;   // bytes
    static constexpr int LDS = OFF_STG + NW * STG_FLOATS * 4;
    static constexpr int CHUNKS = BLK / 8;             // 16-byte chunks of one block
};

struct TokArgs {
    const uint16_t* K;
    const uint16_t* V;
    const uint16_t* P;
    const uint16_t* Pjm;
    const uint16_t* Ymj;
    const uint16_t* Yjm;
    const float* lse;
    const int32_t* items;
    const int32_t* wg_start;
    int64_t max_items;
    int64_t T;
    int32_t B, H, M;
    float scale;
    float* dK;
    float* dV;
    float* dX;      // XV: dX = dV + dK (K and V are the same tensor X)
    float* Dbuf;
    bool p_user;    // P, Pjm hold one block per (user, head)
    bool dx_add;    // XV: add to dX instead of overwriting it
};

// XV: K and V are one tensor X (the SA layer aggregates its own history and its
// key projection is folded into P).  X is loaded once, and the second sweep keeps
// accumulating into the dV registers with scale folded into dS, so the kernel
// writes dX = dV + dK once.
template <int D, int NW, bool XV>
__global__ __launch_bounds__(NW * 64, 8 / NW) void bwd_token_kernel(TokArgs a) {
    using C = TokCfg<D, NW>;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int l32 = lane & 31, hl = lane >> 5;
    float* stg = reinterpret_cast<float*>(smem + C::OFF_STG) + w * C::STG_FLOATS;

    // The workgroups of one XCD take the token blocks of that XCD's ranges in
    // turn (workgroup i of the XCD: blocks i, i + nx, i + 2 nx, ...), so that at
    // any time they work on neighbouring blocks, mostly of one (user, head),
    // whose prototype-block stream then stays in that XCD's L2.
    const int64_t nr = gridDim.x, xq = nr / 8, xrem = nr % 8, xcd = blockIdx.x % 8;
    const int64_t lw = blockIdx.x / 8, nx = xq + (xcd < xrem ? 1 : 0);
    const int64_t first_range = xcd * xq + (xcd < xrem ? xcd : xrem);
    const int64_t k0 = a.wg_start[first_range], k1 = a.wg_start[first_range + nx];
    if (k0 < 0 || k1 < k0 || k1 > a.max_items) return;
    const float ks2 = a.scale * kLog2e;
    const int nblk = a.M / 32;   // >= 4
    const int64_t MD = (int64_t)a.M * D;

    using Blk = TokBlk;
    const TokSeq<C::TB> seq{a.items, k1, a.T, a.B, a.H};
    auto next_of = [&](const Blk& c, Blk& o) -> bool { return seq.advance(c, nx, o); };

    // K as B operands (lane (hl, t) holds 8 consecutive j of its token) and the
    // lane's lse, for block c.  Lanes past the block's end take its last token
    // (finite weights in columns that are never stored), so the loads carry no
    // predicate, and nothing is computed from them here: they stay in flight
    // until their first use.
    bf16x8 kb[C::KS], vb[C::KS];
    float lse_t = 0.f;
    auto load_k = [&](const Blk& c) __attribute__((always_inline)) {
        const int tok = min(c.tb + 32 * w + l32, c.te - 1);
        const int64_t row = ((int64_t)tok * a.H + c.h) * D;
#pragma unroll
        for (int kk = 0; kk < C::KS; ++kk)
            kb[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(a.K + row + 16 * kk + 8 * hl));
        lse_t = a.lse[(int64_t)tok * a.H + c.h];
    };

    // Prototype block mb of the matrices a sweep reads, straight into LDS buffer
    // `buf` (sweep 0: Pmj, Yjm; sweep 1: Pmj, Pjm, Ymj).  Lane l of a wave fetches
    // the global chunk that belongs at LDS chunk position p = 64 q + l of the
    // swizzled layout (the XOR swizzle is its own inverse).
    auto fetch = [&](const Blk& c, int mb, int sweep, int buf) __attribute__((always_inline)) {
        const int64_t pkey = a.p_user ? (int64_t)c.b * a.H + c.h : c.h;
        const uint16_t* Pmj_g = a.P + pkey * MD;
        const uint16_t* Pjm_g = a.Pjm + pkey * MD;
        const uint16_t* Ymj_g = a.Ymj + ((int64_t)c.b * a.H + c.h) * MD;
        const uint16_t* Yjm_g = a.Yjm + ((int64_t)c.b * a.H + c.h) * MD;
        uint16_t* L = lds + buf * C::BUF;
        constexpr int NQ = C::CHUNKS / 64;   // wave-loads per matrix block
        for (int q = w; q < NQ; q += NW) {
            const int p = q * 64 + lane;
            {   // row-major [32 prototypes][D]: Pmj, and Ymj in sweep 1
                const int r = p / C::KCH, cc = (p % C::KCH) ^ swz_x<D>(r);
                const int64_t src = (int64_t)(mb * 32 + r) * D + cc * 8;
                load_lds16(Pmj_g + src, L + q * 512);
                if (sweep == 1) load_lds16(Ymj_g + src, L + 2 * C::BLK + q * 512);
            }
            {   // [D][32 prototypes], prototype index permuted: Yjm or Pjm
                const int j = p / 4, cc = (p % 4) ^ swz_x<32>(j);
                const int64_t srcj = (int64_t)j * a.M + mb * 32 + cc * 8;
                load_lds16((sweep == 1 ? Pjm_g : Yjm_g) + srcj, L + (sweep == 1 ? C::BLK : 3 * C::BLK) + q * 512);
            }
        }
    };
    // S^T tile of a prototype block (rows = its 32 prototypes, cols = tokens)
    auto st_tile = [&](const uint16_t* L) {
        f32x16 s;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
        for (int kk = 0; kk < C::KS; ++kk)
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(L, swz<D>(l32, 2 * kk + hl)), kb[kk], s, 0, 0, 0);
        return s;
    };
    auto store_rows = [&](const f32x16 (&acc)[C::JT], float* out, float f, int tb, int te, int h, bool add)
        __attribute__((always_inline)) {
        store_token_rows<D, C::ROWF>(acc, stg, out, f, tb + 32 * w, te, a.H, h, add, lane);
    };

    Blk cur;
    if (!seq.first_from(k0, cur) || !seq.advance(cur, lw, cur)) return;
    load_k(cur);
    fetch(cur, 0, 0, 0);
    fetch(cur, 1, 0, 1);
    wait_vmem();
    __syncthreads();

    // Per block: a stream of 2 nblk stages (sweep 1's prototype blocks, then sweep
    // 2's) through three LDS buffers, continued from block to block: the next
    // block's first two stages are fetched during the last two stages of this one,
    // so that at the block's entry its K and stages 0 and 1 (buffers ring and
    // ring + 1) are resident.  The V rows (sweep 1's last stage) and the next
    // block's K (sweep 2's last stage) are loaded beside a stage's compute too:
    // each stage ends by waiting for every load it issued.
    auto inc3 = [](int x) { return x == 2 ? 0 : x + 1; };
    int ring = 0;
    while (true) {
        const int tb = cur.tb, te = cur.te, h = cur.h;
        const int tok = tb + 32 * w + l32;   // this lane's token (column of S^T)
        const bool tv = tok < te;
        const float nl = -lse_t * kLog2e;
        Blk nxt;
        const bool more = next_of(cur, nxt);

        // ---------------- sweep 1: dV^T[j, t] = sum_m dY[m, j] A[t, m]
        // The S^T tile of block mb + 1 is issued before the exponentials of block
        // mb, so the matrix core works through them while the VALU runs; the
        // scheduling groups interleave the two instruction streams.
        f32x16 dvt[C::JT];
#pragma unroll
        for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
            for (int r = 0; r < 16; ++r) dvt[jt][r] = 0.f;
        f32x16 s_next = st_tile(lds + ring * C::BUF);
        auto s1_stage = [&](int mb, int bc) __attribute__((always_inline)) {
            const int bn = inc3(bc), bnn = inc3(bn);
            const uint16_t* L = lds + bc * C::BUF;
            if (mb + 2 < nblk) fetch(cur, mb + 2, 0, bnn);
            else fetch(cur, mb + 2 - nblk, 1, bnn);
            const f32x16 s = s_next;
            s_next = st_tile(lds + (mb + 1 < nblk ? bn : bc) * C::BUF);   // last block: unused
            float e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], ks2, nl));
            const bf16x8 ab0 = pack8(e), ab1 = pack8(e + 8);
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt) {
                const uint16_t* Y = L + 3 * C::BLK;
                dvt[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Y, swz<32>(jt * 32 + l32, 0 + hl)), ab0, dvt[jt], 0, 0, 0);
                dvt[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Y, swz<32>(jt * 32 + l32, 2 + hl)), ab1, dvt[jt], 0, 0, 0);
            }
            // S^T(mb + 1) with the exponentials of mb, then dV(mb)
            sched_ds<2>();
            sched_mfma_ds_valu<C::KS, 1, 40 / C::KS>();
            sched_mfma_ds_valu<2 * C::JT, 1, 0>();
            wait_vmem();   // stage mb + 2 has landed in LDS
            __syncthreads();
        };
        int bc1 = ring;
        for (int mb = 0; mb + 1 < nblk; ++mb, bc1 = inc3(bc1)) s1_stage(mb, bc1);
        if constexpr (!XV) {
            // V of this wave's tokens (for D_t and sweep 2), in flight during the
            // last stage
            const int64_t row = ((int64_t)min(tok, te - 1) * a.H + h) * D;
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk)
                vb[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(a.V + row + 16 * kk + 8 * hl));
        }
        s1_stage(nblk - 1, bc1);
        if constexpr (XV) {
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) vb[kk] = kb[kk];
        }
        // D_t = <V_t, dV_t>
        float Dt = dot_v_dv<D>(vb, dvt);
        Dt = tv ? xhalf_sum(Dt) : 0.f;
        if (tv && hl == 0) a.Dbuf[(int64_t)tok * a.H + h] = Dt;
        // dV rows now (frees their registers); they drain under sweep 2's first stage
        if constexpr (!XV) store_rows(dvt, a.dV, 1.0f, tb, te, h, false);

        // ---------------- sweep 2: dK^T[j, t] = scale sum_m P[m, j] dS[t, m]
        // (XV: continues from dV^T, with scale folded into the weights)
        f32x16 dkt[C::JT];
#pragma unroll
        for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
            for (int r = 0; r < 16; ++r) dkt[jt][r] = XV ? dvt[jt][r] : 0.f;
        const float nl2 = XV ? nl + __log2f(a.scale) : nl;
        // sweep 2's block mb is stage nblk + mb: blocks 0 and 1 are resident
        const int b0 = (ring + nblk) % 3;
        // stage mb + 2 of the stream: this sweep's, or the next block's first two
        auto fetch2 = [&](int mb, int buf) __attribute__((always_inline)) {
            if (mb + 2 < nblk) fetch(cur, mb + 2, 1, buf);
            else if (more) fetch(nxt, mb + 2 - nblk, 0, buf);
        };
        // Pipelined form: iteration mb runs the elementwise work of block mb
        // beside the S^T MFMAs of block mb + 1, then the dK MFMAs of mb beside
        // the dA MFMAs of mb + 1 (two independent chains).  It holds 16 more
        // registers than the plain form; with separate K and V operands at
        // d = 128 it fits only at the full 256 VGPRs and runs slower, so that
        // instance keeps the plain form.
        constexpr bool kPipe2 = XV || D == 64;
        auto da_tile = [&](const uint16_t* Lb) {
            f32x16 da;
#pragma unroll
            for (int r = 0; r < 16; ++r) da[r] = 0.f;
            const uint16_t* Ym = Lb + 2 * C::BLK;
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk)
                da = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Ym, swz<D>(l32, 2 * kk + hl)), vb[kk], da, 0, 0, 0);
            return da;
        };
        auto dk_acc = [&](const uint16_t* Lb, const f32x16& s, const f32x16& da) __attribute__((always_inline)) {
            float e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float A = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], ks2, nl2));
                e[r] = A * (da[r] - Dt);
            }
            const bf16x8 d0 = pack8(e), d1 = pack8(e + 8);
            const uint16_t* Pj = Lb + C::BLK;
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt) {
                dkt[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Pj, swz<32>(jt * 32 + l32, 0 + hl)), d0, dkt[jt], 0, 0, 0);
                dkt[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Pj, swz<32>(jt * 32 + l32, 2 + hl)), d1, dkt[jt], 0, 0, 0);
            }
        };
        if constexpr (kPipe2) {
            s_next = st_tile(lds + b0 * C::BUF);
            f32x16 da_next = da_tile(lds + b0 * C::BUF);
            int bc = b0;
            for (int mb = 0; mb + 1 < nblk; ++mb, bc = inc3(bc)) {
                const int bn = inc3(bc), bnn = inc3(bn);
                const uint16_t* L = lds + bc * C::BUF;
                fetch2(mb, bnn);
                const uint16_t* Ln = lds + bn * C::BUF;
                const f32x16 s = s_next, da = da_next;
                s_next = st_tile(Ln);
                dk_acc(L, s, da);
                da_next = da_tile(Ln);
                sched_ds<2>();
                sched_mfma_ds_valu<C::KS, 1, 72 / C::KS>();
                sched_mfma_ds_valu<C::KS + 2 * C::JT, 1, 0>();
                wait_vmem();
                __syncthreads();
            }
            // the last block: the next block's K goes out first (this block's S^T
            // tiles are all done)
            if (more) load_k(nxt);
            fetch2(nblk - 1, inc3(inc3(bc)));
            dk_acc(lds + bc * C::BUF, s_next, da_next);
            wait_vmem();
            __syncthreads();
        } else {
            auto s2_stage = [&](int mb, int bc, bool last) __attribute__((always_inline)) {
                const int bnn = bc == 0 ? 2 : bc - 1;   // (bc + 2) % 3
                const uint16_t* L = lds + bc * C::BUF;
                fetch2(mb, bnn);
                const f32x16 s = st_tile(L);
                // the last block: the next block's K right after its last S^T tile
                if (last && more) load_k(nxt);
                const f32x16 da = da_tile(L);
                dk_acc(L, s, da);
                wait_vmem();
                __syncthreads();
            };
            int bc = b0;
            for (int mb = 0; mb + 1 < nblk; ++mb, bc = inc3(bc)) s2_stage(mb, bc, false);
            s2_stage(nblk - 1, bc, true);
        }

        // The dK rows drain under the next block's first stage.
        store_rows(dkt, XV ? a.dX : a.dK, XV ? 1.0f : a.scale, tb, te, h, XV && a.dx_add);
        if (!more) break;
        cur = nxt;
        ring = (ring + 2 * nblk) % 3;
    }
}

// ------------------------------------------------------------------ token side, weights held
// For M <= 512 the first sweep's bf16 weights A^T of a wave's 32 tokens (M/32
// tiles of 16 values per lane, at most 128 registers) stay in registers until
// the second sweep, which then computes only dA and dK: 8
// instead of 10 M d matrix FLOPs per (token, head) and one exponential per
// (token, prototype) instead of two.  That takes one wave per SIMD (four per
// workgroup, 128 tokens per block).  The second sweep uses the weights as
// rounded to bf16 for the dV contraction (about 2^-9 relative).
//
// The prototype blocks stream through eight LDS buffers (stage s of a token
// block's 2 M/32 stages in buffer s % 8, fetched six stages ahead), so a fetch
// has four stages to land and every LDS address is a constant offset from a
// lane register: the row-major matrices of the eight buffers fill the first
// 64 KB (the reach of an instruction offset), the transposed ones the next.  A
// stage ends by waiting for the fetch of stage s + 2 only (a vector-memory
// count computed per stage: the fetches, row loads and row stores each wave
// issues are fixed in number and complete in issue order), so that the row
// loads of K and V stay in flight across five stages and no stage waits for
// the row stores.
//
// The stages are pipelined by one prototype block: stage mb contracts block
// mb - 1 (its weights and operands prepared in the previous stage) beside the
// exponentials (or dS) of block mb, then runs the S^T (or dA) chain of block
// mb + 1, reading block mb's contraction operands between the chain's steps.
template <int D, int NBLK>
struct HeldCfg {
    static constexpr int NW = 4;
    static constexpr int THREADS = NW * 64;
    static constexpr int TB = 32 * NW;                 // tokens per block
    static constexpr int KS = D / 16;
    static constexpr int JT = D / 32;
    static constexpr int KCH = D / 8;                  // 16-byte chunks per row
    static constexpr int BLK = 32 * D;                 // bf16 elements of one 32-row block
    static constexpr int NSTG = 2 * NBLK;              // stages per token block
    static constexpr int NBUF = 8;
    static constexpr int AHEAD = 6;
    static constexpr int OFF_COL = NBUF * BLK * 2;     // bytes: the transposed matrices
    static constexpr int ROWF = 36;
    static constexpr int STG_FLOATS = 32 * ROWF;
    static constexpr int OFF_STG = 2 * NBUF * BLK * 2;
    static constexpr int LDS = OFF_STG + NW * STG_FLOATS * 4;
    static constexpr int NQ = BLK / 8 / 64;            // wave-loads per matrix block
    static constexpr int FL = 2 * NQ / NW;             // fetch loads per wave per stage
    static_assert(NSTG % NBUF == 0 && NQ % NW == 0 && NSTG >= AHEAD + 2, "held-weights configuration");
    static_assert(OFF_COL <= 65536 && LDS <= 160 * 1024, "LDS layout");

    // vector-memory operations a wave issues in stage s after its fetch: the V
    // rows in stage 1 (separate K and V), the next block's K rows and lse in
    // stage NBLK + 1
    template <bool XV>
    static constexpr int extra(int s) {
        return (!XV && s == 1) ? KS : (s == NBLK + 1 ? KS + 1 : 0);
    }
    // ... and between stage s - 1's barrier and stage s's fetch: D_t and the dV
    // rows before stage NBLK, the dK (or dX) rows of the previous block before
    // stage 0
    template <bool XV>
    static constexpr int bnd(int s) {
        return s == NBLK ? 1 + (XV ? 0 : 4 * JT) : (s == 0 ? 4 * JT : 0);
    }
    // The count a wave waits down to at the end of stage s: the fetch of stage
    // s + 2, issued in stage s - 4 (of the previous block if negative), must have
    // landed; everything issued after it may stay in flight.  Vector-memory
    // operations complete in issue order (loads and stores alike), so this
    // count is exact.  (The first block's early fetches precede a full wait.)
    template <bool XV>
    static constexpr int wait_count(int s) {
        const int first = s - (AHEAD - 2);
        int n = extra<XV>((first % NSTG + NSTG) % NSTG);
        for (int x = first + 1; x <= s; ++x) {
            const int y = (x % NSTG + NSTG) % NSTG;
            n += bnd<XV>(y) + FL + extra<XV>(y);
        }
        return n;
    }
    // the stages whose window holds the previous block's row stores (their
    // count is data dependent when the rows are added to dX: full waits then)
    static constexpr bool after_rows(int s) { return s < AHEAD - 2; }
};

template <int D, int NBLK, bool XV>
__global__ __launch_bounds__(256, 1) void bwd_token_held_kernel(TokArgs a) {
    using C = HeldCfg<D, NBLK>;
    constexpr int NW = C::NW, KS = C::KS, JT = C::JT, NSTG = C::NSTG, NBUF = C::NBUF;
    // static LDS, so that buffer addresses are constants
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: LDS bases in scalar registers
    const int l32 = lane & 31, hl = lane >> 5;
    float* stg = reinterpret_cast<float*>(smem + C::OFF_STG) + w * C::STG_FLOATS;

    // block assignment as in bwd_token_kernel: the workgroups of an XCD take the
    // token blocks of that XCD's ranges in turn
    const int64_t nr = gridDim.x, xq = nr / 8, xrem = nr % 8, xcd = blockIdx.x % 8;
    const int64_t lw = blockIdx.x / 8, nx = xq + (xcd < xrem ? 1 : 0);
    const int64_t first_range = xcd * xq + (xcd < xrem ? xcd : xrem);
    const int64_t k0 = a.wg_start[first_range], k1 = a.wg_start[first_range + nx];
    if (k0 < 0 || k1 < k0 || k1 > a.max_items) return;
    const TokSeq<C::TB> seq{a.items, k1, a.T, a.B, a.H};
    const float ks2 = a.scale * kLog2e;
    const int64_t MD = (int64_t)a.M * D;

    // byte offsets inside a prototype block of the chunks this lane fetches (the
    // same for every block), added to a wave-uniform block address
    uint32_t rofs[C::NQ / NW], tofs[C::NQ / NW];
#pragma unroll
    for (int i = 0; i < C::NQ / NW; ++i) {
        const int p = (w + NW * i) * 64 + lane;
        const int r = p / C::KCH, cc = (p % C::KCH) ^ swz_x<D>(r);
        rofs[i] = (uint32_t)((r * D + cc * 8) * 2);
        const int j = p / 4, cj = (p % 4) ^ swz_x<32>(j);
        tofs[i] = (uint32_t)((j * a.M + cj * 8) * 2);
    }
    // LDS byte offsets of this lane's operand reads: chunk 2 kk + hl of row l32 of
    // a row-major block (plus buffer * BLK * 2), and the two k halves of row
    // 32 jt + l32 of a transposed block (plus OFF_COL + buffer * BLK * 2 + jt * 2048)
    uint32_t roff[KS], coff[2];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) roff[kk] = (uint32_t)swz<D>(l32, 2 * kk + hl) * 2;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        coff[c] = (uint32_t)(C::OFF_COL + swz<32>(l32, 2 * c + hl) * 2);
        asm volatile("" : "+v"(coff[c]));   // one base register, buffers as instruction offsets
    }
    auto rd = [&](uint32_t off) __attribute__((always_inline)) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(smem + off));
    };

    // Prototype block mb of the two matrices a sweep reads, straight into LDS
    // buffer b (sweep 0: P rows [32][D] and dY^T [D][32]; sweep 1: dY rows and
    // P^T).  Lane l of a wave fetches the global chunk that belongs at LDS chunk
    // position p = 64 q + l of the swizzled layout (the XOR swizzle is its own
    // inverse).  FL loads per wave.
    auto fetch = [&](const TokBlk& c, int mb, int sweep, int b) __attribute__((always_inline)) {
        const int64_t pkey = a.p_user ? (int64_t)c.b * a.H + c.h : c.h;
        const int64_t ykey = (int64_t)c.b * a.H + c.h;
        const char* Rg = reinterpret_cast<const char*>((sweep == 0 ? a.P + pkey * MD : a.Ymj + ykey * MD) + mb * 32 * D);
        const char* Tg = reinterpret_cast<const char*>((sweep == 0 ? a.Yjm + ykey * MD : a.Pjm + pkey * MD) + mb * 32);
#pragma unroll
        for (int i = 0; i < C::NQ / NW; ++i) {
            const int q = w + NW * i;
            load_lds16(Rg + rofs[i], smem + b * C::BLK * 2 + q * 1024);
            load_lds16(Tg + tofs[i], smem + C::OFF_COL + b * C::BLK * 2 + q * 1024);
        }
    };
    // stage X of the stream: this block's, the next block's stage X - NSTG, or
    // after the last block this block's stage X - NSTG again into a buffer that
    // is not read any more (so that every stage issues the same loads)
    auto fetch_stage = [&](auto xc, const TokBlk& cur, const TokBlk& nxt, bool more) __attribute__((always_inline)) {
        constexpr int X = decltype(xc)::value;
        constexpr int Y = X < NSTG ? X : X - NSTG;   // the stage within its block
        static_assert(Y < NSTG, "fetch distance");
        if constexpr (X < NSTG) fetch(cur, Y % NBLK, Y / NBLK, X % NBUF);
        else fetch(more ? nxt : cur, Y % NBLK, Y / NBLK, X % NBUF);
    };
    // rows of this wave's tokens as B operands (lane (hl, t) holds 8 consecutive
    // j of its token); lanes past the block's end take its last token, so the
    // loads carry no predicate
    auto load_rows = [&](const uint16_t* src, const TokBlk& c, bf16x8 (&dst)[KS]) __attribute__((always_inline)) {
        const int t = min(32 * w + l32, c.te - 1 - c.tb);
        const char* base = reinterpret_cast<const char*>(src + ((int64_t)c.tb * a.H + c.h) * D);
        const uint32_t off = (uint32_t)(t * a.H * D + 8 * hl) * 2;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
            dst[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(base + off + 32 * kk));
    };
    auto load_lse = [&](const TokBlk& c) __attribute__((always_inline)) {
        const int t = min(32 * w + l32, c.te - 1 - c.tb);
        const char* base = reinterpret_cast<const char*>(a.lse + (int64_t)c.tb * a.H + c.h);
        return *reinterpret_cast<const float*>(base + (uint32_t)(t * a.H) * 4);
    };
    // operands of a [32 prototypes] x [32 tokens] tile from the row-major block
    // of buffer b (P, or dY in sweep 2), and of the contraction over the block's
    // prototypes from its transposed block (dY^T, or P^T in sweep 2)
    auto row_ops = [&](int b, bf16x8 (&op)[KS]) __attribute__((always_inline)) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) op[kk] = rd(roff[kk] + b * C::BLK * 2);
    };
    auto col_ops = [&](int b, bf16x8 (&op)[2 * JT]) __attribute__((always_inline)) {
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
            for (int c = 0; c < 2; ++c) op[2 * jt + c] = rd(coff[c] + b * C::BLK * 2 + jt * 2048);
    };
    auto col_acc = [&](const bf16x8 (&op)[2 * JT], const bf16x8& w0, const bf16x8& w1, f32x16 (&acc)[JT])
        __attribute__((always_inline)) {
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
            acc[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[2 * jt], w0, acc[jt], 0, 0, 0);
            acc[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[2 * jt + 1], w1, acc[jt], 0, 0, 0);
        }
    };
    auto row_tile = [&](const bf16x8 (&op)[KS], const bf16x8 (&b)[KS]) __attribute__((always_inline)) {
        f32x16 s;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[kk], b[kk], s, 0, 0, 0);
        return s;
    };
    const bool add = XV && a.dx_add;   // dX rows read and added: masked, so counted by a full wait
    // the score (or dA) chain of the next block, one read of this block's
    // contraction operands (for the next stage) issued after each of its steps,
    // so that the reads land while the dependent chain runs
    auto chain_and_reads = [&](const bf16x8 (&op)[KS], const bf16x8 (&b)[KS], f32x16& s, int bufc,
                               bf16x8 (&cnext)[2 * JT]) __attribute__((always_inline)) {
        static_assert(2 * JT <= KS, "one read per chain step");
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[kk], b[kk], s, 0, 0, 0);
            if (kk < 2 * JT) {
                const int jt = kk >> 1, c = kk & 1;
                cnext[kk] = rd(coff[c] + bufc * C::BLK * 2 + jt * 2048);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    auto stage_end = [&](auto sc) __attribute__((always_inline)) {
        constexpr int S = decltype(sc)::value;
        if (C::after_rows(S) && add) stage_barrier<0>();
        else stage_barrier<C::template wait_count<XV>(S)>();
    };

    TokBlk cur;
    if (!seq.first_from(k0, cur) || !seq.advance(cur, lw, cur)) return;
    // kb: K rows (the score chains of sweep 1); vb: V rows (D_t and the dA chains
    // of sweep 2).  XV: kb holds X for both, and vb receives the next block's X.
    bf16x8 kb[KS], vb[KS];
    bf16x8 (&vop)[KS] = XV ? kb : vb;
    load_rows(a.K, cur, kb);
    float lse_n = load_lse(cur);
    static_for<C::AHEAD>([&](auto xc) { fetch_stage(xc, cur, cur, false); });
    wait_vmem();
    __syncthreads();
    f32x16 s_cur;
    {
        bf16x8 op[KS];
        row_ops(0, op);
        s_cur = row_tile(op, kb);
    }
    float nl = -lse_n * kLog2e;

    // The stages are software-pipelined by one prototype block: stage mb runs the
    // contraction of block mb - 1 (its weights packed and its operands read in
    // the previous stage) beside the elementwise work of block mb (whose score
    // or dA tile the previous stage computed), then the score or dA chain of
    // block mb + 1 (its operands read at the top of the stage), and reads the
    // operands of block mb's contraction for the next stage.  So every matrix
    // instruction's operands were requested a phase earlier, and the VALU work
    // runs beside independent matrix instructions.
    constexpr int RPS = 16 / (2 * JT);   // elementwise rows per contraction instruction
    while (true) {
        const int tb = cur.tb, te = cur.te, h = cur.h;
        const int tok = tb + 32 * w + l32;   // this lane's token (column of S^T)
        TokBlk nxt;
        const bool more = seq.advance(cur, nx, nxt);

        // ---------------- sweep 1: A^T tiles (held), dV^T[j, t] = sum_m dY[m, j] A[t, m]
        bf16x8 ah[NBLK][2];
        f32x16 dvt[JT];
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
            for (int r = 0; r < 16; ++r) dvt[jt][r] = 0.f;
        bf16x8 cop[2 * JT];   // contraction operands of the previous block
        static_for<NBLK>([&](auto mbc) {
            constexpr int mb = decltype(mbc)::value, S = mb, B = S % NBUF;
            fetch_stage(std::integral_constant<int, S + C::AHEAD>{}, cur, nxt, more);
            if constexpr (!XV && S == 1) load_rows(a.V, cur, vb);
            bf16x8 pop[KS];
            if constexpr (mb + 1 < NBLK) row_ops((S + 1) % NBUF, pop);
            // dV(mb - 1) beside the exponentials of block mb
            float e[16];
#pragma unroll
            for (int q = 0; q < 2 * JT; ++q) {
                if constexpr (mb > 0) {
                    const int jt = q >> 1, c = q & 1;
                    dvt[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cop[q], ah[mb - 1][c], dvt[jt], 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < RPS; ++u) {
                    const int r = q * RPS + u;
                    e[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s_cur[r], ks2, nl));
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            ah[mb][0] = pack8(e);
            ah[mb][1] = pack8(e + 8);
            // S^T chain of block mb + 1, and block mb's dV operands for the next stage
            if constexpr (mb + 1 < NBLK) chain_and_reads(pop, kb, s_cur, B, cop);
            else col_ops(B, cop);
            stage_end(std::integral_constant<int, S>{});
        });
        // sweep 2's first dA tile beside the last dV contraction
        f32x16 da_cur;
        {
            bf16x8 op[KS];
            row_ops(NBLK % NBUF, op);
            col_acc(cop, ah[NBLK - 1][0], ah[NBLK - 1][1], dvt);
            da_cur = row_tile(op, vop);
        }
        // D_t = <V_t, dV_t>; the V rows are not touched before this point
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) asm volatile("" : "+v"(vop[kk]));
        // (lanes past the block's end hold the last token's values, stored to its row)
        const float Dt = xhalf_sum(dot_v_dv<D>(vop, dvt));
        if (hl == 0) a.Dbuf[(int64_t)min(tok, te - 1) * a.H + h] = Dt;
        if constexpr (!XV)
            store_token_rows<D, C::ROWF, true>(dvt, stg, a.dV, 1.0f, tb + 32 * w, te, a.H, h, false, lane);

        // ---------------- sweep 2: dK^T[j, t] = scale sum_m P[m, j] dS[t, m] with
        // dS = A (dA - D_t) from the held A (XV: continues from dV^T, scale folded
        // into dS)
        f32x16 dkt[JT];
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
            for (int r = 0; r < 16; ++r) dkt[jt][r] = XV ? dvt[jt][r] : 0.f;
        bf16x8 dsp[2];   // dS of the previous block, packed
        static_for<NBLK>([&](auto mbc) {
            constexpr int mb = decltype(mbc)::value, S = NBLK + mb, B = S % NBUF;
            fetch_stage(std::integral_constant<int, S + C::AHEAD>{}, cur, nxt, more);
            if constexpr (S == NBLK + 1) {
                load_rows(a.K, more ? nxt : cur, XV ? vb : kb);
                lse_n = load_lse(more ? nxt : cur);
            }
            bf16x8 yop[KS];
            if constexpr (mb + 1 < NBLK) row_ops((S + 1) % NBUF, yop);
            // dK(mb - 1) beside dS of block mb
            float e[16];
#pragma unroll
            for (int q = 0; q < 2 * JT; ++q) {
                if constexpr (mb > 0) {
                    const int jt = q >> 1, c = q & 1;
                    dkt[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cop[q], dsp[c], dkt[jt], 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < RPS; ++u) {
                    const int r = q * RPS + u;
                    const float A = (float)ah[mb][r >> 3][r & 7];
                    const float g = da_cur[r] - Dt;
                    e[r] = XV ? A * (g * a.scale) : A * g;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            dsp[0] = pack8(e);
            dsp[1] = pack8(e + 8);
            // dA chain of block mb + 1, and block mb's dK operands for the next stage
            if constexpr (mb + 1 < NBLK) chain_and_reads(yop, vop, da_cur, B, cop);
            else col_ops(B, cop);
            stage_end(std::integral_constant<int, S>{});
        });

        // the next block's first S^T tile (its stage 0 has landed) beside the last
        // dK contraction, before the row stores, whose completion the next stage's
        // end waits for
        if (more) {
            if constexpr (XV) {
#pragma unroll
                for (int kk = 0; kk < KS; ++kk) kb[kk] = vb[kk];
            }
            bf16x8 op[KS];
            row_ops(0, op);
            col_acc(cop, dsp[0], dsp[1], dkt);
            s_cur = row_tile(op, kb);
            nl = -lse_n * kLog2e;
        } else {
            col_acc(cop, dsp[0], dsp[1], dkt);
        }
        if (add)
            store_token_rows<D, C::ROWF>(dkt, stg, a.dX, 1.0f, tb + 32 * w, te, a.H, h, true, lane);
        else
            store_token_rows<D, C::ROWF, true>(dkt, stg, XV ? a.dX : a.dK, XV ? 1.0f : a.scale, tb + 32 * w, te,
                                               a.H, h, false, lane);
        if (!more) break;
        cur = nxt;
    }
}

// ------------------------------------------------------------------ prototype side
template <int D, int MW, int NW_>
struct ProtoCfg {
    static constexpr int NW = NW_;
    static constexpr int THREADS = NW * 64;
    static constexpr int MP = MW * NW;      // prototypes of one part
    static constexpr int MT = MW / 32;
    static constexpr int KS = D / 16;
    static constexpr int JT = D / 32;
    static constexpr int KCH = D / 8;
    static constexpr int LD_CHUNKS = 32 * KCH;
    static constexpr int NCH = (LD_CHUNKS + THREADS - 1) / THREADS;
    // With one 32-prototype tile per wave the wave's P and dY rows are held in
    // registers for the segment (loaded from global memory); otherwise the part's
    // P and dY slices stay in LDS.
    static constexpr bool HOLD = MT == 1;
    static constexpr int SLICE = HOLD ? 0 : MP * D * 2;
    // Two waves per SIMD with one prototype tile each run phase-shifted (see the
    // kernel); their token tiles rotate through three buffers, otherwise two.
    static constexpr bool PING = NW == 8 && MT == 1;
    static constexpr int NBUF = PING ? 3 : 2;
    static constexpr int TILE = 32 * D * 2;                // one [32][D] bf16 token tile
    static constexpr int OFF_P = 0;                        // [MP][D]
    static constexpr int OFF_Y = OFF_P + SLICE;            // [MP][D]
    static constexpr int OFF_K = OFF_Y + SLICE;            // NBUF x [32][D] token-major K tiles
    static constexpr int OFF_V = OFF_K + NBUF * TILE;      // NBUF x [32][D] V tiles
    static constexpr int OFF_L = OFF_V + NBUF * TILE;      // NBUF x [32] -lse*log2e
    static constexpr int OFF_D = OFF_L + NBUF * 32 * 4;    // NBUF x [32] D_t
    static constexpr int LDS = OFF_D + NBUF * 32 * 4;
};

struct ProtoArgs {
    const uint16_t* K;
    const uint16_t* V;
    const uint16_t* P;
    const uint16_t* Ymj;
    const float* lse;
    const float* Dbuf;
    const int32_t* items;
    const int32_t* wg_start;
    int64_t max_items;
    int64_t T;
    int64_t n_ranges;
    int32_t B, H, M;
    int32_t parts;    // M / MP
    float scale;
    float* partials;  // [max_items][M][D]
    bool p_user;      // P holds one block per (user, head)
};

// XV: K and V are one tensor (one tile load serves both operands).
template <int D, int MW, int NW, bool XV>
__global__ __launch_bounds__(NW * 64, 1) void bwd_proto_kernel(ProtoArgs a) {
    using C = ProtoCfg<D, MW, NW>;
    constexpr bool kHold = C::HOLD;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* Ps = reinterpret_cast<uint16_t*>(smem + C::OFF_P);
    uint16_t* Ys = reinterpret_cast<uint16_t*>(smem + C::OFF_Y);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int l32 = lane & 31, hl = lane >> 5;

    // Workgroup -> (range, part): the XCD of workgroup L is L % 8; on each XCD the
    // parts of one range are dispatched back to back (their K and V reads share
    // that XCD's L2) and the ranges are consecutive (see xcd_range).
    const int64_t xcd = blockIdx.x % 8, jx = blockIdx.x / 8;
    const int part = (int)(jx % a.parts);          // prototypes [part*MP, (part+1)*MP)
    const int64_t ix = jx / a.parts;
    const int64_t q8 = a.n_ranges / 8, r8 = a.n_ranges % 8;
    if (ix >= q8 + (xcd < r8 ? 1 : 0)) return;     // this XCD has fewer ranges
    const int64_t range = xcd * q8 + (xcd < r8 ? xcd : r8) + ix;
    const int64_t k0 = a.wg_start[range], k1 = a.wg_start[range + 1];
    if (k0 < 0 || k1 < k0 || k1 > a.max_items) return;
    const float ks2 = a.scale * kLog2e;
    const int64_t MD = (int64_t)a.M * D;
    const uint32_t row_stride = (uint32_t)a.H * D;
    int64_t cur_p = -1;

    for (int64_t k = k0; k < k1; ++k) {
        const int32_t* it = a.items + k * IT_WORDS;
        const int b = it[IT_B], h = it[IT_H], t0 = it[IT_T0], t1 = it[IT_T1];
        if (b < 0 || b >= a.B || h < 0 || h >= a.H || t0 < 0 || t1 < t0 || t1 > a.T) continue;
        const int64_t pkey = a.p_user ? (int64_t)b * a.H + h : h;
        const uint16_t* Pg = a.P + pkey * MD + (int64_t)part * C::MP * D;
        const uint16_t* Yg = a.Ymj + ((int64_t)b * a.H + h) * MD + (int64_t)part * C::MP * D;

        // token tiles: global -> registers one tile ahead, registers -> LDS buffer
        u32x4 kreg[C::NCH], vreg[C::NCH];
        float lse_r = 0.f, d_r = 0.f;
        auto fetch = [&](int ts) __attribute__((always_inline)) {
            const int64_t tb = ((int64_t)ts * a.H + h) * D;
#pragma unroll
            for (int c = 0; c < C::NCH; ++c) {
                const int idx = tid + c * C::THREADS;
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                u32x4 kv = (u32x4){0u, 0u, 0u, 0u}, vv = kv;
                if (idx < C::LD_CHUNKS && ts + tok < t1) {
                    const uint32_t off = (uint32_t)tok * row_stride + (uint32_t)(ch * 8);
                    kv = *reinterpret_cast<const u32x4*>(a.K + tb + off);
                    if constexpr (!XV) vv = *reinterpret_cast<const u32x4*>(a.V + tb + off);
                }
                kreg[c] = kv;
                vreg[c] = vv;
            }
            if (tid < 32) {
                // raw values: arithmetic on them here would wait for the loads
                const bool v = ts + tid < t1;
                lse_r = v ? a.lse[(int64_t)(ts + tid) * a.H + h] : 0.f;
                d_r = v ? a.Dbuf[(int64_t)(ts + tid) * a.H + h] : 0.f;
            }
        };
        auto store = [&](int buf) __attribute__((always_inline)) {
            uint16_t* Kd = reinterpret_cast<uint16_t*>(smem + C::OFF_K + buf * C::TILE);
            uint16_t* Vd = reinterpret_cast<uint16_t*>(smem + C::OFF_V + buf * C::TILE);
#pragma unroll
            for (int c = 0; c < C::NCH; ++c) {
                const int idx = tid + c * C::THREADS;
                if (idx < C::LD_CHUNKS) {
                    const int tok = idx / C::KCH, ch = idx % C::KCH;
                    *reinterpret_cast<u32x4*>(Kd + swz<D>(tok, ch)) = kreg[c];
                    if constexpr (!XV) *reinterpret_cast<u32x4*>(Vd + swz<D>(tok, ch)) = vreg[c];
                }
            }
            if (tid < 32) {
                reinterpret_cast<float*>(smem + C::OFF_L)[buf * 32 + tid] = -lse_r * kLog2e;
                reinterpret_cast<float*>(smem + C::OFF_D)[buf * 32 + tid] = d_r;
            }
        };

        fetch(t0);
        // With one prototype tile per wave, this wave's rows of P and dY are B
        // operands held in registers for the whole segment (each K / V operand is
        // then used once); with more, K and V operands are read once per tile and
        // reused, and P and dY are read from the LDS slices.
        constexpr int HK = kHold ? C::KS : 1;
        bf16x8 pop[HK], yop[HK];
        if constexpr (kHold) {
            const int prow = w * MW + l32;
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) {
                pop[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(Pg + prow * D + 16 * kk + 8 * hl));
                yop[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(Yg + prow * D + 16 * kk + 8 * hl));
            }
        }
        __syncthreads();  // the previous segment is done with every LDS buffer
        if constexpr (!kHold) {
            for (int i = tid; i < C::MP * C::KCH; i += C::THREADS) {
                const int r = i / C::KCH, c = i % C::KCH;
                if (pkey != cur_p) *reinterpret_cast<u32x4*>(Ps + swz<D>(r, c)) = reinterpret_cast<const u32x4*>(Pg)[i];
                *reinterpret_cast<u32x4*>(Ys + swz<D>(r, c)) = reinterpret_cast<const u32x4*>(Yg)[i];
            }
        }
        cur_p = pkey;
        store(0);
        __syncthreads();

        f32x16 acc[C::MT][C::JT];
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][jt][r] = 0.f;
        if constexpr (kHold) {
            // Wait here for the held operands.  Otherwise the compiler's
            // load-counter waits for them inside the loop also wait for each
            // iteration's prefetch of the next tile, issued after them, which
            // then lands before the tile's chains are done.
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) asm volatile("" ::"v"(pop[kk]), "v"(yop[kk]));
        }

        // Two waves per SIMD (waves w and w + 4 of the workgroup share a SIMD):
        // waves 0-3 run each tile's phases in order (S and dA chains, elementwise
        // dS, dP chain) while waves 4-7 run them one phase late (the elementwise
        // and dP work of the previous tile, then the chains of this tile), so that
        // between two barriers one wave of a SIMD feeds the matrix core while the
        // other runs its VALU work.  A late wave reads tile i in intervals i and
        // i + 1, so tiles rotate through three buffers; tile i + 1 is written at
        // the end of interval i, into the buffer last read in interval i - 1.
        if constexpr (C::PING) {
            const bool late = __builtin_amdgcn_readfirstlane(w) >= 4;
            const int n = (t1 - t0 + 31) / 32;
            auto chains = [&](int bi, f32x16& s, f32x16& da) __attribute__((always_inline)) {
                const uint16_t* Ks = reinterpret_cast<const uint16_t*>(smem + C::OFF_K + bi * C::TILE);
                const uint16_t* Vs = XV ? Ks : reinterpret_cast<const uint16_t*>(smem + C::OFF_V + bi * C::TILE);
#pragma unroll
                for (int r = 0; r < 16; ++r) s[r] = da[r] = 0.f;
#pragma unroll
                for (int kk = 0; kk < C::KS; ++kk) {
                    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Ks, swz<D>(l32, 2 * kk + hl)), pop[kk], s, 0, 0, 0);
                    da = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Vs, swz<D>(l32, 2 * kk + hl)), yop[kk], da, 0, 0, 0);
                }
            };
            auto ds_dp = [&](int bi, const f32x16& s, const f32x16& da) __attribute__((always_inline)) {
                const uint16_t* Ks = reinterpret_cast<const uint16_t*>(smem + C::OFF_K + bi * C::TILE);
                const float* nls = reinterpret_cast<const float*>(smem + C::OFF_L) + bi * 32;
                const float* Ds = reinterpret_cast<const float*>(smem + C::OFF_D) + bi * 32;
                float e[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int t = srow(r, hl);
                    const float A = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], ks2, nls[t]));
                    e[r] = A * (da[r] - Ds[t]);
                }
                const bf16x8 d0 = pack8(e), d1 = pack8(e + 8);
#pragma unroll
                for (int jt = 0; jt < C::JT; ++jt) {
                    const bf16x8 k0v = lds_tr_tokens<D>(Ks, lane, jt, 0);
                    const bf16x8 k1v = lds_tr_tokens<D>(Ks, lane, jt, 1);
                    acc[0][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(d0, k0v, acc[0][jt], 0, 0, 0);
                    acc[0][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(d1, k1v, acc[0][jt], 0, 0, 0);
                }
            };
            f32x16 s, da;   // a late wave carries its chains across the barrier
            // interval i with buffer BI = i % 3 (a constant, so that every tile
            // address is a fixed offset from the same lane registers)
            auto interval = [&](int i, auto bic) __attribute__((always_inline)) {
                constexpr int BI = decltype(bic)::value;
                constexpr int BP = (BI + 2) % 3, BN = (BI + 1) % 3;
                const bool more = i + 1 < n;
                if (more) fetch(t0 + 32 * (i + 1));
                if (!late && i < n) chains(BI, s, da);
                if (late ? i > 0 : i < n) ds_dp(late ? BP : BI, s, da);
                // the chains' operand reads are not hoisted into the dP work
                __builtin_amdgcn_sched_barrier(0);
                if (late && i < n) chains(BI, s, da);
                if (more) store(BN);
                __syncthreads();
            };
            for (int i = 0; i <= n; i += 3) {
                interval(i, std::integral_constant<int, 0>{});
                if (i + 1 <= n) interval(i + 1, std::integral_constant<int, 1>{});
                if (i + 2 <= n) interval(i + 2, std::integral_constant<int, 2>{});
            }
        } else {
        int buf = 0;
        for (int ts = t0; ts < t1; ts += 32, buf ^= 1) {
            const bool more = ts + 32 < t1;
            if (more) fetch(ts + 32);
            const uint16_t* Ks = reinterpret_cast<const uint16_t*>(smem + C::OFF_K + buf * C::TILE);
            const uint16_t* Vs = XV ? Ks : reinterpret_cast<const uint16_t*>(smem + C::OFF_V + buf * C::TILE);
            const float* nls = reinterpret_cast<const float*>(smem + C::OFF_L) + buf * 32;
            const float* Ds = reinterpret_cast<const float*>(smem + C::OFF_D) + buf * 32;

            constexpr int OK = kHold ? 1 : C::KS;
            bf16x8 kop[OK], vop[OK];
            if constexpr (!kHold) {
#pragma unroll
                for (int kk = 0; kk < C::KS; ++kk) {
                    kop[kk] = lds_b128(Ks, swz<D>(l32, 2 * kk + hl));
                    vop[kk] = lds_b128(Vs, swz<D>(l32, 2 * kk + hl));
                }
            }
            bf16x8 dso[C::MT][2];
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt) {
                f32x16 s, da;
#pragma unroll
                for (int r = 0; r < 16; ++r) s[r] = da[r] = 0.f;
                const int prow = w * MW + mt * 32 + l32;
#pragma unroll
                for (int kk = 0; kk < C::KS; ++kk) {
                    if constexpr (kHold) {
                        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Ks, swz<D>(l32, 2 * kk + hl)), pop[kk], s, 0, 0, 0);
                        da = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Vs, swz<D>(l32, 2 * kk + hl)), yop[kk], da, 0, 0, 0);
                    } else {
                        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kk], lds_b128(Ps, swz<D>(prow, 2 * kk + hl)), s, 0, 0, 0);
                        da = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[kk], lds_b128(Ys, swz<D>(prow, 2 * kk + hl)), da, 0, 0, 0);
                    }
                }
                float e[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int t = srow(r, hl);
                    const float A = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], ks2, nls[t]));
                    e[r] = A * (da[r] - Ds[t]);
                }
                dso[mt][0] = pack8(e);
                dso[mt][1] = pack8(e + 8);
            }
            // dP[m, j] += dS^T[m, t] K[t, j]: K^T operands straight from the row-major tile
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt) {
                const bf16x8 k0v = lds_tr_tokens<D>(Ks, lane, jt, 0);
                const bf16x8 k1v = lds_tr_tokens<D>(Ks, lane, jt, 1);
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    acc[mt][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dso[mt][0], k0v, acc[mt][jt], 0, 0, 0);
                    acc[mt][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dso[mt][1], k1v, acc[mt][jt], 0, 0, 0);
                }
            }
            // the next tile goes to the other buffer, whose readers (the previous
            // tile) passed the barrier at the end of the previous iteration
            if (more) store(buf ^ 1);
            __syncthreads();
        }
        }
        // partial of this segment for this part's prototype rows
        float* out = a.partials + k * MD + (int64_t)part * C::MP * D;
        uint32_t lane_off = (uint32_t)((w * MW + 4 * hl) * D + l32);
        asm volatile("" : "+v"(lane_off));
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const uint32_t o = lane_off + (uint32_t)((mt * 32 + 8 * (r >> 2) + (r & 3)) * D + jt * 32);
                    out[o] = a.scale * acc[mt][jt][r];
                }
    }
}

// dP[h] = sum of the partials of the segments of head h, in segment order
__global__ __launch_bounds__(256) void dp_sum_kernel(const int32_t* __restrict__ pair_start,
                                                     int64_t B, int32_t H, int64_t max_items,
                                                     const float* __restrict__ partials,
                                                     int64_t MD, float* __restrict__ dP) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= (int64_t)H * MD) return;
    const int64_t h = i / MD, rest = i % MD;
    int64_t s0 = pair_start[h * B], s1 = pair_start[(h + 1) * B];
    s0 = s0 < 0 ? 0 : (s0 > max_items ? max_items : s0);
    s1 = s1 < s0 ? s0 : (s1 > max_items ? max_items : s1);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8   // several segments' loads in flight; the sum keeps segment order
    for (int64_t k = s0; k < s1; ++k) {
        const float4 v = *reinterpret_cast<const float4*>(partials + k * MD + rest);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    *reinterpret_cast<float4*>(dP + i) = acc;
}

// dP[b,h] = sum of the partials of the segments of pair (b, h), in segment order
// (per-user prototypes); zero for a pair without tokens
__global__ __launch_bounds__(256) void dp_pair_sum_kernel(const int32_t* __restrict__ pair_start, int64_t B,
                                                          int32_t H, int64_t max_items,
                                                          const float* __restrict__ partials, int64_t MD,
                                                          float* __restrict__ dP) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= B * H * MD) return;
    const int64_t bh = i / MD, rest = i % MD;
    const int64_t b = bh / H, h = bh % H;
    const int64_t pr = h * B + b;   // head-major pair order of the work list
    int64_t s0 = pair_start[pr], s1 = pair_start[pr + 1];
    s0 = s0 < 0 ? 0 : (s0 > max_items ? max_items : s0);
    s1 = s1 < s0 ? s0 : (s1 > max_items ? max_items : s1);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8   // several segments' loads in flight; the sum keeps segment order
    for (int64_t k = s0; k < s1; ++k) {
        const float4 v = *reinterpret_cast<const float4*>(partials + k * MD + rest);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    *reinterpret_cast<float4*>(dP + i) = acc;
}

template <int D, int NW, bool XV>
hipError_t launch_token(const TokArgs& a, int64_t n_ranges, hipStream_t stream) {
    using C = TokCfg<D, NW>;
    auto kern = bwd_token_kernel<D, NW, XV>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)n_ranges), dim3(C::THREADS), C::LDS, stream, a);
    return hipGetLastError();
}

template <int D, int MW, int NW, bool XV>
hipError_t launch_proto_t(const ProtoArgs& a, int64_t n_ranges, hipStream_t stream) {
    using C = ProtoCfg<D, MW, NW>;
    auto kern = bwd_proto_kernel<D, MW, NW, XV>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    ProtoArgs b = a;
    b.n_ranges = n_ranges;
    b.parts = a.M / C::MP;
    const int64_t per_xcd = (n_ranges + 7) / 8;
    hipLaunchKernelGGL(kern, dim3((unsigned)(8 * per_xcd * b.parts)), dim3(C::THREADS), C::LDS, stream, b);
    return hipGetLastError();
}

template <int D, int MW, int NW>
hipError_t launch_proto(const ProtoArgs& a, bool xv, int64_t n_ranges, hipStream_t stream) {
    return xv ? launch_proto_t<D, MW, NW, true>(a, n_ranges, stream)
              : launch_proto_t<D, MW, NW, false>(a, n_ranges, stream);
}

template <int D, int NBLK, bool XV>
hipError_t launch_token_held(const TokArgs& a, int64_t n_ranges, hipStream_t stream) {
    using C = HeldCfg<D, NBLK>;
    auto kern = bwd_token_held_kernel<D, NBLK, XV>;
    hipLaunchKernelGGL(kern, dim3((unsigned)n_ranges), dim3(C::THREADS), 0, stream, a);
    return hipGetLastError();
}

template <int D, bool XV>
hipError_t launch_token_xv(const TokArgs& a, int64_t n_ranges, hipStream_t stream) {
    switch (a.M) {
        case 128: return launch_token_held<D, 4, XV>(a, n_ranges, stream);
        case 256: return launch_token_held<D, 8, XV>(a, n_ranges, stream);
        case 384: return launch_token_held<D, 12, XV>(a, n_ranges, stream);
        case 512: return launch_token_held<D, 16, XV>(a, n_ranges, stream);
        default: return launch_token<D, kTokWaves, XV>(a, n_ranges, stream);
    }
}

template <int D>
hipError_t launch_token_d(const TokArgs& a, bool xv, int64_t n_ranges, hipStream_t stream) {
    return xv ? launch_token_xv<D, true>(a, n_ranges, stream) : launch_token_xv<D, false>(a, n_ranges, stream);
}

}  // namespace

int32_t fused_bwd_ranges_per_cu() { return 8 / kTokWaves; }

// prototypes per part of the dP kernel: P and dY slices of MP x d bf16 each fit in LDS
int32_t fused_bwd_part(int32_t M, int32_t d) {
    const int cap = d == 64 ? 512 : 256;
    for (int mp = cap; mp >= 128; mp -= 128)
        if (M % mp == 0 && (mp == 128 || mp == 256 || mp == 512)) return mp;
    return 0;
}

bool fused_bwd_supported(int32_t M, int32_t d) {
    return (d == 64 || d == 128) && M % 128 == 0 && M <= 4096 && fused_bwd_part(M, d) > 0;
}

hipError_t launch_fused_bwd(const FusedBwdArgs& f, hipStream_t stream) {
    const int64_t MD = (int64_t)f.M * f.d;
    // dY (R summed) and P in the layouts the contractions read
    {
        ProfScope ps("bwd_prep", stream);
        const int64_t n_p = f.p_user ? f.B * f.H : f.H;
        const int64_t nblocks = (f.B * f.H + n_p) * (f.M / 32);
        if (f.d == 64)
            hipLaunchKernelGGL(prep_kernel<64>, dim3((unsigned)nblocks), dim3(256), 0, stream,
                               f.dsketch, f.B, f.R, f.H, f.M, n_p, f.P, f.Ymj, f.Yjm, f.Pjm);
        else
            hipLaunchKernelGGL(prep_kernel<128>, dim3((unsigned)nblocks), dim3(256), 0, stream,
                               f.dsketch, f.B, f.R, f.H, f.M, n_p, f.P, f.Ymj, f.Yjm, f.Pjm);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (f.n_ranges > 0) {
        TokArgs t;
        t.K = f.K; t.V = f.V; t.P = f.P; t.Pjm = f.Pjm; t.Ymj = f.Ymj; t.Yjm = f.Yjm;
        t.lse = f.lse; t.items = f.items; t.wg_start = f.wg_start; t.max_items = f.max_items;
        t.T = f.T; t.B = (int32_t)f.B; t.H = f.H; t.M = f.M; t.scale = f.scale;
        t.dK = f.dK; t.dV = f.dV; t.dX = f.dX; t.Dbuf = f.Dbuf; t.p_user = f.p_user; t.dx_add = f.dx_add;
        const bool xv = f.dX != nullptr;
        hipError_t e;
        {
            ProfScope ps("bwd_token", stream);
            e = f.d == 64 ? launch_token_d<64>(t, xv, f.n_ranges, stream)
                          : launch_token_d<128>(t, xv, f.n_ranges, stream);
        }
        if (e != hipSuccess) return e;
        ProtoArgs p;
        p.K = f.K; p.V = f.V; p.P = f.P; p.Ymj = f.Ymj; p.lse = f.lse; p.Dbuf = f.Dbuf;
        p.items = f.items; p.wg_start = f.wg_start; p.max_items = f.max_items; p.T = f.T;
        p.B = (int32_t)f.B; p.H = f.H; p.M = f.M; p.scale = f.scale; p.partials = f.partials;
        p.p_user = f.p_user;
        const int mp = fused_bwd_part(f.M, f.d);
        ProfScope ps("bwd_proto", stream);
        // eight waves (two per SIMD) when the part has at least 32 prototypes per wave
        if (f.d == 64) {
            e = mp == 128 ? launch_proto<64, 32, 4>(p, xv, f.n_ranges, stream)
              : mp == 256 ? launch_proto<64, 32, 8>(p, xv, f.n_ranges, stream)
                          : launch_proto<64, 64, 8>(p, xv, f.n_ranges, stream);
        } else {
            e = mp == 128 ? launch_proto<128, 32, 4>(p, xv, f.n_ranges, stream)
                          : launch_proto<128, 32, 8>(p, xv, f.n_ranges, stream);
        }
        if (e != hipSuccess) return e;
    }
    ProfScope ps("bwd_dp_sum", stream);
    if (f.p_user) {
        const int64_t n = f.B * f.H * MD / 4;
        hipLaunchKernelGGL(dp_pair_sum_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                           f.pair_start, f.B, f.H, f.max_items, f.partials, MD, f.dP);
    } else {
        const int64_t n = (int64_t)f.H * MD / 4;
        hipLaunchKernelGGL(dp_sum_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                           f.pair_start, f.B, f.H, f.max_items, f.partials, MD, f.dP);
    }
    return hipGetLastError();
}

}  // namespace sa

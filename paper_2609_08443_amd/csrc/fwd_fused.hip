// Fused bf16 forward of the SA sketching step on gfx950 matrix cores.
//
// Per token tile of 32 tokens of one (user, head) segment, without writing the
// T x M affinities anywhere (section 4.4, FlashSA: block-wise affinities,
// prototype-wise softmax statistics, aggregation into the sketch):
//
//   S   = K_tile . P^T                  32 x M, bf16 MFMA 32x32x16, fp32 accumulate
//   E   = exp(scale * S - c_t)           c_t >= max_m scale * S[t, m]   (see below)
//   z_t = sum_m E,   lse_t = c_t + log z_t
//   acc[M, d] += E^T . (V_tile / z)      bf16 MFMA, fp32 accumulate
//
// The softmax over the M prototypes of a token (section 3.1) is shift
// invariant, so any shift c_t works as long as exp neither overflows nor
// underflows.  The shift used is the Cauchy-Schwarz bound
// c_t = scale * |K_t| * max_m |P_m|, which is known before the logits are:
// each 32x32 tile of S is exponentiated as soon as its MFMAs finish (no pass
// over all M logits first), and the exponentials of one tile can overlap the
// MFMAs of the next.  When the bound is so loose that a token's
// sum z_t would underflow (z_t < 2^-64, i.e. logits far below the bound), the
// tile is recomputed with the exact per-token max.
//
// Workgroup = 4 waves (one per SIMD); wave w owns prototypes
// [w*MW, (w+1)*MW) for both GEMMs, so the M x d fp32 accumulator is spread
// over the four SIMDs' register files.  The per-token sums over the M
// prototypes are reduced in registers (over the wave's 32x32 tiles), across
// the 32 lanes of a row (DPP and permlane, no LDS), and across waves through
// LDS.
//
// Layouts: see tile_ops.h.  S is computed with tokens as rows, so its C layout
// (lane = prototype, register = token) is directly the A operand of the
// aggregation acc[m, j] += sum_t E[t, m] V'[t, j], with the k slots in the perm16
// token order; V' is staged row-major in LDS and read as the matching B operand
// with the transposing LDS load.  1/z is folded into V' (d values per token
// instead of M).
//
// Pipeline per tile i (two workgroup barriers on the common path):
//   S/exp over the wave's prototype tiles  (K(i) in LDS buffer i%2)
//   stage K(i+1) into buffer (i+1)%2; per-token partial sums to LDS
//   --- barrier ---
//   z, lse; stage V(i)/z; issue the global loads of tile i+2
//   --- barrier ---
//   aggregation MFMAs
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

using namespace tile;

// z below this means the shift was too far above the largest logit
constexpr float kUnderflowZ = 5.421010862427522e-20f;  // 2^-64
// relative margin on the bound for the rounding of the fp32 norms and logits
constexpr float kBoundMargin = 1.0f + 1.0f / 1024.0f;

__device__ inline float sumsq8(uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float a = bf16_lo(w[i]), b = bf16_hi(w[i]);
        s = __builtin_fmaf(a, a, s);
        s = __builtin_fmaf(b, b, s);
    }
    return s;
}

// Cross-lane moves without LDS: DPP inside rows of 16 lanes, then
// v_permlane16_swap between the two rows of each 32-lane half.
template <int CTRL>
__device__ inline float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;
constexpr int kRowRor4 = 0x124;
constexpr int kRowRor8 = 0x128;

// One step of a logits chain overlapped with exponentials: one MFMA of the
// chain that accumulates the next 32x32 logits tile into sn, then two rows of
// the current tile, e = 2^(s * ks + n), added into their sums and packed to
// bf16.  The VALU work is independent of the MFMA, so it issues while the
// matrix core runs.  Each exponential's first use is one instruction after it
// (the transcendental forwarding gap); sn must not be read for 32 states after
// the last step of a chain.
template <bool FIRST>
__device__ inline void chain_exp_step(f32x16& sn, const bf16x8& k, const bf16x8& b, float s0, float s1,
                                      float n0, float n1, float ks, float& z0, float& z1, uint32_t& ep) {
    float t0, t1;
    if constexpr (FIRST) {
        asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %[sn], %[k], %[b], 0\n\t"
            "v_fma_f32 %[t0], %[s0], %[ks], %[n0]\n\tv_fma_f32 %[t1], %[s1], %[ks], %[n1]\n\t"
            "v_exp_f32 %[t0], %[t0]\n\tv_exp_f32 %[t1], %[t1]\n\t"
            "v_add_f32 %[z0], %[z0], %[t0]\n\tv_add_f32 %[z1], %[z1], %[t1]\n\t"
            "v_cvt_pk_bf16_f32 %[ep], %[t0], %[t1]"
            : [sn] "=&v"(sn), [t0] "=&v"(t0), [t1] "=&v"(t1), [z0] "+v"(z0), [z1] "+v"(z1), [ep] "=&v"(ep)
            : [k] "v"(k), [b] "v"(b), [s0] "v"(s0), [s1] "v"(s1), [n0] "v"(n0), [n1] "v"(n1), [ks] "v"(ks));
    } else {
        asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %[sn], %[k], %[b], %[sn]\n\t"
            "v_fma_f32 %[t0], %[s0], %[ks], %[n0]\n\tv_fma_f32 %[t1], %[s1], %[ks], %[n1]\n\t"
            "v_exp_f32 %[t0], %[t0]\n\tv_exp_f32 %[t1], %[t1]\n\t"
            "v_add_f32 %[z0], %[z0], %[t0]\n\tv_add_f32 %[z1], %[z1], %[t1]\n\t"
            "v_cvt_pk_bf16_f32 %[ep], %[t0], %[t1]"
            : [sn] "+v"(sn), [t0] "=&v"(t0), [t1] "=&v"(t1), [z0] "+v"(z0), [z1] "+v"(z1), [ep] "=&v"(ep)
            : [k] "v"(k), [b] "v"(b), [s0] "v"(s0), [s1] "v"(s1), [n0] "v"(n0), [n1] "v"(n1), [ks] "v"(ks));
    }
}

// reduce across the 32 lanes of each half-wave; every lane gets the result
__device__ inline float half_max(float v) {
    v = fmaxf(v, dpp<kQuadXor1>(v));
    v = fmaxf(v, dpp<kQuadXor2>(v));
    v = fmaxf(v, dpp<kRowRor4>(v));
    v = fmaxf(v, dpp<kRowRor8>(v));
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float half_sum(float v) {
    v += dpp<kQuadXor1>(v);
    v += dpp<kQuadXor2>(v);
    v += dpp<kRowRor4>(v);
    v += dpp<kRowRor8>(v);
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// sum over aligned groups of G = 8 or 16 consecutive lanes; every lane gets it
template <int G>
__device__ inline float group_sum(float v) {
    v += dpp<kQuadXor1>(v);
    v += dpp<kQuadXor2>(v);
    v += dpp<kRowHalfMirror>(v);
    if constexpr (G == 16) v += dpp<kRowMirror>(v);
    return v;
}
// Sums of 16 values across the 32 lanes of each half-wave, one value kept per
// lane: the lanes exchange halves of their remaining values at each level
// (partners l ^ 16, l ^ 8, l ^ 7, l ^ 2, l ^ 1), so 38 instructions do what 16
// full reductions (96) would.  Afterwards lanes 2 t and 2 t + 1 of the half hold
// the total of value t.  Every value is summed over the same tree of lanes (the
// pairings are xor masks), whatever its index.
__device__ inline float half_sum16(const float (&v)[16], int l32) {
    float u[8], w[4], x[2];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        // lanes 0-15 keep value i, lanes 16-31 value i + 8
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + 8]), false,
                                                        false);
        u[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    const bool b3 = (l32 & 8) != 0, b2 = (l32 & 4) != 0, b1 = (l32 & 2) != 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = (b3 ? u[j + 4] : u[j]) + dpp<kRowRor8>(b3 ? u[j] : u[j + 4]);
#pragma unroll
    for (int k = 0; k < 2; ++k) x[k] = (b2 ? w[k + 2] : w[k]) + dpp<kRowHalfMirror>(b2 ? w[k] : w[k + 2]);
    const float y = (b1 ? x[1] : x[0]) + dpp<kQuadXor2>(b1 ? x[0] : x[1]);
    return y + dpp<kQuadXor1>(y);
}

__device__ inline float wave_max(float v) {
    v = half_max(v);
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

template <int D, int MW, int NW>
struct Cfg {
    static constexpr int M = MW * NW;
    static constexpr int MT = MW / 32;          // 32x32 tiles of S per wave
    static constexpr int KS = D / 16;           // k steps of the S GEMM
    static constexpr int JT = D / 32;           // column tiles of the accumulator
    static constexpr int KCH = D / 8;           // 16-byte chunks per K/V row
    static constexpr int THREADS = NW * 64;
    static constexpr int LD_CHUNKS = 32 * KCH;  // 16-byte chunks per K (or V) tile
    static constexpr int NLD = (LD_CHUNKS + THREADS - 1) / THREADS;
    // LDS layout (bytes)
    static constexpr int P_BYTES = M * D * 2;
    static constexpr int K_BYTES = 32 * D * 2;  // one K tile buffer (two are kept)
    static constexpr int V_BYTES = D * 32 * 2;
    static constexpr int RED_BYTES = NW * 32 * 4;
    static constexpr int OFF_K = P_BYTES;
    static constexpr int OFF_V = OFF_K + 2 * K_BYTES;
    static constexpr int OFF_SUM = OFF_V + V_BYTES;      // [NW][32] partial sums (bound path)
    static constexpr int OFF_MAX = OFF_SUM + RED_BYTES;  // [NW][32] partial maxima (exact path)
    static constexpr int OFF_SUM2 = OFF_MAX + RED_BYTES; // [NW][32] partial sums (exact path)
    static constexpr int OFF_KN = OFF_SUM2 + RED_BYTES;  // [2][32] token norms
    static constexpr int OFF_NB = OFF_KN + 2 * 32 * 4;   // [2][32] the tokens' shifts, -c_t log2(e)
    static constexpr int OFF_PN = OFF_NB + 2 * 32 * 4;   // [NW] prototype norm maxima
    static constexpr int OFF_SH = OFF_PN + 16 * 4;       // [32] exact-path shifts
    static constexpr int LDS = OFF_SH + 32 * 4;
};

template <int D, int MW, int NW>
__global__ __launch_bounds__(NW * 64, 1) void fwd_fused_kernel(FusedFwdArgs a) {
    using C = Cfg<D, MW, NW>;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* Ps = reinterpret_cast<uint16_t*>(smem);
    uint16_t* Kbuf = reinterpret_cast<uint16_t*>(smem + C::OFF_K);
    uint16_t* Vt = reinterpret_cast<uint16_t*>(smem + C::OFF_V);
    float* red_sum = reinterpret_cast<float*>(smem + C::OFF_SUM);
    float* red_max = reinterpret_cast<float*>(smem + C::OFF_MAX);
    float* red_sum2 = reinterpret_cast<float*>(smem + C::OFF_SUM2);
    float* knorm = reinterpret_cast<float*>(smem + C::OFF_KN);
    float* kshift = reinterpret_cast<float*>(smem + C::OFF_NB);
    float* pnorm = reinterpret_cast<float*>(smem + C::OFF_PN);
    float* shift_s = reinterpret_cast<float*>(smem + C::OFF_SH);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int l32 = lane & 31;
    const int hl = lane >> 5;  // half of the wave

    const int64_t range = xcd_range(blockIdx.x, gridDim.x);
    const int64_t k0 = a.wg_start[range];
    const int64_t k1 = a.wg_start[range + 1];
    if (k0 < 0 || k1 < k0 || k1 > a.max_items) return;  // malformed offsets: nothing safe to do

    const float ks2 = a.scale * kLog2e;
    const int64_t MD = (int64_t)C::M * D;
    const uint32_t row_stride = (uint32_t)a.H * D;
    int64_t cur_p = -1;   // prototype block in LDS: head, or (user, head) with per-user P
    float pmax = 0.f;  // max_m |P[h, m]| of the loaded head

    for (int64_t k = k0; k < k1; ++k) {
        const int32_t* it = a.items + k * IT_WORDS;
        const int b = it[IT_B];
        const int h = it[IT_H];
        const int t0 = it[IT_T0];
        const int t1 = it[IT_T1];
        const int split = it[IT_SPLIT];
        if (b < 0 || b >= a.B || h < 0 || h >= a.H || t0 < 0 || t1 < t0 || t1 > a.T) continue;

        // ---- prototypes of head h into LDS, with max_m |P_m|
        const int64_t pkey = a.p_user ? (int64_t)b * a.H + h : h;
        if (pkey != cur_p) {
            const uint4* src = reinterpret_cast<const uint4*>(a.P + pkey * C::M * D);
            float nmax = 0.f;
            for (int i = tid; i < C::M * C::KCH; i += C::THREADS) {
                const int r = i / C::KCH, c = i % C::KCH;
                const uint4 v = src[i];
                *reinterpret_cast<uint4*>(Ps + swz<D>(r, c)) = v;
                // the KCH chunks of a row sit in KCH consecutive lanes
                nmax = fmaxf(nmax, group_sum<C::KCH>(sumsq8(v)));
            }
            nmax = wave_max(nmax);
            if (lane == 0) pnorm[w] = nmax;
            __syncthreads();
            float m2 = pnorm[0];
#pragma unroll
            for (int ww = 1; ww < NW; ++ww) m2 = fmaxf(m2, pnorm[ww]);
            pmax = __builtin_sqrtf(m2);
            cur_p = pkey;
        }
        // shift bound of token t = cb * |K_t|
        const float cb = a.scale * pmax * kBoundMargin;

        f32x16 acc[C::MT][C::JT];
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][jt][r] = 0.f;

        // global tile loads into registers: 32-bit per-lane offsets, uniform tile base
        // K is loaded two tiles ahead of its use and V one tile ahead: both are
        // issued at the end of a tile, so neither register set is copied
        // between tiles.  Rows past the end of the range read its last token
        // when every chunk slot is used (unpredicated loads; their V is zeroed
        // at staging), else they are zero.
        uint4 kreg[C::NLD], vreg[C::NLD];
        auto load_rows = [&](const uint16_t* X, int ts, uint4 (&dst)[C::NLD]) {
            const uint16_t* Xb = X + ((int64_t)ts * a.H + h) * D;
            const int last = t1 - 1 - ts;
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                const int idx = tid + i * C::THREADS;
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                if constexpr (C::LD_CHUNKS % C::THREADS == 0) {
                    const uint32_t off = (uint32_t)min(tok, last) * row_stride + (uint32_t)(ch * 8);
                    dst[i] = *reinterpret_cast<const uint4*>(Xb + off);
                } else {
                    uint4 x = make_uint4(0, 0, 0, 0);
                    if (idx < C::LD_CHUNKS && tok <= last)
                        x = *reinterpret_cast<const uint4*>(Xb + (uint32_t)tok * row_stride + (uint32_t)(ch * 8));
                    dst[i] = x;
                }
            }
        };
        // K tile (from kreg) into LDS buffer `buf`, with the token norms
        auto stage_k = [&](int kb) {
            uint16_t* Kd = Kbuf + kb * (32 * D);
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                int idx = tid + i * C::THREADS;
                asm volatile("" : "+v"(idx));
                if (idx < C::LD_CHUNKS) {
                    const int tok = idx / C::KCH, ch = idx % C::KCH;
                    *reinterpret_cast<uint4*>(Kd + swz<D>(tok, ch)) = kreg[i];
                    const float ss = group_sum<C::KCH>(sumsq8(kreg[i]));
                    if (ch == 0) {
                        const float kn = __builtin_sqrtf(ss);
                        knorm[kb * 32 + tok] = kn;
                        kshift[kb * 32 + tok] = -cb * kLog2e * kn;
                    }
                }
            }
        };
        // one 32x32 tile of S for this wave's prototype tile mt
        // one 32x32 tile of S for this wave's prototype tile mt.  The matrix-core
        // chain is written out so that the tile lands in VGPRs (the exponentials
        // read it) while the accumulator stays in AGPRs; the compiler does not
        // model these instructions, so each waits 2 states after any VALU write
        // of its operands, and the tile is read 32 states after the last one.
        auto read_bp = [&](bf16x8* bp, int mt) {
            const int prow = w * MW + mt * 32 + l32;
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) bp[kk] = lds_b128(Ps, swz<D>(prow, 2 * kk + hl));
        };
        auto s_chain = [&](const bf16x8* kop, const bf16x8* bp) {
            f32x16 s;
            __builtin_amdgcn_sched_barrier(0);
            asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(kop[0]), "v"(bp[0]));
#pragma unroll
            for (int kk = 1; kk < C::KS; ++kk)
                asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(kop[kk]), "v"(bp[kk]));
            asm volatile("s_nop 15\n\ts_nop 15" : "+v"(s));
            return s;
        };
        auto s_tile = [&](const bf16x8* kop, int mt) {
            bf16x8 bp[C::KS];
            read_bp(bp, mt);
            return s_chain(kop, bp);
        };

        const int ntiles = (t1 - t0 + 31) / 32;
        // prologue: tile 0 staged, tile 1 in flight
        load_rows(a.K, t0, kreg);
        load_rows(a.V, t0, vreg);
        stage_k(0);
        if (ntiles > 1) load_rows(a.K, t0 + 32, kreg);
        __syncthreads();

        for (int ti = 0; ti < ntiles; ++ti) {
            const int ts = t0 + ti * 32;
            const int kb = ti & 1;
            const uint16_t* Ks = Kbuf + kb * (32 * D);

            // ---- per-row shift: -c_t * log2(e) for this lane's 16 rows, c_t = cb * |K_t|
            float nb[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) nb[r] = kshift[kb * 32 + srow(r, hl)];

            // ---- S tiles, exponentiated as they complete
            bf16x8 kop[C::KS];
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) kop[kk] = lds_b128(Ks, swz<D>(l32, 2 * kk + hl));
            float rsum[16];
            bf16x8 eop[C::MT][2];
            bf16x8 bp[C::KS];
            read_bp(bp, 0);
            if constexpr (C::KS == 8 && C::MT > 1) {
                // the chain of prototype tile mt+1 runs on the matrix cores while
                // the exponentials of tile mt are taken, one MFMA per two rows
#pragma unroll
                for (int r = 0; r < 16; ++r) rsum[r] = 0.f;
                f32x16 s = s_chain(kop, bp);
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    uint32_t ep[8];
                    if (mt + 1 < C::MT) {
                        read_bp(bp, mt + 1);
                        // the eight operand reads are issued together, not each
                        // just before its MFMA
                        __builtin_amdgcn_sched_barrier(0);
                        f32x16 sn;
                        chain_exp_step<true>(sn, kop[0], bp[0], s[0], s[1], nb[0], nb[1], ks2, rsum[0], rsum[1], ep[0]);
#pragma unroll
                        for (int kk = 1; kk < 8; ++kk)
                            chain_exp_step<false>(sn, kop[kk], bp[kk], s[2 * kk], s[2 * kk + 1], nb[2 * kk],
                                                  nb[2 * kk + 1], ks2, rsum[2 * kk], rsum[2 * kk + 1], ep[kk]);
                        asm volatile("s_nop 15\n\ts_nop 15" : "+v"(sn));
                        s = sn;
                    } else {
#pragma unroll
                        for (int kk = 0; kk < 8; ++kk) {
                            const float e0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2 * kk], ks2, nb[2 * kk]));
                            const float e1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2 * kk + 1], ks2, nb[2 * kk + 1]));
                            rsum[2 * kk] += e0;
                            rsum[2 * kk + 1] += e1;
                            ep[kk] = pack_bf16x2(e0, e1);
                        }
                    }
                    eop[mt][0] = __builtin_bit_cast(bf16x8, make_uint4(ep[0], ep[1], ep[2], ep[3]));
                    eop[mt][1] = __builtin_bit_cast(bf16x8, make_uint4(ep[4], ep[5], ep[6], ep[7]));
                    asm volatile("" : "+v"(eop[mt][0]), "+v"(eop[mt][1]));
                }
            } else
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt) {
                const f32x16 s = s_chain(kop, bp);
                // the chain has completed: the next prototype tile's operands load
                // under this tile's exponentials
                if (mt + 1 < C::MT) read_bp(bp, mt + 1);
                float e[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    e[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], ks2, nb[r]));
                    rsum[r] = mt == 0 ? e[r] : rsum[r] + e[r];
                }
                eop[mt][0] = pack8(e);
                eop[mt][1] = pack8(e + 8);
                // packed here: left to the compiler, the packing sinks past the
                // branch below and the fp32 exponentials stay live through it
                asm volatile("" : "+v"(eop[mt][0]), "+v"(eop[mt][1]));
            }
            {
                const float z = half_sum16(rsum, l32);
                if ((l32 & 1) == 0) red_sum[w * 32 + srow(l32 >> 1, hl)] = z;
            }
            // ---- next K tile into the other buffer
            if (ti + 1 < ntiles) stage_k(kb ^ 1);
            __syncthreads();  // B_z

            // ---- tile-uniform check that the bound did not underflow any z_t
            bool exact;
            {
                const int tt = lane & 31;
                float z = 0.f;
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) z += red_sum[ww * 32 + tt];
                exact = __builtin_amdgcn_ballot_w64(z < kUnderflowZ && ts + tt < t1) != 0;
            }
            if (exact) {
                // rare: exact per-token max over the prototypes, then the exponentials
                // again (rsum holds the running max first; its sums are in LDS)
#pragma unroll
                for (int r = 0; r < 16; ++r) rsum[r] = -INFINITY;
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    const f32x16 s = s_tile(kop, mt);
#pragma unroll
                    for (int r = 0; r < 16; ++r) rsum[r] = fmaxf(rsum[r], s[r]);
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) rsum[r] = half_max(rsum[r]);
                if (l32 == 0) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) red_max[w * 32 + srow(r, hl)] = rsum[r];
                }
                __syncthreads();
                if (tid < 32) {
                    float mu = red_max[tid];
#pragma unroll
                    for (int ww = 1; ww < NW; ++ww) mu = fmaxf(mu, red_max[ww * 32 + tid]);
                    shift_s[tid] = -mu * ks2;
                }
                __syncthreads();
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    nb[r] = shift_s[srow(r, hl)];
                    rsum[r] = 0.f;
                }
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    const f32x16 s = s_tile(kop, mt);
                    float e[16];
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        e[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], ks2, nb[r]));
                        rsum[r] += e[r];
                    }
                    eop[mt][0] = pack8(e);
                    eop[mt][1] = pack8(e + 8);
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) rsum[r] = half_sum(rsum[r]);
                if (l32 == 0) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) red_sum2[w * 32 + srow(r, hl)] = rsum[r];
                }
                __syncthreads();
            }
            const float* zsrc = exact ? red_sum2 : red_sum;

            // ---- lse of the tile's tokens: thread tt of wave 0 handles token tt
            if (tid < 32 && a.lse && ts + tid < t1) {
                float z = 0.f;
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) z += zsrc[ww * 32 + tid];
                float c;
                if (exact) {
                    c = -shift_s[tid] / kLog2e;
                } else {
                    c = cb * knorm[kb * 32 + tid];
                }
                a.lse[(int64_t)(ts + tid) * a.H + h] = c + __logf(z);
            }

            // ---- stage V / z (row-major; the aggregation reads it transposed)
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                int idx = tid + i * C::THREADS;
                asm volatile("" : "+v"(idx));  // addresses built here, not hoisted
                if (idx < C::LD_CHUNKS) {
                    const int tok = idx / C::KCH, ch = idx % C::KCH;
                    float z = 0.f;
#pragma unroll
                    for (int ww = 0; ww < NW; ++ww) z += zsrc[ww * 32 + tok];
                    const float inv = ts + tok < t1 ? 1.0f / z : 0.0f;
                    *reinterpret_cast<uint4*>(Vt + swz<D>(tok, ch)) = scale8(vreg[i], inv);
                }
            }
            // K of tile i+2 and V of tile i+1 (kreg was staged above, vreg just now)
            if (ti + 2 < ntiles) load_rows(a.K, ts + 64, kreg);
            if (ti + 1 < ntiles) load_rows(a.V, ts + 32, vreg);
            // B_v: V' staged, K(i+1) visible; the loads of tile i+2 stay in flight
            // (they have the aggregation of this tile and the logits of the next)
            lds_barrier();

            // ---- acc[m, j] += E^T . V'
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt) {
                const bf16x8 v0 = lds_tr_tokens<D>(Vt, lane, jt, 0);
                const bf16x8 v1 = lds_tr_tokens<D>(Vt, lane, jt, 1);
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    acc[mt][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eop[mt][0], v0, acc[mt][jt], 0, 0, 0);
                    acc[mt][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eop[mt][1], v1, acc[mt][jt], 0, 0, 0);
                }
            }
        }

        // ---- flush: the whole sketch of the pair, or this segment's partial
        float* out = split ? a.partials + k * MD : a.sketch + ((int64_t)b * a.H + h) * MD;
        uint32_t lane_off = (uint32_t)((w * MW + 4 * hl) * D + l32);
        // keep the per-store addresses from being hoisted out of the loops (they
        // would stay live in registers through the whole tile loop)
        asm volatile("" : "+v"(lane_off));
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const uint32_t o = lane_off + (uint32_t)((mt * 32 + 8 * (r >> 2) + (r & 3)) * D + jt * 32);
                    out[o] = acc[mt][jt][r];
                }
        __syncthreads();  // LDS tiles and norms are reused by the next segment
    }
}

template <int D, int MW, int NW>
hipError_t launch_inst(const FusedFwdArgs& a, hipStream_t stream) {
    using C = Cfg<D, MW, NW>;
    auto kern = fwd_fused_kernel<D, MW, NW>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)a.n_ranges), dim3(C::THREADS), C::LDS, stream, a);
    return hipGetLastError();
}

template <int D, int MW, int NW>
hipError_t occ_inst(int* blocks) {
    using C = Cfg<D, MW, NW>;
    auto kern = fwd_fused_kernel<D, MW, NW>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, kern, C::THREADS, C::LDS);
}

}  // namespace

// Instances (d, prototypes per wave, waves): M = MW * NW, four waves (one per
// SIMD), each holding its MW x d share of the fp32 accumulator in registers.
#define SA_FUSED_CASES(X)  \
    X(64, 32, 4)           \
    X(64, 64, 4)           \
    X(64, 96, 4)           \
    X(64, 128, 4)          \
    X(64, 160, 4)          \
    X(64, 192, 4)          \
    X(64, 224, 4)          \
    X(64, 256, 4)          \
    X(128, 32, 4)          \
    X(128, 64, 4)          \
    X(128, 96, 4)          \
    X(128, 128, 4)

// Waves per workgroup for an (M, d) (every instance uses four, one per SIMD).
int fused_waves(int32_t, int32_t) { return 4; }

bool fused_fwd_supported(int32_t M, int32_t d) {
    if (M % 128 != 0) return false;
#define X(DD, MWW, NWW) if (d == DD && M == NWW * MWW) return true;
    SA_FUSED_CASES(X)
#undef X
    return false;
}

size_t fused_fwd_lds_bytes(int32_t M, int32_t d) {
    const int nw = fused_waves(M, d);
#define X(DD, MWW, NWW) if (d == DD && M == NWW * MWW && nw == NWW) return Cfg<DD, MWW, NWW>::LDS;
    SA_FUSED_CASES(X)
#undef X
    return 0;
}

hipError_t fused_fwd_occupancy(int32_t M, int32_t d, int* blocks) {
    const int nw = fused_waves(M, d);
#define X(DD, MWW, NWW) if (d == DD && M == NWW * MWW && nw == NWW) return occ_inst<DD, MWW, NWW>(blocks);
    SA_FUSED_CASES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_fused_fwd(const FusedFwdArgs& a, hipStream_t stream) {
    if (a.n_ranges == 0) return hipSuccess;
    const int nw = fused_waves(a.M, a.d);
#define X(DD, MWW, NWW) if (a.d == DD && a.M == NWW * MWW && nw == NWW) return launch_inst<DD, MWW, NWW>(a, stream);
    SA_FUSED_CASES(X)
#undef X
    return hipErrorInvalidValue;
}

}  // namespace sa

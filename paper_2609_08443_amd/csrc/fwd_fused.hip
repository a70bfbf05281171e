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
// over the four SIMDs' register files (accumulation registers).  The per-token
// sums over the M prototypes are reduced in registers (over the wave's 32x32
// tiles), across the 32 lanes of a row (DPP and permlane, no LDS), and across
// waves through LDS.
//
// Layouts: see tile_ops.h.  S is computed with tokens as rows, so its C layout
// (lane = prototype, register = token) is directly the A operand of the
// aggregation acc[m, j] += sum_t E[t, m] V'[t, j], with the k slots in the perm16
// token order; V' is staged row-major in LDS and read as the matching B operand
// with the transposing LDS load.  1/z is folded into V' (d values per token
// instead of M).  The shift enters the logits as the initial value of each
// score chain's accumulator (-c_t / scale per token row), so an exponential
// costs one multiply.
//
// Software pipeline, iteration j (two workgroup barriers):
//   prototype tile mt = 0 .. MT-1 of token tile j: its score chain, one matrix
//     instruction per step, each step also issuing one aggregation instruction
//     of token tile j-1 (prototype tile mt) and the exponentials of two (d=128)
//     or four (d=64) rows of prototype tile mt-1 of token tile j, so that the
//     matrix core and the VALU work side by side
//   exponentials of the last prototype tile; per-token partial sums to LDS;
//   stage K(j+1) into the other K buffer
//   --- barrier ---
//   z of tile j (one LDS round trip also gives each thread the sums of the
//   tokens whose V chunks it stages); the next tile's first operands; stage
//   V(j)/z; then the lse stores and the global loads of K(j+2), V(j+1), so
//   that the staging's wait for V(j) covers none of them
//   --- barrier ---
// Iteration 0 aggregates zero weights and the last iteration exponentiates a
// tile of clamped rows past the range (finite, masked out), so every iteration
// runs the same code.
#include "reduce_ops.h"
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

using namespace tile;

constexpr float kLn2 = 0.6931471805599453f;
// z below this means the shift was too far above the largest logit
constexpr float kUnderflowZ = 5.421010862427522e-20f;  // 2^-64
// relative margin on the bound for the rounding of the fp32 norms and logits
constexpr float kBoundMargin = 1.0f + 1.0f / 1024.0f;

// One step of the pipelined tile loop: one matrix instruction of the score
// chain that accumulates the next 32x32 logits tile into sn (VGPRs), one
// aggregation instruction acc += e^T v of the previous token tile (accumulation
// registers) and, with ROWS > 0, ROWS rows of the current logits tile
// exponentiated, e = 2^(s * ks), added into their sums and packed to bf16.  The
// VALU work is independent of both matrix instructions, so it issues while the
// matrix core runs.  Each exponential's first use is at least one instruction
// after it (the transcendental forwarding gap).  No wait states precede the
// matrix instructions: their operands are written by LDS loads or by other
// matrix instructions, and the weights e by the VALU a whole pipeline region
// or more earlier.
template <int ROWS>
__device__ inline void pipe_step(f32x16& sn, const bf16x8& k, const bf16x8& b, f32x16& acc, const bf16x8& e,
                                 const bf16x8& v, const float* s, float ks, float* z, uint32_t* ep) {
    if constexpr (ROWS == 0) {
        asm volatile(
            "v_mfma_f32_32x32x16_bf16 %[sn], %[k], %[b], %[sn]\n\t"
            "v_mfma_f32_32x32x16_bf16 %[acc], %[e], %[v], %[acc]"
            : [sn] "+v"(sn), [acc] "+a"(acc)
            : [k] "v"(k), [b] "v"(b), [e] "v"(e), [v] "v"(v));
    } else if constexpr (ROWS == 2) {
        float t0, t1;
        asm volatile(
            "v_mfma_f32_32x32x16_bf16 %[sn], %[k], %[b], %[sn]\n\t"
            "v_mul_f32 %[t0], %[s0], %[ks]\n\tv_mul_f32 %[t1], %[s1], %[ks]\n\t"
            "v_exp_f32 %[t0], %[t0]\n\tv_exp_f32 %[t1], %[t1]\n\t"
            "v_mfma_f32_32x32x16_bf16 %[acc], %[e], %[v], %[acc]\n\t"
            "v_add_f32 %[z0], %[z0], %[t0]\n\tv_add_f32 %[z1], %[z1], %[t1]\n\t"
            "v_cvt_pk_bf16_f32 %[ep], %[t0], %[t1]"
            : [sn] "+v"(sn), [acc] "+a"(acc), [t0] "=&v"(t0), [t1] "=&v"(t1), [z0] "+v"(z[0]),
              [z1] "+v"(z[1]), [ep] "=&v"(ep[0])
            : [k] "v"(k), [b] "v"(b), [e] "v"(e), [v] "v"(v), [s0] "v"(s[0]), [s1] "v"(s[1]), [ks] "v"(ks));
    } else {
        static_assert(ROWS == 4, "rows per step");
        float t0, t1, t2, t3;
        asm volatile(
            "v_mfma_f32_32x32x16_bf16 %[sn], %[k], %[b], %[sn]\n\t"
            "v_mul_f32 %[t0], %[s0], %[ks]\n\tv_mul_f32 %[t1], %[s1], %[ks]\n\t"
            "v_mul_f32 %[t2], %[s2], %[ks]\n\tv_mul_f32 %[t3], %[s3], %[ks]\n\t"
            "v_exp_f32 %[t0], %[t0]\n\tv_exp_f32 %[t1], %[t1]\n\t"
            "v_exp_f32 %[t2], %[t2]\n\tv_exp_f32 %[t3], %[t3]\n\t"
            "v_mfma_f32_32x32x16_bf16 %[acc], %[e], %[v], %[acc]\n\t"
            "v_add_f32 %[z0], %[z0], %[t0]\n\tv_add_f32 %[z1], %[z1], %[t1]\n\t"
            "v_add_f32 %[z2], %[z2], %[t2]\n\tv_add_f32 %[z3], %[z3], %[t3]\n\t"
            "v_cvt_pk_bf16_f32 %[ep0], %[t0], %[t1]\n\tv_cvt_pk_bf16_f32 %[ep1], %[t2], %[t3]"
            : [sn] "+v"(sn), [acc] "+a"(acc), [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3),
              [z0] "+v"(z[0]), [z1] "+v"(z[1]), [z2] "+v"(z[2]), [z3] "+v"(z[3]), [ep0] "=&v"(ep[0]),
              [ep1] "=&v"(ep[1])
            : [k] "v"(k), [b] "v"(b), [e] "v"(e), [v] "v"(v), [s0] "v"(s[0]), [s1] "v"(s[1]), [s2] "v"(s[2]),
              [s3] "v"(s[3]), [ks] "v"(ks));
    }
}

// sum of the squares of eight bf16 values, two per packed dot product
// (exact products, fp32 sums), in two independent chains
__device__ inline float sumsq8_dot(uint4 v) {
    using b2 = __bf16 __attribute__((ext_vector_type(2)));
    const b2 x = __builtin_bit_cast(b2, v.x), y = __builtin_bit_cast(b2, v.y);
    const b2 z = __builtin_bit_cast(b2, v.z), u = __builtin_bit_cast(b2, v.w);
    const float s0 = __builtin_amdgcn_fdot2_f32_bf16(z, z, __builtin_amdgcn_fdot2_f32_bf16(x, x, 0.f, false), false);
    const float s1 = __builtin_amdgcn_fdot2_f32_bf16(u, u, __builtin_amdgcn_fdot2_f32_bf16(y, y, 0.f, false), false);
    return s0 + s1;
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
    static constexpr int OFF_SUM = OFF_V + V_BYTES;      // [32][NW] partial sums (bound path)
    static constexpr int OFF_MAX = OFF_SUM + RED_BYTES;  // [NW][32] partial maxima (exact path)
    static constexpr int OFF_SUM2 = OFF_MAX + RED_BYTES; // [32][NW] partial sums (exact path)
    static constexpr int OFF_KN = OFF_SUM2 + RED_BYTES;  // [2][32] token norms
    static constexpr int OFF_NB = OFF_KN + 2 * 32 * 4;   // [2][32] score-chain inits, -c_t / scale
    static constexpr int OFF_PN = OFF_NB + 2 * 32 * 4;   // [NW] prototype norm maxima
    static constexpr int OFF_SH = OFF_PN + 16 * 4;       // [32] exact-path shifts
    static constexpr int LDS = OFF_SH + 32 * 4;
};

template <int D, int MW, int NW>
__global__ __launch_bounds__(NW * 64, 1) void fwd_fused_kernel(FusedFwdArgs a) {
    using C = Cfg<D, MW, NW>;
    constexpr int MT = C::MT, KS = C::KS, JT = C::JT;
    constexpr int ROWS = 16 / KS;   // rows of a logits tile exponentiated per pipeline step
    // The next tile's first operands are read right after the per-token sums'
    // LDS round trip with four or more prototype tiles per wave, after the
    // bound check (and the rare exact path) with fewer: measured, the early
    // reads pay with the longer tile loops and cost with the short ones.
    constexpr bool EARLY_OPS = MT >= 4;
    static_assert(KS == 2 * JT, "one aggregation instruction per score-chain step");
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* Ps = reinterpret_cast<uint16_t*>(smem);
    uint16_t* Kbuf = reinterpret_cast<uint16_t*>(smem + C::OFF_K);
    uint16_t* Vt = reinterpret_cast<uint16_t*>(smem + C::OFF_V);
    float* red_sum = reinterpret_cast<float*>(smem + C::OFF_SUM);
    float* red_max = reinterpret_cast<float*>(smem + C::OFF_MAX);
    float* red_sum2 = reinterpret_cast<float*>(smem + C::OFF_SUM2);
    float* knorm = reinterpret_cast<float*>(smem + C::OFF_KN);
    float* kinit = reinterpret_cast<float*>(smem + C::OFF_NB);
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
        // (segments of the work list are never empty)
        if (b < 0 || b >= a.B || h < 0 || h >= a.H || t0 < 0 || t1 <= t0 || t1 > a.T) continue;

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
        // shift of token t: c_t = cb |K_t| >= max_m scale <K_t, P_m>; the score
        // chains start from -c_t / scale = -pm |K_t|
        const float pm = pmax * kBoundMargin;
        const float cb = a.scale * pm;

        f32x16 acc[MT][JT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][jt][r] = 0.f;

        // global tile loads into registers: 32-bit per-lane offsets from the
        // segment's first row.  Rows past the end of the range read its last token
        // (their V is zeroed at staging), so every load is issued unconditionally,
        // also for the tiles past the range, and the compiler's waits for one set
        // of loads never include the next set.
        uint4 kreg[C::NLD], vreg[C::NLD];
        static_assert(C::LD_CHUNKS % C::THREADS == 0, "every thread loads whole chunks");
        const int64_t seg_row0 = ((int64_t)t0 * a.H + h) * D;
        auto load_rows = [&](const uint16_t* X, int ts, uint4 (&dst)[C::NLD]) {
            const uint16_t* Xb = X + seg_row0;
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                const int idx = tid + i * C::THREADS;
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                const int row = min(ts + tok, t1 - 1) - t0;
                const uint32_t off = (uint32_t)row * row_stride + (uint32_t)(ch * 8);
                dst[i] = *reinterpret_cast<const uint4*>(Xb + off);
            }
        };
        // K tile (from kreg) into LDS buffer kb, with the token norms and chain
        // inits.  Every lane of a row's KCH consecutive lanes computes the row's
        // norm and stores it (the same value to the same word), so there is no
        // branch; the chunks' squares are summed in independent pairs.
        auto stage_k = [&](int kb) {
            uint16_t* Kd = Kbuf + kb * (32 * D);
            float ss[C::NLD];
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                int idx = tid + i * C::THREADS;
                asm volatile("" : "+v"(idx));
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                *reinterpret_cast<uint4*>(Kd + swz<D>(tok, ch)) = kreg[i];
                ss[i] = sumsq8_dot(kreg[i]);
            }
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) ss[i] = group_sum<C::KCH>(ss[i]);
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                const int tok = (tid + i * C::THREADS) / C::KCH;
                const float kn = __builtin_sqrtf(ss[i]);
                knorm[kb * 32 + tok] = kn;
                kinit[kb * 32 + tok] = -pm * kn;
            }
        };
        auto read_bp = [&](bf16x8* bp, int mt) {
            const int prow = w * MW + mt * 32 + l32;
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) bp[kk] = lds_b128(Ps, swz<D>(prow, 2 * kk + hl));
        };
        // one 32x32 logits tile (no shift), written out so that it lands in VGPRs
        // (exact-maximum path only)
        auto s_chain = [&](const bf16x8* kop, const bf16x8* bp) {
            f32x16 s;
            __builtin_amdgcn_sched_barrier(0);
            asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(kop[0]), "v"(bp[0]));
#pragma unroll
            for (int kk = 1; kk < KS; ++kk)
                asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(kop[kk]), "v"(bp[kk]));
            asm volatile("s_nop 15\n\ts_nop 15" : "+v"(s));
            return s;
        };
        auto s_tile = [&](const bf16x8* kop, int mt) {
            bf16x8 bp[KS];
            read_bp(bp, mt);
            return s_chain(kop, bp);
        };
        // the chain init of a logits tile: -c_t / scale for this lane's 16 rows
        auto chain_init = [&](int kb) {
            f32x16 x;
            const float* src = kinit + kb * 32 + 4 * hl;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 q = *reinterpret_cast<const float4*>(src + 8 * g);
                x[4 * g] = q.x;
                x[4 * g + 1] = q.y;
                x[4 * g + 2] = q.z;
                x[4 * g + 3] = q.w;
            }
            return x;
        };

        const int ntiles = (t1 - t0 + 31) / 32;
        constexpr int NR = 4;   // P operands in flight (a ring, NR chain steps ahead)
        auto p_op = [&](int q) {   // P operand of chain step q (prototype tile q / KS)
            return lds_b128(Ps, swz<D>(w * MW + (q / KS) * 32 + l32, 2 * (q % KS) + hl));
        };
        // operands of a tile's first chain steps: K as A operands, the ring's
        // first NR P operands, and the chain init
        bf16x8 kop[KS], bp[NR];
        f32x16 sn;
        auto read_tile_ops = [&](int kb) {
            const uint16_t* Ks = Kbuf + kb * (32 * D);
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
                kop[kk] = lds_b128(Ks, swz<D>(l32, 2 * kk + hl));
                if (kk < NR) bp[kk] = p_op(kk);
            }
            sn = chain_init(kb);
        };

        // prologue: K(0) staged, K(1) and V(0) in flight, zero weights and V' for
        // iteration 0's aggregation, tile 0's operands read
        load_rows(a.K, t0, kreg);
        stage_k(0);
        load_rows(a.K, t0 + 32, kreg);
        load_rows(a.V, t0, vreg);
        bf16x8 eop[MT][2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) eop[mt][0] = eop[mt][1] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
#pragma unroll
        for (int i = 0; i < C::NLD; ++i) {
            const int idx = tid + i * C::THREADS;
            *reinterpret_cast<uint4*>(Vt + swz<D>(idx / C::KCH, idx % C::KCH)) = make_uint4(0, 0, 0, 0);
        }
        __syncthreads();
        read_tile_ops(0);

        for (int j = 0; j <= ntiles; ++j) {
            const int ts = t0 + j * 32;   // token tile j (past the range when j == ntiles)
            const int kb = j & 1;

            // ---- V'(j-1) as the aggregation's B operands (K(j), the first P
            // operands and the chain init were read before the last barrier)
            bf16x8 vop[JT][2];
#pragma unroll
            for (int jt = 0; jt < JT; ++jt) {
                vop[jt][0] = lds_tr_tokens<D>(Vt, lane, jt, 0);
                vop[jt][1] = lds_tr_tokens<D>(Vt, lane, jt, 1);
            }
            f32x16 sp, snx;
            float rsum[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) rsum[r] = 0.f;

            // ---- prototype tiles: score chain of mt (tile j) + aggregation of mt
            // (tile j-1) + exponentials of mt-1 (tile j)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                uint32_t ep[8];
                if (mt > 0) {
                    sp = sn;
                    sn = snx;
                    // the previous chain's results are read from the first step on
                    asm volatile("s_nop 4" : "+v"(sp));
                }
#pragma unroll
                for (int kk = 0; kk < KS; ++kk) {
                    __builtin_amdgcn_sched_barrier(0);
                    const bf16x8& ev = eop[mt][kk & 1];
                    const bf16x8& vv = vop[kk >> 1][kk & 1];
                    const int q = mt * KS + kk;
                    bf16x8& pb = bp[q % NR];
                    if (mt == 0) {
                        pipe_step<0>(sn, kop[kk], pb, acc[mt][kk >> 1], ev, vv, nullptr, ks2, nullptr, nullptr);
                    } else {
                        float sr[ROWS];
#pragma unroll
                        for (int r = 0; r < ROWS; ++r) sr[r] = sp[ROWS * kk + r];
                        pipe_step<ROWS>(sn, kop[kk], pb, acc[mt][kk >> 1], ev, vv, sr, ks2, rsum + ROWS * kk,
                                        ep + (ROWS / 2) * kk);
                    }
                    if (q + NR < MT * KS) pb = p_op(q + NR);
                    if (mt + 1 < MT && kk == KS - 3) snx = chain_init(kb);
                }
                __builtin_amdgcn_sched_barrier(0);
                if (mt > 0) {
                    eop[mt - 1][0] = __builtin_bit_cast(bf16x8, make_uint4(ep[0], ep[1], ep[2], ep[3]));
                    eop[mt - 1][1] = __builtin_bit_cast(bf16x8, make_uint4(ep[4], ep[5], ep[6], ep[7]));
                }
            }
            // ---- exponentials of the last prototype tile, the per-token partial
            // sums, and K(j+1) into the other buffer (K(j-1)'s) with its norms: three
            // independent chains the compiler interleaves
            asm volatile("s_nop 7" : "+v"(sn));
            {
                float e[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    e[r] = __builtin_amdgcn_exp2f(sn[r] * ks2);
                    rsum[r] += e[r];
                }
                eop[MT - 1][0] = pack8(e);
                eop[MT - 1][1] = pack8(e + 8);
            }
            stage_k(kb ^ 1);
            {
                const float z = half_sum16(rsum, l32);
                // the store address is rebuilt here from the lane id rather than
                // kept live through the tile loop (it would be spilled)
                int ln = tid;
                asm volatile("" : "+v"(ln));
                if ((ln & 1) == 0)
                    reinterpret_cast<float*>(smem + C::OFF_SUM)[srow((ln & 31) >> 1, (ln >> 5) & 1) * NW + (ln >> 6)] = z;
            }
            __syncthreads();  // B_z

            // ---- per-token sums, in one LDS round trip: lane t of each half gets
            // token t's total, and each thread the totals of the tokens of its V
            // chunks; the next tile's operands are read meanwhile
            static_assert(NW == 4, "one 16-byte read per token");
            auto tok_z = [&](const float* part, int tok) {
                const float4 q = *reinterpret_cast<const float4*>(part + tok * NW);
                return (q.x + q.y) + (q.z + q.w);
            };
            const int tt = l32;
            float zt = tok_z(red_sum, tt);
            float zv[C::NLD];
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) zv[i] = tok_z(red_sum, (tid + i * C::THREADS) / C::KCH);
            const float kn_t = knorm[kb * 32 + tt];
            if constexpr (EARLY_OPS) read_tile_ops(kb ^ 1);
            // tile-uniform check that the bound did not underflow any z_t
            const bool exact = __builtin_amdgcn_ballot_w64(zt < kUnderflowZ && ts + tt < t1) != 0;
            float c_t = cb * kn_t;
            if (exact) {
                // rare: exact per-token max over the prototypes, then the exponentials
                // again (rsum holds the running max first); with the next tile's
                // operands already read, the K operands of tile j are read again
                // (those of tile j+1 are back afterwards)
                if constexpr (EARLY_OPS) {
#pragma unroll
                    for (int kk = 0; kk < KS; ++kk)
                        kop[kk] = lds_b128(Kbuf + kb * (32 * D), swz<D>(l32, 2 * kk + hl));
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) rsum[r] = -INFINITY;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
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
                float nb[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    nb[r] = shift_s[srow(r, hl)];
                    rsum[r] = 0.f;
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
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
                    for (int r = 0; r < 16; ++r) red_sum2[srow(r, hl) * NW + w] = rsum[r];
                }
                __syncthreads();
                zt = tok_z(red_sum2, tt);
#pragma unroll
                for (int i = 0; i < C::NLD; ++i) zv[i] = tok_z(red_sum2, (tid + i * C::THREADS) / C::KCH);
                c_t = -shift_s[tt] / kLog2e;
                if constexpr (EARLY_OPS) read_tile_ops(kb ^ 1);
            }
            if constexpr (!EARLY_OPS) read_tile_ops(kb ^ 1);

            // ---- stage V / z (row-major; the aggregation reads it transposed).
            // z >= 2^-64 here (the exact path's z >= 1): the hardware reciprocal
            // (1 ulp) is as good as a division before the bf16 rounding of V / z.
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                int idx = tid + i * C::THREADS;
                asm volatile("" : "+v"(idx));  // addresses built here, not hoisted
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                const float inv = ts + tok < t1 ? __builtin_amdgcn_rcpf(zv[i]) : 0.0f;
                *reinterpret_cast<uint4*>(Vt + swz<D>(tok, ch)) = scale8(vreg[i], inv);
            }
            // ---- then the lse, the K of tile j+2 (kreg was staged before B_z) and the
            // V of tile j+1: issued after the staging, so that its wait for V(j)
            // includes none of them.  The loads are issued in every iteration (rows
            // past the range are clamped), so each wait for them is an exact count.
            static_assert(NW * 8 == 32, "four waves of eight tokens");
            if ((lane >> 3) == w && a.lse && ts + tt < t1)   // lanes 8w .. 8w+7 write tokens 8w .. 8w+7
                a.lse[(int64_t)(ts + tt) * a.H + h] = c_t + __builtin_amdgcn_logf(zt) * kLn2;
            load_rows(a.K, ts + 64, kreg);
            load_rows(a.V, ts + 32, vreg);
            // B_v: V' staged, the next tile's operands read; the loads stay in flight
            lds_barrier();
        }

        // ---- flush: the whole sketch of the pair, or this segment's partial
        float* out = split ? a.partials + k * MD : a.sketch + ((int64_t)b * a.H + h) * MD;
        uint32_t lane_off = (uint32_t)((w * MW + 4 * hl) * D + l32);
        // keep the per-store addresses from being hoisted out of the loops (they
        // would stay live in registers through the whole tile loop)
        asm volatile("" : "+v"(lane_off));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < JT; ++jt)
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

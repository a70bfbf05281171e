// Token-wise normalised variant of the sketching step on gfx950: the weights are
// normalised over each user's tokens for every prototype (the alternative the
// paper compares SA's prototype-wise normalisation with; appendix on
// prototype-wise normalisation, Table 1):
//
//   s_t = scale K_t . P_m,   w_t = exp(s_t) / sum_t' exp(s_t'),
//   sketch[b,h,m,:] = sum_t w_t V_t,   lse_m[b,h,m] = log sum_t exp(s_t).
//
// This is attention with the M prototypes as queries over a user's tokens, so it
// runs as an online softmax over token tiles: a running maximum and sum per
// prototype, with the accumulator rescaled when the maximum rises.  Because the
// normalisation is per prototype, a wave that owns a prototype owns its whole
// softmax: no reduction across waves.  A user cut across work-list ranges
// leaves one unnormalised partial per range with its (max, sum); the merge
// rescales them by the common maximum (the log-sum-exp merge).
//
// Kernels:
//   tw_generic_kernel   one wave per (user, head, prototype), fp32 arithmetic
//                       (fp32 or bf16 inputs); the plain correctness path.
//   tw_fused_kernel     bf16 matrix cores: workgroup = (range, 32*NW prototypes),
//                       each wave 32 prototypes held in registers as B operands;
//                       token tiles of 32 double-buffered in LDS; S = K P^T and the
//                       aggregation E^T V on v_mfma_f32_32x32x16_bf16 (V^T read
//                       with the transposing LDS load).
//   tw_merge_kernel     one wave per (user, head, prototype) row: rescale-and-add
//                       of the partials of a split user, or zero / -inf for an
//                       empty one.
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

using namespace tile;

constexpr float kLn2 = 0.6931471805599453f;

__device__ inline float wave_sum64(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ inline float xhalf_max(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float xhalf_add(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ------------------------------------------------------------------ plain path
template <bool BF16>
__device__ inline float ld(const void* base, int64_t i) {
    if constexpr (BF16) return bf16_lo((uint32_t)reinterpret_cast<const uint16_t*>(base)[i]);
    else return reinterpret_cast<const float*>(base)[i];
}

// one wave per (user, head, prototype); lane j owns columns j and j + 64
template <bool BF16>
__global__ __launch_bounds__(64) void tw_generic_kernel(const void* K, const void* V, const void* P,
                                                        const int64_t* __restrict__ offsets, int64_t B,
                                                        int32_t H, int32_t M, int32_t d, float scale,
                                                        float* __restrict__ sketch,
                                                        float* __restrict__ lse_m) {
    const int64_t pair = blockIdx.x / M;   // b*H + h
    const int m = (int)(blockIdx.x % M);
    const int64_t b = pair / H;
    const int h = (int)(pair % H);
    const int j0 = threadIdx.x, j1 = threadIdx.x + 64;
    const int64_t pbase = ((int64_t)h * M + m) * d;
    const float p0 = j0 < d ? ld<BF16>(P, pbase + j0) : 0.f;
    const float p1 = j1 < d ? ld<BF16>(P, pbase + j1) : 0.f;
    const int64_t t0 = offsets[b], t1 = offsets[b + 1];
    float mu = -INFINITY, l = 0.f, a0 = 0.f, a1 = 0.f;
    for (int64_t t = t0; t < t1; ++t) {
        const int64_t row = (t * H + h) * d;
        const float k0 = j0 < d ? ld<BF16>(K, row + j0) : 0.f;
        const float k1 = j1 < d ? ld<BF16>(K, row + j1) : 0.f;
        const float s = scale * wave_sum64(k0 * p0 + k1 * p1);
        const float mn = fmaxf(mu, s);
        const float al = __expf(mu - mn);      // 0 on the first token
        const float e = __expf(s - mn);
        l = l * al + e;
        const float v0 = j0 < d ? ld<BF16>(V, row + j0) : 0.f;
        const float v1 = j1 < d ? ld<BF16>(V, row + j1) : 0.f;
        a0 = a0 * al + e * v0;
        a1 = a1 * al + e * v1;
        mu = mn;
    }
    float* out = sketch + (pair * M + m) * (int64_t)d;
    const float rl = l > 0.f ? 1.0f / l : 0.f;
    if (j0 < d) out[j0] = a0 * rl;
    if (j1 < d) out[j1] = a1 * rl;
    if (lse_m && threadIdx.x == 0) lse_m[pair * M + m] = l > 0.f ? mu + __logf(l) : -INFINITY;
}

// ------------------------------------------------------------------ fused path
template <int D, int NW_>
struct TwCfg {
    static constexpr int NW = NW_;
    static constexpr int THREADS = NW * 64;
    static constexpr int MP = 32 * NW;                     // prototypes of one part
    static constexpr int KS = D / 16;
    static constexpr int JT = D / 32;
    static constexpr int KCH = D / 8;
    static constexpr int LD_CHUNKS = 32 * KCH;
    static constexpr int NCH = (LD_CHUNKS + THREADS - 1) / THREADS;
    static constexpr int TILE = 32 * D * 2;                // one [32][D] bf16 token tile
    static constexpr int OFF_K = 0;                        // 2 x K tiles
    static constexpr int OFF_V = OFF_K + 2 * TILE;         // 2 x V tiles
    static constexpr int OFF_ROW = OFF_V + 2 * TILE;       // [NW][32] per-prototype factors
    static constexpr int LDS = OFF_ROW + NW * 32 * 4;
};

struct TwArgs {
    const uint16_t* K;
    const uint16_t* V;
    const uint16_t* P;
    const int32_t* items;
    const int32_t* wg_start;
    int64_t n_ranges;
    int64_t max_items;
    int64_t T;
    int32_t B, H, M;
    int32_t parts;
    float scale;
    float* sketch;
    float* lse_m;       // may be null
    float* partials;    // [max_items][M][D]: unnormalised partial of a split user
    float* stats;       // [max_items][M][2]: (max in log2 units, sum)
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64, 1) void tw_fused_kernel(TwArgs a) {
    using C = TwCfg<D, NW>;
    constexpr int KS = C::KS, JT = C::JT;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    float* rowf = reinterpret_cast<float*>(smem + C::OFF_ROW);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int l32 = lane & 31, hl = lane >> 5;

    // workgroup -> (range, part), the parts of a range back to back on one XCD
    const int64_t xcd = blockIdx.x % 8, jx = blockIdx.x / 8;
    const int part = (int)(jx % a.parts);
    const int64_t ix = jx / a.parts;
    const int64_t q8 = a.n_ranges / 8, r8 = a.n_ranges % 8;
    if (ix >= q8 + (xcd < r8 ? 1 : 0)) return;
    const int64_t range = xcd * q8 + (xcd < r8 ? xcd : r8) + ix;
    const int64_t k0 = a.wg_start[range], k1 = a.wg_start[range + 1];
    if (k0 < 0 || k1 < k0 || k1 > a.max_items) return;

    const float ks2 = a.scale * kLog2e;
    const int64_t MD = (int64_t)a.M * D;
    const uint32_t row_stride = (uint32_t)a.H * D;
    const int prow = part * C::MP + w * 32 + l32;   // this lane's prototype (S columns)

    // per-wave exchange of one factor per prototype, from the S layout (lane =
    // prototype) to the accumulator layout (register r = prototype srow(r, hl))
    auto to_rows = [&](float f, float (&out)[16]) __attribute__((always_inline)) {
        if (hl == 0) rowf[w * 32 + l32] = f;
        wave_lds_order();
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float4 v = *reinterpret_cast<const float4*>(rowf + w * 32 + 8 * g + 4 * hl);
            out[4 * g + 0] = v.x;
            out[4 * g + 1] = v.y;
            out[4 * g + 2] = v.z;
            out[4 * g + 3] = v.w;
        }
        wave_lds_order();
    };

    for (int64_t k = k0; k < k1; ++k) {
        const int32_t* it = a.items + k * IT_WORDS;
        const int b = it[IT_B], h = it[IT_H], t0 = it[IT_T0], t1 = it[IT_T1];
        const int split = it[IT_SPLIT];
        if (b < 0 || b >= a.B || h < 0 || h >= a.H || t0 < 0 || t1 < t0 || t1 > a.T) continue;

        // this wave's 32 prototypes as B operands, for the whole segment
        bf16x8 pop[KS];
        {
            const uint16_t* Pg = a.P + (int64_t)h * MD + (int64_t)prow * D;
#pragma unroll
            for (int kk = 0; kk < KS; ++kk)
                pop[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(Pg + 16 * kk + 8 * hl));
        }
        // Token tiles go global -> registers two tiles ahead (two register sets,
        // used alternately) -> LDS buffer.  Every fetch issues the same loads (rows
        // past the range read its last token, threads past the tile's chunks
        // reload a chunk they do not store), so the wait before a store counts
        // exactly the newer set's loads.  Rows past the range need no zeros: their
        // logits are masked to -inf, so their weights are 0 and their V is unused.
        struct Regs { u32x4 k[C::NCH], v[C::NCH]; };
        Regs ra, rb;
        auto fetch = [&](int ts, Regs& r) __attribute__((always_inline)) {
            const char* Kb = reinterpret_cast<const char*>(a.K + ((int64_t)t0 * a.H + h) * D);
            const char* Vb = reinterpret_cast<const char*>(a.V + ((int64_t)t0 * a.H + h) * D);
#pragma unroll
            for (int c = 0; c < C::NCH; ++c) {
                const int idx = (tid + c * C::THREADS) % C::LD_CHUNKS;
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                const int row = min(ts + tok, t1 - 1) - t0;
                const uint32_t off = ((uint32_t)row * row_stride + (uint32_t)(ch * 8)) * 2;
                r.k[c] = *reinterpret_cast<const u32x4*>(Kb + off);
                r.v[c] = *reinterpret_cast<const u32x4*>(Vb + off);
            }
        };
        auto store = [&](int buf, const Regs& r) __attribute__((always_inline)) {
            uint16_t* Kd = reinterpret_cast<uint16_t*>(smem + C::OFF_K + buf * C::TILE);
            uint16_t* Vd = reinterpret_cast<uint16_t*>(smem + C::OFF_V + buf * C::TILE);
#pragma unroll
            for (int c = 0; c < C::NCH; ++c) {
                const int idx = tid + c * C::THREADS;
                if (idx < C::LD_CHUNKS) {
                    const int tok = idx / C::KCH, ch = idx % C::KCH;
                    *reinterpret_cast<u32x4*>(Kd + swz<D>(tok, ch)) = r.k[c];
                    *reinterpret_cast<u32x4*>(Vd + swz<D>(tok, ch)) = r.v[c];
                }
            }
        };
        const bool any = t1 > t0;   // (an empty segment still writes its zero output)
        if (any) {
            fetch(t0, ra);
            fetch(t0 + 32, rb);
        }
        __syncthreads();  // the previous segment is done with every LDS buffer
        if (any) store(0, ra);
        __syncthreads();

        f32x16 acc[JT];
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[jt][r] = 0.f;
        float mu = -INFINITY;   // running max of this lane's prototype, log2 units
        float lsum = 0.f;       // running sum over this lane's 16 token rows per tile
        // Wait here for the held operands.  Otherwise the compiler's load-counter
        // waits for them inside the loop also wait for each iteration's prefetch
        // of the next tile, issued after them, which then lands before the
        // tile's logits are done.
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) asm volatile("" ::"v"(pop[kk]));

        // tile at ts in LDS buffer buf; the next tile is in `nxt` (stored at the end
        // of this step into the other buffer), the one after it fetched into `far`
        auto step = [&](int ts, int buf, Regs& far, const Regs& nxt) __attribute__((always_inline)) {
            const bool more = ts + 32 < t1;
            fetch(ts + 64, far);
            const uint16_t* Ks = reinterpret_cast<const uint16_t*>(smem + C::OFF_K + buf * C::TILE);
            const uint16_t* Vs = reinterpret_cast<const uint16_t*>(smem + C::OFF_V + buf * C::TILE);
            // S[t, m]: lane = prototype, register r = token srow(r, hl)
            f32x16 s;
#pragma unroll
            for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
            for (int kk = 0; kk < KS; ++kk)
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_b128(Ks, swz<D>(l32, 2 * kk + hl)), pop[kk], s, 0, 0, 0);
            float x[16];
            float tmax = -INFINITY;
            const bool ragged = ts + 32 > t1;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                x[r] = s[r] * ks2;
                if (ragged && ts + srow(r, hl) >= t1) x[r] = -INFINITY;   // past the user's end
                tmax = fmaxf(tmax, x[r]);
            }
            tmax = xhalf_max(tmax);
            const float mnew = fmaxf(mu, tmax);
            // rescale the accumulator rows whose maximum rose (wave-uniform branch)
            if (__builtin_amdgcn_ballot_w64(mnew > mu) != 0) {
                const float al = exp2f(mu - mnew);     // 0 when mu = -inf
                lsum *= al;
                float alr[16];
                to_rows(al, alr);
#pragma unroll
                for (int jt = 0; jt < JT; ++jt)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[jt][r] *= alr[r];
                mu = mnew;
            }
            float e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                e[r] = __builtin_amdgcn_exp2f(x[r] - mu);
                lsum += e[r];
            }
            const bf16x8 e0 = pack8(e), e1 = pack8(e + 8);
            // acc[m, j] += E^T[m, t] V[t, j]
#pragma unroll
            for (int jt = 0; jt < JT; ++jt) {
                acc[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(e0, lds_tr_tokens<D>(Vs, lane, jt, 0), acc[jt], 0, 0, 0);
                acc[jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(e1, lds_tr_tokens<D>(Vs, lane, jt, 1), acc[jt], 0, 0, 0);
            }
            if (more) store(buf ^ 1, nxt);
            __syncthreads();
        };
        // two tiles per trip; the exits sit after each step, so that the path back
        // to the top always comes from the second step (whose pending loads fill
        // the other register set)
        if (any) {
            for (int ts = t0;; ts += 64) {
                step(ts, 0, ra, rb);
                if (ts + 32 >= t1) break;
                step(ts + 32, 1, rb, ra);
                if (ts + 64 >= t1) break;
            }
        }
        const float ltot = xhalf_add(lsum);   // both halves hold the same prototype
        // rows of this wave: prototypes part*MP + w*32 + srow(r, hl), columns jt*32 + l32
        uint32_t lane_off = (uint32_t)((part * C::MP + w * 32 + 4 * hl) * D + l32);
        asm volatile("" : "+v"(lane_off));
        if (!split) {
            float rl[16];
            to_rows(ltot > 0.f ? 1.0f / ltot : 0.f, rl);
            float* out = a.sketch + ((int64_t)b * a.H + h) * MD;
#pragma unroll
            for (int jt = 0; jt < JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    out[lane_off + (uint32_t)((8 * (r >> 2) + (r & 3)) * D + jt * 32)] = acc[jt][r] * rl[r];
            if (a.lse_m && hl == 0)
                a.lse_m[((int64_t)b * a.H + h) * a.M + prow] = mu * kLn2 + __logf(ltot);
        } else {
            float* out = a.partials + k * MD;
#pragma unroll
            for (int jt = 0; jt < JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    out[lane_off + (uint32_t)((8 * (r >> 2) + (r & 3)) * D + jt * 32)] = acc[jt][r];
            if (hl == 0) {
                a.stats[(k * a.M + prow) * 2 + 0] = mu;
                a.stats[(k * a.M + prow) * 2 + 1] = ltot;
            }
        }
    }
}

// One wave per (user, head, prototype) row: the (max, sum) of the row's segments
// are read once, then lane j rescales and adds columns j and j + 64.
__global__ __launch_bounds__(256) void tw_merge_kernel(const int32_t* __restrict__ pair_start, int64_t B,
                                                       int32_t H, int32_t M, int32_t d, int64_t max_items,
                                                       const float* __restrict__ partials,
                                                       const float* __restrict__ stats,
                                                       float* __restrict__ sketch, float* __restrict__ lse_m) {
    const int64_t p = blockIdx.x;   // head-major pair h*B + b
    int64_t s0 = pair_start[p], s1 = pair_start[p + 1];
    s0 = s0 < 0 ? 0 : (s0 > max_items ? max_items : s0);
    s1 = s1 < s0 ? s0 : (s1 > max_items ? max_items : s1);
    if (s1 - s0 == 1) return;       // written directly by the fused kernel
    const int64_t m = (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6);
    if (m >= M) return;
    const int lane = threadIdx.x & 63;
    const int64_t h = p / B, b = p % B;
    const int64_t MD = (int64_t)M * d;
    // (unrolled so that the loads of several segments are in flight at once; the
    // sums keep segment order)
    float mx = -INFINITY;
#pragma unroll 8
    for (int64_t k = s0; k < s1; ++k) mx = fmaxf(mx, stats[(k * M + m) * 2]);
    float l = 0.f, v0 = 0.f, v1 = 0.f;
#pragma unroll 4
    for (int64_t k = s0; k < s1; ++k) {
        const float f = exp2f(stats[(k * M + m) * 2] - mx);
        l += f * stats[(k * M + m) * 2 + 1];
        const float* row = partials + k * MD + m * d;
        v0 += f * row[lane];
        if (lane + 64 < d) v1 += f * row[lane + 64];
    }
    float* out = sketch + (b * H + h) * MD + m * d;
    const float rl = l > 0.f ? 1.0f / l : 0.f;
    out[lane] = v0 * rl;
    if (lane + 64 < d) out[lane + 64] = v1 * rl;
    if (lse_m && lane == 0) lse_m[(b * H + h) * M + m] = l > 0.f ? mx * kLn2 + __logf(l) : -INFINITY;
}

template <int D, int NW>
hipError_t launch_tw_inst(const TwArgs& a0, hipStream_t stream) {
    using C = TwCfg<D, NW>;
    auto kern = tw_fused_kernel<D, NW>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    TwArgs a = a0;
    a.parts = a.M / C::MP;
    const int64_t per_xcd = (a.n_ranges + 7) / 8;
    hipLaunchKernelGGL(kern, dim3((unsigned)(8 * per_xcd * a.parts)), dim3(C::THREADS), C::LDS, stream, a);
    return hipGetLastError();
}

}  // namespace

bool tokenwise_fused_supported(int32_t M, int32_t d) {
    return (d == 64 || d == 128) && M % 128 == 0 && M <= 4096;
}

hipError_t launch_tokenwise_fused(const int32_t* items, const int32_t* wg_start, int64_t n_ranges,
                                  int64_t max_items, const void* K, const void* V, const void* P,
                                  int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                                  float* sketch, float* lse_m, float* partials, float* stats,
                                  hipStream_t stream) {
    if (n_ranges == 0) return hipSuccess;
    TwArgs a;
    a.K = reinterpret_cast<const uint16_t*>(K);
    a.V = reinterpret_cast<const uint16_t*>(V);
    a.P = reinterpret_cast<const uint16_t*>(P);
    a.items = items;
    a.wg_start = wg_start;
    a.n_ranges = n_ranges;
    a.max_items = max_items;
    a.T = T;
    a.B = (int32_t)B;
    a.H = H;
    a.M = M;
    a.parts = 1;
    a.scale = scale;
    a.sketch = sketch;
    a.lse_m = lse_m;
    a.partials = partials;
    a.stats = stats;
    // eight waves (256 prototypes per workgroup) when M allows, else four
    const bool eight = M % 256 == 0;
    if (d == 64) return eight ? launch_tw_inst<64, 8>(a, stream) : launch_tw_inst<64, 4>(a, stream);
    return eight ? launch_tw_inst<128, 8>(a, stream) : launch_tw_inst<128, 4>(a, stream);
}

hipError_t launch_tokenwise_merge(const int32_t* pair_start, int64_t B, int32_t H, int32_t M, int32_t d,
                                  int64_t max_items, const float* partials, const float* stats,
                                  float* sketch, float* lse_m, hipStream_t stream) {
    const int64_t npairs = (int64_t)H * B;
    if (npairs == 0) return hipSuccess;
    hipLaunchKernelGGL(tw_merge_kernel, dim3((unsigned)npairs, (unsigned)((M + 3) / 4)), dim3(256), 0, stream,
                       pair_start, B, H, M, d, max_items, partials, stats, sketch, lse_m);
    return hipGetLastError();
}

hipError_t launch_tokenwise_generic(const void* K, const void* V, const void* P, const int64_t* offsets,
                                    int64_t B, int32_t H, int32_t M, int32_t d, float scale, bool bf16,
                                    float* sketch, float* lse_m, hipStream_t stream) {
    const int64_t n = B * H * (int64_t)M;
    if (n == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(tw_generic_kernel<true>, dim3((unsigned)n), dim3(64), 0, stream, K, V, P, offsets, B,
                           H, M, d, scale, sketch, lse_m);
    else
        hipLaunchKernelGGL(tw_generic_kernel<false>, dim3((unsigned)n), dim3(64), 0, stream, K, V, P, offsets, B,
                           H, M, d, scale, sketch, lse_m);
    return hipGetLastError();
}

}  // namespace sa

// Fused bf16 forward of the SA sketching step on gfx950 matrix cores.
//
// Per token tile of 32 tokens of one (user, head) segment, without writing the
// T x M affinities anywhere (section 4.4, FlashSA: block-wise affinities,
// prototype-wise softmax statistics, aggregation into the sketch):
//
//   S   = K_tile . P^T                  32 x M, bf16 MFMA 32x32x16, fp32 accumulate
//   mu  = max over the M prototypes      per token (section 3.1: softmax over prototypes)
//   E   = exp(scale * (S - mu)),  z = sum_m E,  lse = scale*mu + log z
//   acc[M, d] += E^T . (V_tile / z)      bf16 MFMA, fp32 accumulate
//
// Workgroup = NW waves (one per SIMD); wave w owns prototypes
// [w*MW, (w+1)*MW) for both GEMMs, so the M x d fp32 accumulator is spread
// over the four SIMDs' register files.  The per-token max and sum over the M
// prototypes are reduced in registers (over the wave's 32x32 tiles), across
// the 32 lanes of a row, and across waves through LDS.
//
// Layouts (v_mfma_f32_32x32x16_bf16, checked on the device):
//   A operand: lane l holds row l%32, k = (l/32)*8 + 0..7
//   B operand: lane l holds col l%32, k = (l/32)*8 + 0..7
//   C/D      : lane l holds col l%32, rows 8*(r/4) + 4*(l/32) + r%4, r = 0..15
// S is computed with tokens as rows, so its C layout (lane = prototype,
// register = token) is directly the A operand of the aggregation
// acc[m, j] += sum_t E[t, m] V'[t, j] once the token index of the k slots is
// permuted accordingly; V' is staged in LDS transposed and in that permuted
// token order.  1/z is folded into V' (d values per token instead of M).
#include "sa_internal.h"

namespace sa {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 -> packed bf16x2 (round to nearest even), first value in the low half.
__device__ inline uint32_t pack_bf16x2(float a, float b) {
    bf16x2 v = __builtin_convertvector((f32x2){a, b}, bf16x2);
    return __builtin_bit_cast(uint32_t, v);
}

// LDS element offset (in bf16 units) of 16-byte chunk c of row r of a matrix
// with `cols` bf16 per row; chunks are XOR-swizzled with the row so that the
// 32 rows read by one operand load fall in different banks.
template <int COLS>
__device__ inline int swz(int r, int c) {
    if constexpr (COLS == 32) {
        return r * 32 + ((c ^ ((r >> 1) & 3)) << 3);
    } else {
        return r * COLS + ((c ^ (r & 7)) << 3);
    }
}

__device__ inline bf16x8 lds_b128(const uint16_t* base, int off) {
    uint4 v = *reinterpret_cast<const uint4*>(base + off);
    return __builtin_bit_cast(bf16x8, v);
}

// token position of tile row t inside the k slots of the aggregation MFMA:
// swap bits 2 and 3 of t (see the header comment)
__device__ inline int perm_tok(int t) {
    return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1);
}

// reduce across the 32 lanes of each half-wave (lanes l and l^k, k < 32)
__device__ inline float half_max(float v) {
#pragma unroll
    for (int k = 1; k < 32; k <<= 1) v = fmaxf(v, __shfl_xor(v, k, 64));
    return v;
}
__device__ inline float half_sum(float v) {
#pragma unroll
    for (int k = 1; k < 32; k <<= 1) v += __shfl_xor(v, k, 64);
    return v;
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
    static constexpr int K_BYTES = 32 * D * 2;
    static constexpr int V_BYTES = D * 32 * 2;
    static constexpr int RED_BYTES = NW * 32 * 4;
    static constexpr int LDS = P_BYTES + K_BYTES + V_BYTES + 2 * RED_BYTES;
};

template <int D, int MW, int NW>
__global__ __launch_bounds__(NW * 64, 1) void fwd_fused_kernel(FusedFwdArgs a) {
    using C = Cfg<D, MW, NW>;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* Ps = reinterpret_cast<uint16_t*>(smem);
    uint16_t* Ks = reinterpret_cast<uint16_t*>(smem + C::P_BYTES);
    uint16_t* Vt = reinterpret_cast<uint16_t*>(smem + C::P_BYTES + C::K_BYTES);
    float* red_max = reinterpret_cast<float*>(smem + C::P_BYTES + C::K_BYTES + C::V_BYTES);
    float* red_sum = red_max + NW * 32;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int l32 = lane & 31;
    const int hl = lane >> 5;  // half of the wave

    const int64_t range = blockIdx.x;
    int64_t k0 = a.wg_start[range];
    int64_t k1 = a.wg_start[range + 1];
    if (k0 < 0 || k1 < k0 || k1 > a.max_items) return;  // malformed offsets: nothing safe to do

    const float ks2 = a.scale * kLog2e;
    const int64_t MD = (int64_t)C::M * D;
    int cur_h = -1;

    for (int64_t k = k0; k < k1; ++k) {
        const int32_t* it = a.items + k * IT_WORDS;
        const int b = it[IT_B];
        const int h = it[IT_H];
        const int t0 = it[IT_T0];
        const int t1 = it[IT_T1];
        const int split = it[IT_SPLIT];
        if (b < 0 || b >= a.B || h < 0 || h >= a.H || t0 < 0 || t1 < t0 || t1 > a.T) continue;

        if (h != cur_h) {
            __syncthreads();  // every wave is done with the previous P
            const uint4* src = reinterpret_cast<const uint4*>(a.P + (int64_t)h * C::M * D);
            for (int i = tid; i < C::M * C::KCH; i += C::THREADS) {
                const int r = i / C::KCH, c = i % C::KCH;
                *reinterpret_cast<uint4*>(Ps + swz<D>(r, c)) = src[i];
            }
            cur_h = h;
        }

        f32x16 acc[C::MT][C::JT];
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][jt][r] = 0.f;

        // prefetch the first tile
        uint4 kreg[C::NLD], vreg[C::NLD];
        // per-lane 32-bit element offsets inside a tile; the tile base is uniform
        const uint32_t row_stride = (uint32_t)a.H * D;
        auto load_tile = [&](int ts) {
            const int64_t tb = ((int64_t)ts * a.H + h) * D;
            const uint16_t* Kb = a.K + tb;
            const uint16_t* Vb = a.V + tb;
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                const int idx = tid + i * C::THREADS;
                const int tok = idx / C::KCH, ch = idx % C::KCH;
                uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
                if (idx < C::LD_CHUNKS && ts + tok < t1) {
                    const uint32_t off = (uint32_t)tok * row_stride + (uint32_t)(ch * 8);
                    kv = *reinterpret_cast<const uint4*>(Kb + off);
                    vv = *reinterpret_cast<const uint4*>(Vb + off);
                }
                kreg[i] = kv;
                vreg[i] = vv;
            }
        };
        load_tile(t0);

        for (int ts = t0; ts < t1; ts += 32) {
            // ---- stage K tile
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                const int idx = tid + i * C::THREADS;
                if (idx < C::LD_CHUNKS) {
                    const int tok = idx / C::KCH, ch = idx % C::KCH;
                    *reinterpret_cast<uint4*>(Ks + swz<D>(tok, ch)) = kreg[i];
                }
            }
            uint4 vcur[C::NLD];
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) vcur[i] = vreg[i];
            __syncthreads();  // B1: K tile and P visible
            if (ts + 32 < t1) load_tile(ts + 32);

            // ---- S = K . P^T for this wave's prototypes
            f32x16 s[C::MT];
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) s[mt][r] = 0.f;
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) {
                const bf16x8 ak = lds_b128(Ks, swz<D>(l32, 2 * kk + hl));
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    const bf16x8 bp = lds_b128(Ps, swz<D>(w * MW + mt * 32 + l32, 2 * kk + hl));
                    s[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak, bp, s[mt], 0, 0, 0);
                }
                // keep the operand loads of one k step in flight at a time
                __builtin_amdgcn_sched_barrier(0);
            }

            // ---- per-token max over prototypes
            float rmax[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float v = s[0][r];
#pragma unroll
                for (int mt = 1; mt < C::MT; ++mt) v = fmaxf(v, s[mt][r]);
                rmax[r] = half_max(v);
            }
            if (l32 == 0) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    red_max[w * 32 + 8 * (r >> 2) + 4 * hl + (r & 3)] = rmax[r];
            }
            __syncthreads();  // B2
            float nmu[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int t = 8 * (r >> 2) + 4 * hl + (r & 3);
                float mu = red_max[t];
#pragma unroll
                for (int ww = 1; ww < NW; ++ww) mu = fmaxf(mu, red_max[ww * 32 + t]);
                nmu[r] = -mu * ks2;
            }

            // ---- E = exp2((S - mu) * scale * log2 e), partial sums, bf16 operands
            float rsum[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) rsum[r] = 0.f;
            bf16x8 eop[C::MT][2];
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt) {
                float e[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    e[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mt][r], ks2, nmu[r]));
                    rsum[r] += e[r];
                }
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    uint4 pk;
                    pk.x = pack_bf16x2(e[8 * q + 0], e[8 * q + 1]);
                    pk.y = pack_bf16x2(e[8 * q + 2], e[8 * q + 3]);
                    pk.z = pack_bf16x2(e[8 * q + 4], e[8 * q + 5]);
                    pk.w = pack_bf16x2(e[8 * q + 6], e[8 * q + 7]);
                    eop[mt][q] = __builtin_bit_cast(bf16x8, pk);
                }
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) rsum[r] = half_sum(rsum[r]);
            if (l32 == 0) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    red_sum[w * 32 + 8 * (r >> 2) + 4 * hl + (r & 3)] = rsum[r];
            }
            __syncthreads();  // B3

            // ---- lse of the tile's tokens: thread tt of wave 0 handles token tt
            if (tid < 32 && a.lse && ts + tid < t1) {
                float mu = red_max[tid], z = red_sum[tid];
#pragma unroll
                for (int ww = 1; ww < NW; ++ww) {
                    mu = fmaxf(mu, red_max[ww * 32 + tid]);
                    z += red_sum[ww * 32 + tid];
                }
                a.lse[(int64_t)(ts + tid) * a.H + h] = mu * a.scale + __logf(z);
            }

            // ---- stage V / z transposed, in the permuted token order
#pragma unroll
            for (int i = 0; i < C::NLD; ++i) {
                const int idx = tid + i * C::THREADS;
                if (idx < C::LD_CHUNKS) {
                    const int tok = idx / C::KCH, ch = idx % C::KCH;
                    float z = 0.f;
#pragma unroll
                    for (int ww = 0; ww < NW; ++ww) z += red_sum[ww * 32 + tok];
                    const float rz = 1.0f / z;
                    const uint32_t wv[4] = {vcur[i].x, vcur[i].y, vcur[i].z, vcur[i].w};
                    const int p = perm_tok(tok);
#pragma unroll
                    for (int e2 = 0; e2 < 4; ++e2) {
                        const uint32_t pk = pack_bf16x2(bf16_lo(wv[e2]) * rz, bf16_hi(wv[e2]) * rz);
                        const int j0 = ch * 8 + 2 * e2;
                        Vt[swz<32>(j0, p >> 3) + (p & 7)] = (uint16_t)(pk & 0xffffu);
                        Vt[swz<32>(j0 + 1, p >> 3) + (p & 7)] = (uint16_t)(pk >> 16);
                    }
                }
            }
            __syncthreads();  // B4

            // ---- acc[m, j] += E^T . V'
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt) {
                const bf16x8 v0 = lds_b128(Vt, swz<32>(jt * 32 + l32, 0 + hl));
                const bf16x8 v1 = lds_b128(Vt, swz<32>(jt * 32 + l32, 2 + hl));
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    acc[mt][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eop[mt][0], v0, acc[mt][jt], 0, 0, 0);
                    acc[mt][jt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eop[mt][1], v1, acc[mt][jt], 0, 0, 0);
                }
            }
        }

        // ---- flush: the whole sketch of the pair, or this segment's partial
        float* out = split ? a.partials + k * MD : a.sketch + ((int64_t)b * a.H + h) * MD;
        const uint32_t lane_off = (uint32_t)((w * MW + 4 * hl) * D + l32);
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int jt = 0; jt < C::JT; ++jt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const uint32_t o = lane_off + (uint32_t)((mt * 32 + 8 * (r >> 2) + (r & 3)) * D + jt * 32);
                    out[o] = acc[mt][jt][r];
                }
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

// Instances: NW = 4 waves; MW = M / 4 prototypes per wave.
#define SA_FUSED_CASES(X)  \
    X(64, 32)              \
    X(64, 64)              \
    X(64, 96)              \
    X(64, 128)             \
    X(64, 160)             \
    X(64, 192)             \
    X(64, 224)             \
    X(64, 256)             \
    X(128, 32)             \
    X(128, 64)             \
    X(128, 96)             \
    X(128, 128)

bool fused_fwd_supported(int32_t M, int32_t d) {
    if (M % 128 != 0) return false;
#define X(DD, MWW) if (d == DD && M == 4 * MWW) return true;
    SA_FUSED_CASES(X)
#undef X
    return false;
}

size_t fused_fwd_lds_bytes(int32_t M, int32_t d) {
#define X(DD, MWW) if (d == DD && M == 4 * MWW) return Cfg<DD, MWW, 4>::LDS;
    SA_FUSED_CASES(X)
#undef X
    return 0;
}

hipError_t fused_fwd_occupancy(int32_t M, int32_t d, int* blocks) {
#define X(DD, MWW) if (d == DD && M == 4 * MWW) return occ_inst<DD, MWW, 4>(blocks);
    SA_FUSED_CASES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_fused_fwd(const FusedFwdArgs& a, hipStream_t stream) {
    if (a.n_ranges == 0) return hipSuccess;
#define X(DD, MWW) if (a.d == DD && a.M == 4 * MWW) return launch_inst<DD, MWW, 4>(a, stream);
    SA_FUSED_CASES(X)
#undef X
    return hipErrorInvalidValue;
}

}  // namespace sa

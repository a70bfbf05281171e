// Row kernels of the reordered single-query STCA over the sketch (Appendix G.2):
// the softmax over the k sketch rows of each (user, target, head) logit row and
// its backward.  The products around them run on the batched matrix-core GEMM.
//
// Rows are [rows][k] logits already multiplied by the attention scale, fp32, or
// bf16 in bf16 mode (written so by the logits product; the backward recomputes
// alpha from the same rounded logits).  One wave per row.  With k a multiple of 4 and at most 1024, a row is read once into
// registers (16 bytes per lane per 256 columns) and every pass runs on them;
// otherwise lanes stride the row in each pass.
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

__device__ inline float wave_max(float v) {
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) v = fmaxf(v, __shfl_xor(v, k, 64));
    return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) v += __shfl_xor(v, k, 64);
    return v;
}

// logit j of a row (SB: bf16 logits)
template <bool SB>
__device__ inline float get(const void* s, int64_t j) {
    if constexpr (SB) return tile::bf16_lo((uint32_t)reinterpret_cast<const uint16_t*>(s)[j]);
    else return reinterpret_cast<const float*>(s)[j];
}
template <bool BF16>
__device__ inline void put(void* p, int64_t i, float v) {
    if constexpr (BF16) reinterpret_cast<uint16_t*>(p)[i] = tile::to_bf16(v);
    else reinterpret_cast<float*>(p)[i] = v;
}

// lse = log sum_j exp(s_j); alpha_j = exp(s_j - lse)
template <bool BF16, bool SB>
__global__ __launch_bounds__(256) void stca_softmax_kernel(const void* __restrict__ S, int64_t rows, int32_t k,
                                                           void* __restrict__ alpha, float* __restrict__ lse) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int lane = threadIdx.x & 63;
    const int64_t s0 = row * k;
    float mx = -INFINITY;
    for (int j = lane; j < k; j += 64) mx = fmaxf(mx, get<SB>(S, s0 + j));
    mx = wave_max(mx);
    float z = 0.f;
    for (int j = lane; j < k; j += 64) z += __expf(get<SB>(S, s0 + j) - mx);
    const float l = mx + __logf(wave_sum(z));
    for (int j = lane; j < k; j += 64) put<BF16>(alpha, row * k + j, __expf(get<SB>(S, s0 + j) - l));
    if (lane == 0) lse[row] = l;
}

// ds_j = scale alpha_j (da_j - sum_i alpha_i da_i), alpha_j = exp(s_j - lse)
template <bool BF16, bool SB>
__global__ __launch_bounds__(256) void stca_softmax_bwd_kernel(const void* __restrict__ S,
                                                               const float* __restrict__ lse,
                                                               const float* __restrict__ dA, int64_t rows, int32_t k,
                                                               float scale, void* __restrict__ ds) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int lane = threadIdx.x & 63;
    const int64_t s0 = row * k;
    const float* da = dA + row * k;
    const float l = lse[row];
    float dot = 0.f;
    for (int j = lane; j < k; j += 64) dot = __builtin_fmaf(__expf(get<SB>(S, s0 + j) - l), da[j], dot);
    dot = wave_sum(dot);
    for (int j = lane; j < k; j += 64)
        put<BF16>(ds, row * k + j, scale * __expf(get<SB>(S, s0 + j) - l) * (da[j] - dot));
}

// logits c .. c + 3 of the row (4 consecutive per lane and piece: 16 bytes of
// fp32 or 8 of bf16); padding columns read as -inf
template <bool SB, int NV>
__device__ inline void load_row(const void* S, int64_t s0, int k, int lane, float4 (&v)[NV]) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = 4 * (lane + 64 * i);
        if (c >= k) {
            v[i] = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        } else if constexpr (SB) {
            const uint2 q = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(S) + s0 + c);
            v[i] = make_float4(tile::bf16_lo(q.x), tile::bf16_hi(q.x), tile::bf16_lo(q.y), tile::bf16_hi(q.y));
        } else {
            v[i] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(S) + s0 + c);
        }
    }
}
template <bool BF16>
__device__ inline void put4(void* p, int64_t i, float a, float b, float c, float d) {
    if constexpr (BF16)
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(p) + i) =
            make_uint2(tile::pack_bf16x2(a, b), tile::pack_bf16x2(c, d));
    else
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(p) + i) = make_float4(a, b, c, d);
}

// the register-resident forms of the two kernels above (NV 16-byte pieces per lane)
template <bool BF16, bool SB, int NV>
__global__ __launch_bounds__(256) void stca_softmax_reg_kernel(const void* __restrict__ S, int64_t rows, int32_t k,
                                                               void* __restrict__ alpha, float* __restrict__ lse) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int lane = threadIdx.x & 63;
    float4 v[NV];
    load_row<SB, NV>(S, row * k, k, lane, v);
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) mx = fmaxf(fmaxf(mx, fmaxf(v[i].x, v[i].y)), fmaxf(v[i].z, v[i].w));
    mx = wave_max(mx);
    // each exponential once: alpha = exp(s - max) / z
    float z = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {   // (padding columns hold -inf: exp gives 0)
        v[i] = make_float4(__expf(v[i].x - mx), __expf(v[i].y - mx), __expf(v[i].z - mx), __expf(v[i].w - mx));
        z += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    }
    z = wave_sum(z);
    const float inv = 1.f / z;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = 4 * (lane + 64 * i);
        if (c < k) put4<BF16>(alpha, row * k + c, v[i].x * inv, v[i].y * inv, v[i].z * inv, v[i].w * inv);
    }
    if (lane == 0) lse[row] = mx + __logf(z);
}

template <bool BF16, bool SB, int NV>
__global__ __launch_bounds__(256) void stca_softmax_bwd_reg_kernel(const void* __restrict__ S,
                                                                   const float* __restrict__ lse,
                                                                   const float* __restrict__ dA, int64_t rows,
                                                                   int32_t k, float scale, void* __restrict__ ds) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int lane = threadIdx.x & 63;
    const float l = lse[row];
    float4 v[NV], g[NV];
    load_row<SB, NV>(S, row * k, k, lane, v);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = 4 * (lane + 64 * i);
        g[i] = c < k ? *reinterpret_cast<const float4*>(dA + row * k + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        v[i] = make_float4(__expf(v[i].x - l), __expf(v[i].y - l), __expf(v[i].z - l), __expf(v[i].w - l));
    }
    float dot = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        dot = __builtin_fmaf(v[i].x, g[i].x, dot);
        dot = __builtin_fmaf(v[i].y, g[i].y, dot);
        dot = __builtin_fmaf(v[i].z, g[i].z, dot);
        dot = __builtin_fmaf(v[i].w, g[i].w, dot);
    }
    dot = wave_sum(dot);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = 4 * (lane + 64 * i);
        if (c < k)
            put4<BF16>(ds, row * k + c, scale * v[i].x * (g[i].x - dot), scale * v[i].y * (g[i].y - dot),
                       scale * v[i].z * (g[i].z - dot), scale * v[i].w * (g[i].w - dot));
    }
}

// bf16 logits with k a multiple of 8: each lane reads 8 consecutive logits per
// 16-byte load (NV loads per lane) and writes their 8 weights at once
template <bool BF16, int NV>
__global__ __launch_bounds__(256) void stca_softmax_b8_kernel(const uint16_t* __restrict__ S, int64_t rows, int32_t k,
                                                              void* __restrict__ alpha, float* __restrict__ lse) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int lane = threadIdx.x & 63;
    float v[NV][8];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = 8 * (lane + 64 * i);
        if (c < k) {
            const uint4 q = *reinterpret_cast<const uint4*>(S + row * k + c);
            const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[i][2 * e] = tile::bf16_lo(w[e]);
                v[i][2 * e + 1] = tile::bf16_hi(w[e]);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[i][e] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, v[i][e]);
    mx = wave_max(mx);
    float z = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) {   // (padding columns hold -inf: exp gives 0)
            v[i][e] = __expf(v[i][e] - mx);
            z += v[i][e];
        }
    z = wave_sum(z);
    const float inv = 1.f / z;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = 8 * (lane + 64 * i);
        if (c >= k) continue;
        const int64_t o = row * k + c;
        if constexpr (BF16) {
            *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(alpha) + o) =
                make_uint4(tile::pack_bf16x2(v[i][0] * inv, v[i][1] * inv), tile::pack_bf16x2(v[i][2] * inv, v[i][3] * inv),
                           tile::pack_bf16x2(v[i][4] * inv, v[i][5] * inv), tile::pack_bf16x2(v[i][6] * inv, v[i][7] * inv));
        } else {
            put4<false>(alpha, o, v[i][0] * inv, v[i][1] * inv, v[i][2] * inv, v[i][3] * inv);
            put4<false>(alpha, o + 4, v[i][4] * inv, v[i][5] * inv, v[i][6] * inv, v[i][7] * inv);
        }
    }
    if (lane == 0) lse[row] = mx + __logf(z);
}
__global__ __launch_bounds__(256) void to_bf16_kernel(const float* __restrict__ x, uint16_t* __restrict__ y,
                                                      int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) y[i] = tile::to_bf16(x[i]);
}

}  // namespace

// pieces per lane of the register-resident kernels, 0 when k does not fit them
int reg_pieces(int32_t k) {
    if (k % 4 != 0) return 0;
    if (k <= 256) return 1;
    if (k <= 512) return 2;
    if (k <= 1024) return 4;
    return 0;
}

hipError_t launch_stca_softmax(const void* S, bool s_bf16, int64_t rows, int32_t k, bool bf16, void* alpha,
                               float* lse, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    const dim3 grid((unsigned)((rows + 3) / 4));
    if (s_bf16 && k % 8 == 0 && k <= 1024) {
        const uint16_t* Sb = reinterpret_cast<const uint16_t*>(S);
        if (k <= 512) {
            if (bf16) hipLaunchKernelGGL((stca_softmax_b8_kernel<true, 1>), grid, dim3(256), 0, stream, Sb, rows, k,
                                         alpha, lse);
            else hipLaunchKernelGGL((stca_softmax_b8_kernel<false, 1>), grid, dim3(256), 0, stream, Sb, rows, k,
                                    alpha, lse);
        } else {
            if (bf16) hipLaunchKernelGGL((stca_softmax_b8_kernel<true, 2>), grid, dim3(256), 0, stream, Sb, rows, k,
                                         alpha, lse);
            else hipLaunchKernelGGL((stca_softmax_b8_kernel<false, 2>), grid, dim3(256), 0, stream, Sb, rows, k,
                                    alpha, lse);
        }
        return hipGetLastError();
    }
    const int nv = reg_pieces(k);
#define SA_LAUNCH(BF, SB)                                                                                        \
    if (bf16 == BF && s_bf16 == SB) {                                                                           \
        if (nv == 1) hipLaunchKernelGGL((stca_softmax_reg_kernel<BF, SB, 1>), grid, dim3(256), 0, stream, S,    \
                                        rows, k, alpha, lse);                                                   \
        else if (nv == 2) hipLaunchKernelGGL((stca_softmax_reg_kernel<BF, SB, 2>), grid, dim3(256), 0, stream,  \
                                             S, rows, k, alpha, lse);                                           \
        else if (nv == 4) hipLaunchKernelGGL((stca_softmax_reg_kernel<BF, SB, 4>), grid, dim3(256), 0, stream,  \
                                             S, rows, k, alpha, lse);                                           \
        else hipLaunchKernelGGL((stca_softmax_kernel<BF, SB>), grid, dim3(256), 0, stream, S, rows, k, alpha,   \
                                lse);                                                                           \
        return hipGetLastError();                                                                               \
    }
    SA_LAUNCH(true, true)
    SA_LAUNCH(true, false)
    SA_LAUNCH(false, true)
    SA_LAUNCH(false, false)
#undef SA_LAUNCH
    return hipErrorInvalidValue;
}
hipError_t launch_stca_softmax_bwd(const void* S, bool s_bf16, const float* lse, const float* dA, int64_t rows,
                                   int32_t k, float scale, bool bf16, void* ds, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    const dim3 grid((unsigned)((rows + 3) / 4));
    const int nv = reg_pieces(k);
#define SA_LAUNCH(BF, SB)                                                                                          \
    if (bf16 == BF && s_bf16 == SB) {                                                                             \
        if (nv == 1) hipLaunchKernelGGL((stca_softmax_bwd_reg_kernel<BF, SB, 1>), grid, dim3(256), 0, stream, S,  \
                                        lse, dA, rows, k, scale, ds);                                             \
        else if (nv == 2) hipLaunchKernelGGL((stca_softmax_bwd_reg_kernel<BF, SB, 2>), grid, dim3(256), 0,       \
                                             stream, S, lse, dA, rows, k, scale, ds);                             \
        else if (nv == 4) hipLaunchKernelGGL((stca_softmax_bwd_reg_kernel<BF, SB, 4>), grid, dim3(256), 0,       \
                                             stream, S, lse, dA, rows, k, scale, ds);                             \
        else hipLaunchKernelGGL((stca_softmax_bwd_kernel<BF, SB>), grid, dim3(256), 0, stream, S, lse, dA, rows,  \
                                k, scale, ds);                                                                    \
        return hipGetLastError();                                                                                 \
    }
    SA_LAUNCH(true, true)
    SA_LAUNCH(true, false)
    SA_LAUNCH(false, true)
    SA_LAUNCH(false, false)
#undef SA_LAUNCH
    return hipErrorInvalidValue;
}
hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(to_bf16_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, x, y, n);
    return hipGetLastError();
}

}  // namespace sa

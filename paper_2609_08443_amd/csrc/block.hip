// Refinement between the sketching steps of stacked SA (section 3.3):
//
//   Xbar = LN1(Xt + Xhat),   Xt' = LN2(Xbar + FFN(Xbar)),
//   FFN(x) = (silu(x W1) * (x W3)) W2          (SwiGLU, intermediate width 2d)
//
// per (user, head, prototype) row of d features.  The FFN products run on the
// batched product of layer.hip; this file holds the residual + layer norm and
// the gate.  LN(x) = (x - mean) / sqrt(var + eps) * gamma + beta with the
// biased variance over the d features, gamma and beta per head.
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

template <bool BF16>
__device__ inline float ldv(const void* p, int64_t i) {
    if constexpr (BF16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(p)[i] << 16);
    else return reinterpret_cast<const float*>(p)[i];
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) v += __shfl_xor(v, k, 64);
    return v;
}

// One wave per row r of [rows][D]: out[r] = LN(x[r mod x_rows] + y[r]) * gamma[h] + beta[h],
// h = (r / M) % H.  x is the state (fp32, or the shared prototypes in the input
// dtype, whose x_rows = H * M rows repeat for every user); y is fp32.
template <int D, bool XBF16, bool PBF16>
__global__ __launch_bounds__(256) void add_ln_kernel(const void* __restrict__ x, int64_t x_rows,
                                                     const float* __restrict__ y, const void* __restrict__ gamma,
                                                     const void* __restrict__ beta, int64_t rows, int32_t H,
                                                     int32_t M, float eps, float* __restrict__ out) {
    constexpr int E = D / 64;   // features per lane
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= rows) return;
    const int lane = threadIdx.x & 63;
    const int64_t xr = r % x_rows;
    const int64_t h = (r / M) % H;
    float v[E];
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = lane + 64 * e;
        v[e] = ldv<XBF16>(x, xr * D + j) + y[r * D + j];
        s += v[e];
    }
    const float mean = wave_sum(s) * (1.0f / D);
    float q = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        v[e] -= mean;
        q = __builtin_fmaf(v[e], v[e], q);
    }
    const float rstd = 1.0f / __builtin_sqrtf(wave_sum(q) * (1.0f / D) + eps);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = lane + 64 * e;
        out[r * D + j] = v[e] * rstd * ldv<PBF16>(gamma, h * D + j) + ldv<PBF16>(beta, h * D + j);
    }
}

// g[i] = silu(g[i]) * u[i]
__global__ __launch_bounds__(256) void swiglu_gate_kernel(float* __restrict__ g, const float* __restrict__ u,
                                                          int64_t n4) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    float4 a = reinterpret_cast<float4*>(g)[i];
    const float4 b = reinterpret_cast<const float4*>(u)[i];
    a.x = a.x / (1.0f + __expf(-a.x)) * b.x;
    a.y = a.y / (1.0f + __expf(-a.y)) * b.y;
    a.z = a.z / (1.0f + __expf(-a.z)) * b.z;
    a.w = a.w / (1.0f + __expf(-a.w)) * b.w;
    reinterpret_cast<float4*>(g)[i] = a;
}

template <int D>
hipError_t add_ln_d(const void* x, bool x_bf16, int64_t x_rows, const float* y, const void* gamma,
                    const void* beta, bool p_bf16, int64_t rows, int32_t H, int32_t M, float eps, float* out,
                    hipStream_t stream) {
    const dim3 grid((unsigned)((rows + 3) / 4));
#define SA_LN(XB, PB)                                                                                      \
    hipLaunchKernelGGL((add_ln_kernel<D, XB, PB>), grid, dim3(256), 0, stream, x, x_rows, y, gamma, beta, \
                       rows, H, M, eps, out)
    if (x_bf16) {
        if (p_bf16) SA_LN(true, true); else SA_LN(true, false);
    } else {
        if (p_bf16) SA_LN(false, true); else SA_LN(false, false);
    }
#undef SA_LN
    return hipGetLastError();
}

}  // namespace

hipError_t launch_add_ln(const void* x, bool x_bf16, int64_t x_rows, const float* y, const void* gamma,
                         const void* beta, bool p_bf16, int64_t rows, int32_t H, int32_t M, int32_t d, float eps,
                         float* out, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d == 64) return add_ln_d<64>(x, x_bf16, x_rows, y, gamma, beta, p_bf16, rows, H, M, eps, out, stream);
    if (d == 128) return add_ln_d<128>(x, x_bf16, x_rows, y, gamma, beta, p_bf16, rows, H, M, eps, out, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_swiglu_gate(float* g, const float* u, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t n4 = n / 4;   // n is a multiple of 2d
    hipLaunchKernelGGL(swiglu_gate_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, g, u, n4);
    return hipGetLastError();
}

}  // namespace sa

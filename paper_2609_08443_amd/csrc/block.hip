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
                                                     int32_t M, float eps, float* __restrict__ out,
                                                     float* __restrict__ sum_out) {
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
        if (sum_out) sum_out[r * D + j] = v[e];
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

// z = silu(g) * u (g, u kept for the backward)
__global__ __launch_bounds__(256) void swiglu_fwd_kernel(const float* __restrict__ g, const float* __restrict__ u,
                                                         float* __restrict__ z, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float a = g[i];
    z[i] = a / (1.0f + __expf(-a)) * u[i];
}

// Backward of z = silu(g) * u: dg = dz u s (1 + g (1 - s)), du = dz g s, s = sigmoid(g).
// dg overwrites dz.
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(float* __restrict__ dz_dg, const float* __restrict__ g,
                                                         const float* __restrict__ u, float* __restrict__ du,
                                                         int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float a = g[i], dz = dz_dg[i];
    const float sg = 1.0f / (1.0f + __expf(-a));
    dz_dg[i] = dz * u[i] * sg * (1.0f + a * (1.0f - sg));
    du[i] = dz * a * sg;
}

// Backward of out = LN(y) * gamma + beta per row (one wave per row):
// dx = rstd (g - mean(g) - xh mean(g xh)), g = (dy1 + dy2) gamma, xh = (y - mean) rstd.
// dy2 may be null.  Writes (mean, rstd) per row for the gamma / beta reduction.
template <int D, bool PBF16>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const float* __restrict__ dy1, const float* __restrict__ dy2,
                                                     const float* __restrict__ y, const void* __restrict__ gamma,
                                                     int64_t rows, int32_t H, int32_t M, float eps,
                                                     float* __restrict__ dx, float2* __restrict__ stats) {
    constexpr int E = D / 64;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= rows) return;
    const int lane = threadIdx.x & 63;
    const int64_t h = (r / M) % H;
    float v[E], gv[E];
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        v[e] = y[r * D + lane + 64 * e];
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
    float sg = 0.f, sgx = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = lane + 64 * e;
        float d = dy1[r * D + j];
        if (dy2) d += dy2[r * D + j];
        v[e] *= rstd;   // xh
        gv[e] = d * ldv<PBF16>(gamma, h * D + j);
        sg += gv[e];
        sgx = __builtin_fmaf(gv[e], v[e], sgx);
    }
    const float mg = wave_sum(sg) * (1.0f / D), mgx = wave_sum(sgx) * (1.0f / D);
#pragma unroll
    for (int e = 0; e < E; ++e) dx[r * D + lane + 64 * e] = rstd * (gv[e] - mg - v[e] * mgx);
    if (lane == 0) stats[r] = make_float2(mean, rstd);
}

// Column sums for gamma / beta of one layer norm: part[c][h][0][j] = sum over the
// chunk c of head h's rows of (dy1 + dy2) * xh, part[c][h][1][j] of (dy1 + dy2).
// Rows of head h: (b * H + h) * M + m; a chunk covers CH consecutive (b, m).  The
// 256 / D thread groups of a workgroup take every (256 / D)-th row of the chunk
// in order, and their sums are added in group order (deterministic).
template <int D>
__global__ __launch_bounds__(256) void ln_colsum_kernel(const float* __restrict__ dy1, const float* __restrict__ dy2,
                                                        const float* __restrict__ y, const float2* __restrict__ stats,
                                                        int64_t B, int32_t H, int32_t M, int64_t CH,
                                                        float* __restrict__ part) {
    constexpr int G = 256 / D;
    __shared__ float red[2][G][D];
    const int j = threadIdx.x % D, g = threadIdx.x / D;
    const int64_t h = blockIdx.z, c = blockIdx.x;
    const int64_t n = B * M;   // < 2^31 (checked by the host)
    const int64_t i0 = c * CH, i1 = i0 + CH < n ? i0 + CH : n;
    float sx = 0.f, s1 = 0.f;
#pragma unroll 4
    for (int64_t i = i0 + g; i < i1; i += G) {
        const uint32_t b = (uint32_t)i / (uint32_t)M, m = (uint32_t)i - b * (uint32_t)M;
        const int64_t r = ((int64_t)b * H + h) * M + m;
        float d = dy1[r * D + j];
        if (dy2) d += dy2[r * D + j];
        const float2 st = stats[r];
        sx = __builtin_fmaf(d, (y[r * D + j] - st.x) * st.y, sx);
        s1 += d;
    }
    red[0][g][j] = sx;
    red[1][g][j] = s1;
    __syncthreads();
    if (g == 0) {
#pragma unroll
        for (int q = 1; q < G; ++q) {
            sx += red[0][q][j];
            s1 += red[1][q][j];
        }
        float* o = part + ((c * H + h) * 2) * D;
        o[j] = sx;
        o[D + j] = s1;
    }
}

// out[h][k][j] = sum over chunks c of part[c][h][k][j]; out has a stride of
// ostride floats between k = 0 (gamma) and k = 1 (beta).  A workgroup takes 32
// columns of [h][k][j]; its eight thread groups each sum the chunks g, g + 8, ...
// in order, and the eight group sums are added in group order (a fixed order,
// so the result is deterministic).
__global__ __launch_bounds__(256) void ln_chunk_sum_kernel(const float* __restrict__ part, int64_t nch, int32_t H,
                                                           int32_t D, float* __restrict__ out, int64_t ostride) {
    __shared__ float red[8][32];
    const int64_t m = (int64_t)H * 2 * D;
    const int g = threadIdx.x >> 5, col = threadIdx.x & 31;
    const int64_t i = (int64_t)blockIdx.x * 32 + col;
    float s = 0.f;
    if (i < m) {
#pragma unroll 8
        for (int64_t c = g; c < nch; c += 8) s += part[c * m + i];
    }
    red[g][col] = s;
    __syncthreads();
    if (g == 0 && i < m) {
        float t = red[0][col];
#pragma unroll
        for (int q = 1; q < 8; ++q) t += red[q][col];
        const int64_t h = i / (2 * D), k = (i / D) % 2, j = i % D;
        out[k * ostride + h * D + j] = t;
    }
}

__global__ __launch_bounds__(256) void fill_kernel(float* __restrict__ p, int64_t n, float v) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

// out[h][i] = sum over users b, in order, of part[b * H + h][i]  (n values per block)
__global__ __launch_bounds__(256) void sum_users_kernel(const float* __restrict__ part, int64_t B, int32_t H,
                                                        int64_t n, float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)H * n) return;
    const int64_t h = i / n, k = i % n;
    float s = 0.f;
    for (int64_t b = 0; b < B; ++b) s += part[(b * H + h) * n + k];
    out[i] = s;
}

template <int D>
hipError_t add_ln_d(const void* x, bool x_bf16, int64_t x_rows, const float* y, const void* gamma,
                    const void* beta, bool p_bf16, int64_t rows, int32_t H, int32_t M, float eps, float* out,
                    float* sum_out, hipStream_t stream) {
    const dim3 grid((unsigned)((rows + 3) / 4));
#define SA_LN(XB, PB)                                                                                      \
    hipLaunchKernelGGL((add_ln_kernel<D, XB, PB>), grid, dim3(256), 0, stream, x, x_rows, y, gamma, beta, \
                       rows, H, M, eps, out, sum_out)
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
                         float* out, hipStream_t stream, float* sum_out) {
    if (rows <= 0) return hipSuccess;
    if (d == 64)
        return add_ln_d<64>(x, x_bf16, x_rows, y, gamma, beta, p_bf16, rows, H, M, eps, out, sum_out, stream);
    if (d == 128)
        return add_ln_d<128>(x, x_bf16, x_rows, y, gamma, beta, p_bf16, rows, H, M, eps, out, sum_out, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_swiglu_fwd(const float* g, const float* u, float* z, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(swiglu_fwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, g, u, z, n);
    return hipGetLastError();
}

hipError_t launch_swiglu_bwd(float* dz_dg, const float* g, const float* u, float* du, int64_t n,
                             hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, dz_dg, g, u,
                       du, n);
    return hipGetLastError();
}

hipError_t launch_ln_bwd(const float* dy1, const float* dy2, const float* y, const void* gamma, bool p_bf16,
                         int64_t B, int32_t H, int32_t M, int32_t d, float eps, float* dx, float2* stats,
                         float* colpart, int64_t nch, float* dgamma_dbeta, int64_t ostride, hipStream_t stream) {
    const int64_t rows = B * H * M;
    if (rows <= 0) return hipSuccess;
    const dim3 grid((unsigned)((rows + 3) / 4));
    const int64_t n = B * M, CH = (n + nch - 1) / nch;
#define SA_COL(DD)                                                                                            \
    hipLaunchKernelGGL(ln_colsum_kernel<DD>, dim3((unsigned)nch, 1, (unsigned)H), dim3(256), 0, stream, dy1, \
                       dy2, y, stats, B, H, M, CH, colpart)
#define SA_LNB(DD, PB)                                                                                    \
    hipLaunchKernelGGL((ln_bwd_kernel<DD, PB>), grid, dim3(256), 0, stream, dy1, dy2, y, gamma, rows, H, M, \
                       eps, dx, stats)
    // rows first: the column sums read their statistics
    if (d == 64) { if (p_bf16) SA_LNB(64, true); else SA_LNB(64, false); }
    else { if (p_bf16) SA_LNB(128, true); else SA_LNB(128, false); }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (d == 64) SA_COL(64); else SA_COL(128);
#undef SA_COL
#undef SA_LNB
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t m = (int64_t)H * 2 * d;
    hipLaunchKernelGGL(ln_chunk_sum_kernel, dim3((unsigned)((m + 31) / 32)), dim3(256), 0, stream, colpart, nch, H,
                       d, dgamma_dbeta, ostride);
    return hipGetLastError();
}

hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p, n, v);
    return hipGetLastError();
}

hipError_t launch_sum_users(const float* part, int64_t B, int32_t H, int64_t n, float* out, hipStream_t stream) {
    const int64_t m = (int64_t)H * n;
    if (m <= 0) return hipSuccess;
    hipLaunchKernelGGL(sum_users_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, stream, part, B, H, n, out);
    return hipGetLastError();
}

hipError_t launch_swiglu_gate(float* g, const float* u, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t n4 = n / 4;   // n is a multiple of 2d
    hipLaunchKernelGGL(swiglu_gate_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, g, u, n4);
    return hipGetLastError();
}

}  // namespace sa

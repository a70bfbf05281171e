// Projections of the SA layer (Appendix G.3: Q = P W_Q, K = X W_K, the history X
// itself aggregated) around the sketching kernels.
//
// The key projection is absorbed into the prototype side:
//
//   S = scale (P W_Q)(X W_K)^T = scale (P W_Q W_K^T) X^T = scale P' X^T,
//
// the reordering the paper applies to single-query STCA (Appendix G.2), so the
// per-token work is the sketching step with K = V = X and prototypes P'.  X is
// read once, no [T, d] key tensor exists, and the only added work is per head:
// two [M, d] x [d, d] products forward and four backward:
//
//   dW_K = dP'^T Q,   dQ = dP' W_K,   dW_Q = P^T dQ,   dP = dQ W_Q^T
//
// (P' = Q W_K^T, Q = P W_Q), with dP' the prototype gradient of the sketching
// backward and dX = dV + scale dS P' from its token side.
//
// This file holds the small batched product used for those six [M|d] x d
// matrices (fp32 accumulation, strided operands so that transposes are free)
// and the elementwise sum of the plain path's dK and dV.
#include "sa_internal.h"
#include "tile_ops.h"

namespace sa {

namespace {

template <typename T>
__device__ inline float load_el(const T* p, int64_t i);
template <>
__device__ inline float load_el<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ inline float load_el<uint16_t>(const uint16_t* p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

template <typename T>
__device__ inline void store_el(T* p, int64_t i, float v);
template <>
__device__ inline void store_el<float>(float* p, int64_t i, float v) { p[i] = v; }
template <>
__device__ inline void store_el<uint16_t>(uint16_t* p, int64_t i, float v) { p[i] = tile::to_bf16(v); }

// C[h][r][c] = sum_k A[h](r, k) B[h](k, c) for r < R, c < N, k < Kd, with
// A(r, k) = A[h * a_h + r * a_r + k * a_k] and B(k, c) = B[h * b_h + k * b_k + c * b_c];
// C row-major [R][N] per head.  A 32 x 32 output tile per workgroup of 256
// threads; k advances in slabs of 32 staged in LDS, the next slab's loads in
// flight (registers) while the current one is used.  Consecutive lanes walk the
// unit-stride index of each operand so that its loads coalesce.
template <typename TA, typename TB, typename TC>
__global__ __launch_bounds__(256) void small_gemm_kernel(const TA* __restrict__ A, int64_t a_h, int64_t a_r,
                                                         int64_t a_k, const TB* __restrict__ Bm, int64_t b_h,
                                                         int64_t b_k, int64_t b_c, TC* __restrict__ C,
                                                         int32_t R, int32_t N, int32_t Kd) {
    __shared__ float As[32][33];   // [r][k]
    __shared__ float Bs[32][33];   // [k][c]
    const int tid = threadIdx.x, tx = tid & 31, ty = tid >> 5;
    const int r0 = blockIdx.x * 32, c0 = blockIdx.y * 32;
    const int64_t h = blockIdx.z;
    const TA* Ah = A + h * a_h;
    const TB* Bh = Bm + h * b_h;
    const bool a_rows_fast = a_r == 1 && a_k != 1;   // lanes along r
    const bool b_k_fast = b_k == 1 && b_c != 1;      // lanes along k
    float ra[4], rb[4];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int u = ty + 8 * i;
            const int ar = a_rows_fast ? tx : u, ak = a_rows_fast ? u : tx;
            const int r = r0 + ar, k = k0 + ak;
            ra[i] = (r < R && k < Kd) ? load_el(Ah, (int64_t)r * a_r + (int64_t)k * a_k) : 0.f;
            const int bk = b_k_fast ? tx : u, bc = b_k_fast ? u : tx;
            const int kb = k0 + bk, c = c0 + bc;
            rb[i] = (kb < Kd && c < N) ? load_el(Bh, (int64_t)kb * b_k + (int64_t)c * b_c) : 0.f;
        }
    };
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    fetch(0);
    for (int k0 = 0; k0 < Kd; k0 += 32) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int u = ty + 8 * i;
            if (a_rows_fast) As[tx][u] = ra[i]; else As[u][tx] = ra[i];
            if (b_k_fast) Bs[tx][u] = rb[i]; else Bs[u][tx] = rb[i];
        }
        __syncthreads();
        if (k0 + 32 < Kd) fetch(k0 + 32);
#pragma unroll 8
        for (int kk = 0; kk < 32; ++kk) {
            const float b = Bs[kk][tx];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(As[ty + 8 * i][kk], b, acc[i]);
        }
        __syncthreads();
    }
    TC* Ch = C + h * (int64_t)R * N;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = r0 + ty + 8 * i, c = c0 + tx;
        if (r < R && c < N) store_el(Ch, (int64_t)r * N + c, acc[i]);
    }
}

__global__ __launch_bounds__(256) void add_kernel(const float* __restrict__ a, const float* __restrict__ b,
                                                  float* __restrict__ out, int64_t n4) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    const float4 x = reinterpret_cast<const float4*>(a)[i];
    const float4 y = reinterpret_cast<const float4*>(b)[i];
    reinterpret_cast<float4*>(out)[i] = make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
}

template <typename TA, typename TB, typename TC>
hipError_t gemm_t(const MatView& a, const MatView& b, void* c, int32_t H, int32_t R, int32_t N, int32_t Kd,
                  hipStream_t stream) {
    const dim3 grid((unsigned)((R + 31) / 32), (unsigned)((N + 31) / 32), (unsigned)H);
    hipLaunchKernelGGL((small_gemm_kernel<TA, TB, TC>), grid, dim3(256), 0, stream,
                       reinterpret_cast<const TA*>(a.p), a.s_h, a.s_0, a.s_1,
                       reinterpret_cast<const TB*>(b.p), b.s_h, b.s_0, b.s_1, reinterpret_cast<TC*>(c), R,
                       N, Kd);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_small_gemm(const MatView& a, const MatView& b, void* c, bool c_bf16, int32_t H, int32_t R,
                             int32_t N, int32_t Kd, hipStream_t stream) {
    if (H <= 0 || R <= 0 || N <= 0) return hipSuccess;
    if (a.bf16 && b.bf16)
        return c_bf16 ? gemm_t<uint16_t, uint16_t, uint16_t>(a, b, c, H, R, N, Kd, stream)
                      : gemm_t<uint16_t, uint16_t, float>(a, b, c, H, R, N, Kd, stream);
    if (a.bf16)
        return c_bf16 ? gemm_t<uint16_t, float, uint16_t>(a, b, c, H, R, N, Kd, stream)
                      : gemm_t<uint16_t, float, float>(a, b, c, H, R, N, Kd, stream);
    if (b.bf16)
        return c_bf16 ? gemm_t<float, uint16_t, uint16_t>(a, b, c, H, R, N, Kd, stream)
                      : gemm_t<float, uint16_t, float>(a, b, c, H, R, N, Kd, stream);
    return c_bf16 ? gemm_t<float, float, uint16_t>(a, b, c, H, R, N, Kd, stream)
                  : gemm_t<float, float, float>(a, b, c, H, R, N, Kd, stream);
}

hipError_t launch_add(const float* a, const float* b, float* out, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t n4 = n / 4;   // n is a multiple of d (64 or 128)
    hipLaunchKernelGGL(add_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, a, b, out, n4);
    return hipGetLastError();
}

}  // namespace sa

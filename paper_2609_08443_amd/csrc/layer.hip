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

// C[z][r][c] = sum_k A[z](r, k) B[z % b_mod](k, c) for r < R, c < N, k < Kd, with
// A(r, k) = A[z * a_h + r * a_r + k * a_k] and B(k, c) = B[z' * b_h + k * b_k + c * b_c];
// C[z * c_h + r * c_r + c] (with accumulate, C += alpha A B instead of C = alpha A B).  A 64 x 64 output tile per workgroup of 256
// threads, 4 x 4 outputs per thread; k advances in slabs of 16 staged in LDS
// (k-major, so each k step is two 16-byte LDS reads for 16 FMAs), the next
// slab's loads in flight while the current one is used.  Consecutive lanes walk
// the unit-stride index of each operand so that its loads coalesce.
template <typename TA, typename TB, typename TC>
__global__ __launch_bounds__(256) void small_gemm_kernel(const TA* __restrict__ A, int64_t a_h, int64_t a_r,
                                                         int64_t a_k, const TB* __restrict__ Bm, int64_t b_h,
                                                         int64_t b_k, int64_t b_c, int32_t b_mod,
                                                         TC* __restrict__ C, int64_t c_h, int64_t c_r, int32_t R,
                                                         int32_t N, int32_t Kd, float alpha, bool accumulate) {
    constexpr int TR = 64, TC_ = 64, TK = 16, PAD = 4;
    __shared__ __attribute__((aligned(16))) float As[TK][TR + PAD];   // [k][r]
    __shared__ __attribute__((aligned(16))) float Bs[TK][TC_ + PAD];  // [k][c]
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int r0 = blockIdx.x * TR, c0 = blockIdx.y * TC_;
    const int64_t z = blockIdx.z;
    const TA* Az = A + z * a_h;
    const TB* Bz = Bm + (z % b_mod) * b_h;
    const bool a_rows_fast = a_r == 1 && a_k != 1;   // lanes along r, else along k
    const bool b_k_fast = b_k == 1 && b_c != 1;      // lanes along k, else along c
    float ra[4], rb[4];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ar = a_rows_fast ? tid & 63 : (tid >> 4) + 16 * i;
            const int ak = a_rows_fast ? (tid >> 6) + 4 * i : tid & 15;
            const int r = r0 + ar, k = k0 + ak;
            ra[i] = (r < R && k < Kd) ? load_el(Az, (int64_t)r * a_r + (int64_t)k * a_k) : 0.f;
            const int bk = b_k_fast ? tid & 15 : (tid >> 6) + 4 * i;
            const int bc = b_k_fast ? (tid >> 4) + 16 * i : tid & 63;
            const int kb = k0 + bk, c = c0 + bc;
            rb[i] = (kb < Kd && c < N) ? load_el(Bz, (int64_t)kb * b_k + (int64_t)c * b_c) : 0.f;
        }
    };
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
    fetch(0);
    for (int k0 = 0; k0 < Kd; k0 += TK) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ar = a_rows_fast ? tid & 63 : (tid >> 4) + 16 * i;
            const int ak = a_rows_fast ? (tid >> 6) + 4 * i : tid & 15;
            As[ak][ar] = ra[i];
            const int bk = b_k_fast ? tid & 15 : (tid >> 6) + 4 * i;
            const int bc = b_k_fast ? (tid >> 4) + 16 * i : tid & 63;
            Bs[bk][bc] = rb[i];
        }
        __syncthreads();
        if (k0 + TK < Kd) fetch(k0 + TK);
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            const float4 av = *reinterpret_cast<const float4*>(&As[kk][ty * 4]);
            const float4 bv = *reinterpret_cast<const float4*>(&Bs[kk][tx * 4]);
            const float a4[4] = {av.x, av.y, av.z, av.w}, b4[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a4[i], b4[j], acc[i][j]);
        }
        __syncthreads();
    }
    TC* Cz = C + z * c_h;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = r0 + ty * 4 + i;
        if (r >= R) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = c0 + tx * 4 + j;
            if (c >= N) continue;
            const int64_t o = (int64_t)r * c_r + c;
            const float v = alpha * acc[i][j];
            store_el(Cz, o, accumulate ? v + load_el(Cz, o) : v);
        }
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
hipError_t gemm_t(const MatView& a, const MatView& b, int32_t b_mod, void* c, int64_t c_h, int64_t c_r, int32_t H,
                  int32_t R, int32_t N, int32_t Kd, float alpha, bool accumulate, hipStream_t stream) {
    const dim3 grid((unsigned)((R + 63) / 64), (unsigned)((N + 63) / 64), (unsigned)H);
    hipLaunchKernelGGL((small_gemm_kernel<TA, TB, TC>), grid, dim3(256), 0, stream,
                       reinterpret_cast<const TA*>(a.p), a.s_h, a.s_0, a.s_1,
                       reinterpret_cast<const TB*>(b.p), b.s_h, b.s_0, b.s_1, b_mod, reinterpret_cast<TC*>(c),
                       c_h, c_r, R, N, Kd, alpha, accumulate);
    return hipGetLastError();
}

hipError_t small_gemm_dispatch(const MatView& a, const MatView& b, void* c, bool c_bf16, int64_t c_h, int64_t c_r,
                               int32_t H, int32_t R, int32_t N, int32_t Kd, int32_t b_mod, float alpha,
                               bool accumulate, hipStream_t stream) {
    if (H <= 0 || R <= 0 || N <= 0) return hipSuccess;
    if (H > 65535) return hipErrorInvalidValue;
#define SA_GEMM(TA, TB) \
    return c_bf16 ? gemm_t<TA, TB, uint16_t>(a, b, b_mod, c, c_h, c_r, H, R, N, Kd, alpha, accumulate, stream) \
                  : gemm_t<TA, TB, float>(a, b, b_mod, c, c_h, c_r, H, R, N, Kd, alpha, accumulate, stream)
    if (a.bf16 && b.bf16) SA_GEMM(uint16_t, uint16_t);
    if (a.bf16) SA_GEMM(uint16_t, float);
    if (b.bf16) SA_GEMM(float, uint16_t);
    SA_GEMM(float, float);
#undef SA_GEMM
}

}  // namespace

hipError_t launch_small_gemm(const MatView& a, const MatView& b, void* c, bool c_bf16, int32_t H, int32_t R,
                             int32_t N, int32_t Kd, hipStream_t stream, int32_t b_mod, bool accumulate) {
    if (b_mod <= 0) b_mod = H;
    return small_gemm_dispatch(a, b, c, c_bf16, (int64_t)R * N, N, H, R, N, Kd, b_mod, 1.0f, accumulate, stream);
}

hipError_t launch_small_gemm_general(const GemmDesc& d, hipStream_t stream) {
    return small_gemm_dispatch({d.A, d.a_bf16, d.a_z, d.a_m, d.a_k}, {d.B, d.b_bf16, d.b_z, d.b_k, d.b_n}, d.C,
                               d.c_bf16, d.c_z, d.c_m, d.batch, d.M, d.N, d.K, d.b_mod > 0 ? (int32_t)d.b_mod : d.batch,
                               d.alpha, d.accumulate, stream);
}

hipError_t launch_add(const float* a, const float* b, float* out, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t n4 = n / 4;   // n is a multiple of d (64 or 128)
    hipLaunchKernelGGL(add_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, a, b, out, n4);
    return hipGetLastError();
}

}  // namespace sa

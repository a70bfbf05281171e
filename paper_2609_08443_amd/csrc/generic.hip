// Plain fp32-arithmetic path of the SA sketching step: fp32 inputs (no
// sub-fp32 rounding anywhere) and every shape the fused kernels have no
// instance for.  Same ABI and results as the fused path up to rounding.
//
// Forward (section 3.1): a first kernel computes each token's log-sum-exp of
// its scaled logits over the M prototypes (one wave per token and head, lanes
// over the prototypes); a second computes, for a block of 64 prototypes and
// one work-list segment (a user's tokens inside one token range, the ranges
// cutting the head-major token space into equal parts), A[t,m] = exp(s[t,m] -
// lse[t]) and accumulates A[t,m] V[t,:] over the segment.  A (user, head) held
// by one segment writes its sketch directly; split ones write partials that
// the work list's merge adds in segment order.
//
// Backward (chain rule of the forward; the MRLB sum over R target instances of
// section 4.2 is done first): per token, D_t = sum_m A g, dV_t = sum_m A dY_m,
// dS = A (g - D_t), dK_t = scale sum_m dS P_m with g_m = V_t . dY_m; then
// dP[h,m] = scale sum_t dS[t,m] K_t over token chunks, summed in chunk order.
// With per-user prototypes (P, dP [B,H,M,d]) each user's tokens form one chunk
// and write their dP block directly.
#include "sa_internal.h"

namespace sa {

namespace {

template <bool BF16>
__device__ inline float ld(const void* p, int64_t i) {
    if constexpr (BF16) {
        const uint16_t v = reinterpret_cast<const uint16_t*>(p)[i];
        return __uint_as_float((uint32_t)v << 16);
    } else {
        return reinterpret_cast<const float*>(p)[i];
    }
}

__device__ inline int64_t clampT(int64_t x, int64_t T) { return x < 0 ? 0 : (x > T ? T : x); }

// user owning token t, or -1 (binary search over non-decreasing offsets)
__device__ inline int64_t user_of(const int64_t* off, int64_t B, int64_t T, int64_t t) {
    int64_t lo = 0, hi = B - 1;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (clampT(off[mid], T) <= t) lo = mid; else hi = mid - 1;
    }
    if (B <= 0) return -1;
    if (clampT(off[lo], T) <= t && t < clampT(off[lo + 1], T)) return lo;
    return -1;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) v += __shfl_xor(v, k, 64);
    return v;
}

// ---------------------------------------------------------------- forward
// one wave per (t, h): lane l takes prototypes l, l + 64, ...; each lane keeps
// a running maximum and a sum rescaled to it, and the wave combines them
// (maximum first, then the rescaled sums)
template <bool BF16, int D>
__global__ __launch_bounds__(256) void lse_wave_kernel(const void* __restrict__ K, const void* __restrict__ P,
                                                       const int64_t* __restrict__ off, int64_t B, int64_t T,
                                                       int32_t H, int32_t M, float scale, bool p_user,
                                                       float* __restrict__ lse) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= T * H) return;
    const int64_t t = i / H;
    const int32_t h = (int32_t)(i % H);
    int64_t pi = h;
    if (p_user) {
        const int64_t b = user_of(off, B, T, t);
        if (b < 0) return;   // outside every user: no lse row
        pi = b * H + h;
    }
    float kr[D];
#pragma unroll
    for (int j = 0; j < D; ++j) kr[j] = ld<BF16>(K, (t * H + h) * D + j);
    float mu = -INFINITY, z = 0.f;
    for (int m = lane; m < M; m += 64) {
        float s = 0.f;
        const int64_t pb = (pi * M + m) * D;
#pragma unroll
        for (int j = 0; j < D; ++j) s = __builtin_fmaf(kr[j], ld<BF16>(P, pb + j), s);
        s *= scale;
        if (s > mu) {
            z = z * expf(mu - s) + 1.0f;
            mu = s;
        } else {
            z += expf(s - mu);
        }
    }
    float mw = mu;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) mw = fmaxf(mw, __shfl_xor(mw, k, 64));
    const float zw = wave_sum(mu == -INFINITY ? 0.f : z * expf(mu - mw));
    if (lane == 0) lse[i] = mw + logf(zw);
}

// block = 256 threads: 64 prototypes x 4 column quarters; grid = (ranges,
// ceil(M/64)); the block takes the segments of its range in order
template <bool BF16, int D>
__global__ __launch_bounds__(256) void agg_items_kernel(const void* __restrict__ K, const void* __restrict__ V,
                                                        const void* __restrict__ P,
                                                        const int32_t* __restrict__ items,
                                                        const int32_t* __restrict__ wg_start, int64_t max_items,
                                                        int64_t B, int64_t T, int32_t H, int32_t M, float scale,
                                                        bool p_user, const float* __restrict__ lse,
                                                        float* __restrict__ sketch, float* __restrict__ partials) {
    constexpr int dq = D / 4;
    const int mi = threadIdx.x >> 2, jq = threadIdx.x & 3;
    const int m = blockIdx.y * 64 + mi;
    const int jb = jq * dq;
    const bool mv = m < M;
    const int64_t k0 = wg_start[blockIdx.x], k1 = wg_start[blockIdx.x + 1];
    if (k0 < 0 || k1 < k0 || k1 > max_items) return;
    for (int64_t k = k0; k < k1; ++k) {
        const int32_t* it = items + k * IT_WORDS;
        const int b = it[IT_B], h = it[IT_H], t0 = it[IT_T0], t1 = it[IT_T1];
        if (b < 0 || b >= B || h < 0 || h >= H || t0 < 0 || t1 < t0 || t1 > T) continue;
        const int64_t pair = (int64_t)b * H + h;
        float pr[dq], acc[dq];
#pragma unroll
        for (int c = 0; c < dq; ++c) {
            pr[c] = mv ? ld<BF16>(P, ((p_user ? pair : (int64_t)h) * M + m) * D + jb + c) : 0.f;
            acc[c] = 0.f;
        }
        for (int64_t t = t0; t < t1; ++t) {
            const int64_t base = (t * H + h) * D + jb;
            float ps = 0.f;
#pragma unroll
            for (int c = 0; c < dq; ++c) ps = __builtin_fmaf(ld<BF16>(K, base + c), pr[c], ps);
            ps += __shfl_xor(ps, 1, 64);
            ps += __shfl_xor(ps, 2, 64);
            const float aw = expf(ps * scale - lse[t * H + h]);
#pragma unroll
            for (int c = 0; c < dq; ++c) acc[c] = __builtin_fmaf(aw, ld<BF16>(V, base + c), acc[c]);
        }
        if (mv) {
            float* out = (it[IT_SPLIT] ? partials + k * (int64_t)M * D : sketch + pair * (int64_t)M * D) +
                         (int64_t)m * D + jb;
#pragma unroll
            for (int c = 0; c < dq; ++c) out[c] = acc[c];
        }
    }
}

// ---------------------------------------------------------------- backward
__global__ __launch_bounds__(256) void dy_kernel(const float* __restrict__ ds, int64_t B,
                                                 int32_t R, int32_t H, int64_t MD,
                                                 float* __restrict__ dY) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t n = B * H * MD;
    if (i >= n) return;
    const int64_t b = i / (H * MD);
    const int64_t rest = i % (H * MD);
    float s = 0.f;
    for (int r = 0; r < R; ++r) s += ds[(b * R + r) * H * MD + rest];
    dY[i] = s;
}

// one wave per (t, h); lanes over the d columns (d/64 per lane).  Dynamic LDS:
// per wave A[M] and g[M] of the token.
template <bool BF16, int D>
__global__ __launch_bounds__(256) void bwd_token_kernel(
    const void* __restrict__ K, const void* __restrict__ V, const void* __restrict__ P,
    const int64_t* __restrict__ off, int64_t B, int64_t T, int32_t H, int32_t M,
    float scale, const float* __restrict__ dY, const float* __restrict__ lse,
    float* __restrict__ Dbuf, float* __restrict__ dK, float* __restrict__ dV, bool p_user) {
    extern __shared__ float sm[];
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    float* aw = sm + (size_t)w * 2 * M;
    float* gw = aw + M;
    const int64_t i = (int64_t)blockIdx.x * 4 + w;
    if (i >= T * H) return;
    const int64_t t = i / H;
    const int32_t h = (int32_t)(i % H);
    constexpr int d = D;
    constexpr int jpl = D / 64;
    const int64_t rowb = (t * H + h) * d;
    const int64_t b = user_of(off, B, T, t);
    if (b < 0) {
        for (int c = 0; c < jpl; ++c) {
            dK[rowb + lane + 64 * c] = 0.f;
            dV[rowb + lane + 64 * c] = 0.f;
        }
        if (lane == 0) Dbuf[i] = 0.f;
        return;
    }
    float kr[2], vr[2], dv[2] = {0.f, 0.f}, dk[2] = {0.f, 0.f};
    for (int c = 0; c < jpl; ++c) {
        kr[c] = ld<BF16>(K, rowb + lane + 64 * c);
        vr[c] = ld<BF16>(V, rowb + lane + 64 * c);
    }
    const float l = lse[i];
    const float* dYb = dY + ((b * H + h) * (int64_t)M) * d;
    const int64_t pkey = p_user ? b * H + h : h;
    float Dacc = 0.f;
    for (int m = 0; m < M; ++m) {
        const int64_t pb = (pkey * M + m) * d;
        float s = 0.f, g = 0.f;
        for (int c = 0; c < jpl; ++c) {
            s = __builtin_fmaf(kr[c], ld<BF16>(P, pb + lane + 64 * c), s);
            g = __builtin_fmaf(vr[c], dYb[(int64_t)m * d + lane + 64 * c], g);
        }
        s = wave_sum(s);
        g = wave_sum(g);
        const float a = expf(s * scale - l);
        Dacc += a * g;
        for (int c = 0; c < jpl; ++c) dv[c] = __builtin_fmaf(a, dYb[(int64_t)m * d + lane + 64 * c], dv[c]);
        // a and g are the same in every lane; each lane stores and later
        // reloads its own copy, so no cross-lane ordering is needed
        aw[m] = a;
        gw[m] = g;
    }
    for (int m = 0; m < M; ++m) {
        const float dS = aw[m] * (gw[m] - Dacc);
        const int64_t pb = (pkey * M + m) * d;
        for (int c = 0; c < jpl; ++c) dk[c] = __builtin_fmaf(dS, ld<BF16>(P, pb + lane + 64 * c), dk[c]);
    }
    for (int c = 0; c < jpl; ++c) {
        dK[rowb + lane + 64 * c] = scale * dk[c];
        dV[rowb + lane + 64 * c] = dv[c];
    }
    if (lane == 0) Dbuf[i] = Dacc;
}

// grid = (H * ceil(M/64), n_chunks, or B with per-user prototypes); block = 64
// prototypes x 4 column quarters
template <bool BF16, int D>
__global__ __launch_bounds__(256) void bwd_dp_kernel(
    const void* __restrict__ K, const void* __restrict__ V, const void* __restrict__ P,
    const int64_t* __restrict__ off, int64_t B, int64_t T, int32_t H, int32_t M,
    float scale, const float* __restrict__ dY, const float* __restrict__ lse,
    const float* __restrict__ Dbuf, int64_t chunk, bool p_user, float* __restrict__ part) {
    const int mblocks = (M + 63) / 64;
    const int32_t h = blockIdx.x / mblocks;
    const int mb = blockIdx.x % mblocks;
    const int mi = threadIdx.x >> 2, jq = threadIdx.x & 3;
    const int m = mb * 64 + mi;
    const bool mv = m < M;
    constexpr int d = D;
    constexpr int dq = D / 4;
    const int jb = jq * dq;
    const int64_t pkey = p_user ? (int64_t)blockIdx.y * H + h : h;
    float pr[dq], yr[dq], acc[dq];
    for (int c = 0; c < dq; ++c) {
        pr[c] = mv ? ld<BF16>(P, (pkey * M + m) * d + jb + c) : 0.f;
        acc[c] = 0.f;
        yr[c] = 0.f;
    }
    int64_t ta, tb;
    if (p_user) {
        ta = clampT(off[blockIdx.y], T);
        tb = clampT(off[blockIdx.y + 1], T);
        if (tb < ta) tb = ta;
    } else {
        ta = (int64_t)blockIdx.y * chunk;
        tb = ta + chunk < T ? ta + chunk : T;
    }
    int64_t cur_b = -2, bend = -1;
    for (int64_t t = ta; t < tb; ++t) {
        if (t >= bend || cur_b < 0) {
            const int64_t nb = user_of(off, B, T, t);
            if (nb != cur_b) {
                cur_b = nb;
                if (nb >= 0) {
                    const float* src = dY + (((nb * H + h) * (int64_t)M) + (mv ? m : 0)) * d + jb;
                    for (int c = 0; c < dq; ++c) yr[c] = src[c];
                    bend = clampT(off[nb + 1], T);
                } else {
                    bend = t + 1;
                }
            }
        }
        if (cur_b < 0) continue;
        const int64_t base = (t * H + h) * d + jb;
        float ps = 0.f, gs = 0.f;
        for (int c = 0; c < dq; ++c) {
            ps = __builtin_fmaf(ld<BF16>(K, base + c), pr[c], ps);
            gs = __builtin_fmaf(ld<BF16>(V, base + c), yr[c], gs);
        }
        ps += __shfl_xor(ps, 1, 64);
        ps += __shfl_xor(ps, 2, 64);
        gs += __shfl_xor(gs, 1, 64);
        gs += __shfl_xor(gs, 2, 64);
        const float a = expf(ps * scale - lse[t * H + h]);
        const float dS = a * (gs - Dbuf[t * H + h]);
        for (int c = 0; c < dq; ++c) acc[c] = __builtin_fmaf(dS, ld<BF16>(K, base + c), acc[c]);
    }
    if (mv) {
        // per-user prototypes: pkey = blockIdx.y * H + h, the user's dP block
        float* out = part + ((p_user ? pkey : (int64_t)blockIdx.y * H + h) * M + m) * d + jb;
        for (int c = 0; c < dq; ++c) out[c] = scale * acc[c];
    }
}

__global__ __launch_bounds__(256) void dp_reduce_kernel(const float* __restrict__ part,
                                                        int32_t n_chunks, int64_t n,
                                                        float* __restrict__ dP) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float s = 0.f;
    for (int c = 0; c < n_chunks; ++c) s += part[(int64_t)c * n + i];
    dP[i] = s;
}

template <bool BF16, int D>
hipError_t fwd_impl(const void* K, const void* V, const void* P, const int64_t* off, int64_t B,
                    int64_t T, int32_t H, int32_t M, float scale, bool p_user, float* sketch,
                    float* lse, const GenericFwdItems& w, hipStream_t stream) {
    if (T * H > 0) {
        hipLaunchKernelGGL((lse_wave_kernel<BF16, D>), dim3((unsigned)((T * H + 3) / 4)), dim3(256), 0,
                           stream, K, P, off, B, T, H, M, scale, p_user, lse);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (w.n_ranges > 0) {
        hipLaunchKernelGGL((agg_items_kernel<BF16, D>), dim3((unsigned)w.n_ranges, (unsigned)((M + 63) / 64)),
                           dim3(256), 0, stream, K, V, P, w.items, w.wg_start, w.max_items, B, T, H, M, scale,
                           p_user, lse, sketch, w.partials);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <bool BF16, int D>
hipError_t bwd_impl(const void* K, const void* V, const void* P, const int64_t* off, int64_t B,
                    int64_t T, int32_t H, int32_t M, int32_t d, float scale, const float* dY,
                    const float* lse, float* Dbuf, float* dK, float* dV, float* dP, float* part,
                    int32_t n_chunks, bool p_user, hipStream_t stream) {
    hipError_t e;
    if (T * H > 0) {
        const size_t lds = (size_t)4 * 2 * M * sizeof(float);
        auto kern = bwd_token_kernel<BF16, D>;
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, dim3((unsigned)((T * H + 3) / 4)), dim3(256), lds, stream, K, V,
                           P, off, B, T, H, M, scale, dY, lse, Dbuf, dK, dV, p_user);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t chunk = T > 0 ? (T + n_chunks - 1) / n_chunks : 1;
    if (p_user) {
        if (B <= 0) return hipSuccess;
        hipLaunchKernelGGL((bwd_dp_kernel<BF16, D>), dim3((unsigned)(H * ((M + 63) / 64)), (unsigned)B),
                           dim3(256), 0, stream, K, V, P, off, B, T, H, M, scale, dY, lse, Dbuf, chunk, true,
                           dP);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((bwd_dp_kernel<BF16, D>),
                       dim3((unsigned)(H * ((M + 63) / 64)), (unsigned)n_chunks), dim3(256), 0,
                       stream, K, V, P, off, B, T, H, M, scale, dY, lse, Dbuf, chunk, false, part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)H * M * d;
    hipLaunchKernelGGL(dp_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                       part, n_chunks, n, dP);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_generic_fwd(const void* K, const void* V, const void* P, const int64_t* off,
                              int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                              bool bf16, float* sketch, float* lse_out, const GenericFwdItems& w,
                              hipStream_t stream, bool p_user) {
#define SA_FWD(BF, DD) fwd_impl<BF, DD>(K, V, P, off, B, T, H, M, scale, p_user, sketch, lse_out, w, stream)
    if (d == 64) return bf16 ? SA_FWD(true, 64) : SA_FWD(false, 64);
    if (d == 128) return bf16 ? SA_FWD(true, 128) : SA_FWD(false, 128);
#undef SA_FWD
    return hipErrorInvalidValue;
}

hipError_t launch_dy_reduce(const float* dsketch, int64_t B, int32_t R, int32_t H, int64_t MD,
                            float* dY, hipStream_t stream) {
    const int64_t n = B * H * MD;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(dy_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                       dsketch, B, R, H, MD, dY);
    return hipGetLastError();
}

int32_t generic_dp_chunks(int64_t T, int32_t H, int32_t M) {
    // enough blocks to fill the chip a few times over
    const int64_t blocks = (int64_t)H * ((M + 63) / 64);
    int64_t c = (2048 + blocks - 1) / blocks;
    if (c > T) c = T;
    if (c < 1) c = 1;
    if (c > 4096) c = 4096;
    return (int32_t)c;
}

hipError_t launch_generic_bwd(const void* K, const void* V, const void* P, const int64_t* off,
                              int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                              bool bf16, const float* dY, const float* lse, float* Dbuf,
                              float* dK, float* dV, float* dP, float* part, int32_t n_chunks,
                              hipStream_t stream, bool p_user) {
#define SA_BWD(BF, DD) bwd_impl<BF, DD>(K, V, P, off, B, T, H, M, d, scale, dY, lse, Dbuf, dK, dV, dP, part, n_chunks, p_user, stream)
    if (d == 64) return bf16 ? SA_BWD(true, 64) : SA_BWD(false, 64);
    if (d == 128) return bf16 ? SA_BWD(true, 128) : SA_BWD(false, 128);
#undef SA_BWD
    return hipErrorInvalidValue;
}

}  // namespace sa

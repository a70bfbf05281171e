// Ragged scheduling: the work list of (user, head, token range) segments and
// the split-L merge of partial sketches.
//
// Users are ragged (section 4.4: fused kernel under ragged batching).  The
// (head, token) pairs are laid out head-major in one index space of length
// H*T and cut into equal ranges of C tokens, one range per workgroup, so every
// workgroup gets the same number of tokens whatever the length mix.  A (user,
// head) pair is cut at range boundaries into segments.  Because the softmax is
// taken over prototypes for each token separately (section 3.1, A sums to 1
// over prototypes), the sketch of a user is a plain sum over its tokens, so
// the partial sketches of a user cut across ranges merge by addition; there is
// no rescaling step as in a token-wise softmax.
#include "sa_internal.h"

namespace sa {

namespace {

__device__ inline int64_t clamp64(int64_t x, int64_t lo, int64_t hi) {
    return x < lo ? lo : (x > hi ? hi : x);
}

// Inclusive scan of one int64 per thread over a block of kWorklistThreads.
__device__ int64_t block_inclusive_scan(int64_t v, int64_t* buf) {
    const int tid = threadIdx.x;
    buf[tid] = v;
    __syncthreads();
    for (int off = 1; off < kWorklistThreads; off <<= 1) {
        int64_t add = tid >= off ? buf[tid - off] : 0;
        __syncthreads();
        buf[tid] += add;
        __syncthreads();
    }
    int64_t r = buf[tid];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kWorklistThreads) void worklist_kernel(
    const int64_t* __restrict__ offsets, int64_t B, int64_t T, int32_t H, int64_t C,
    int64_t n_ranges, int32_t* __restrict__ items, int64_t max_items,
    int32_t* __restrict__ wg_start, int32_t* __restrict__ pair_start,
    int64_t* __restrict__ n_items) {
    __shared__ int64_t scan_buf[kWorklistThreads];
    const int tid = threadIdx.x;
    if (wg_start) {
        for (int64_t i = tid; i <= n_ranges; i += kWorklistThreads) wg_start[i] = -1;
    }
    __syncthreads();
    const int64_t npairs = (int64_t)H * B;
    int64_t carry = 0;
    for (int64_t base = 0; base < npairs; base += kWorklistThreads) {
        const int64_t p = base + tid;
        int64_t n = 0, lo = 0, hi = 0, i0 = 0;
        int32_t h = 0, b = 0;
        if (p < npairs) {
            h = (int32_t)(p / B);
            b = (int32_t)(p % B);
            lo = clamp64(offsets[b], 0, T);
            hi = clamp64(offsets[b + 1], 0, T);
            if (hi > lo) {
                const int64_t g0 = (int64_t)h * T + lo;
                const int64_t g1 = (int64_t)h * T + hi - 1;
                i0 = g0 / C;
                n = g1 / C - i0 + 1;
            }
        }
        const int64_t incl = block_inclusive_scan(n, scan_buf);
        const int64_t start = carry + incl - n;
        if (p < npairs && pair_start) pair_start[p] = (int32_t)(start < max_items ? start : max_items);
        for (int64_t s = 0; s < n; ++s) {
            const int64_t k = start + s;
            if (k >= max_items) break;
            const int64_t r = i0 + s;
            const int64_t t0 = lo > r * C - (int64_t)h * T ? lo : r * C - (int64_t)h * T;
            const int64_t t1 = hi < (r + 1) * C - (int64_t)h * T ? hi : (r + 1) * C - (int64_t)h * T;
            int32_t* it = items + k * IT_WORDS;
            it[IT_B] = b;
            it[IT_H] = h;
            it[IT_T0] = (int32_t)t0;
            it[IT_T1] = (int32_t)t1;
            it[IT_RANGE] = (int32_t)r;
            it[IT_SPLIT] = n > 1 ? 1 : 0;
            it[IT_PAIR_FIRST] = (int32_t)start;
            it[7] = 0;
            if (wg_start && r < n_ranges && (int64_t)h * T + t0 == r * C) wg_start[r] = (int32_t)k;
        }
        // the last thread's inclusive value is the block total
        if (tid == kWorklistThreads - 1) scan_buf[0] = incl;
        __syncthreads();
        carry += scan_buf[0];
        __syncthreads();
    }
    if (tid == 0) {
        const int64_t fin = carry < max_items ? carry : max_items;
        if (pair_start) pair_start[npairs] = (int32_t)fin;
        if (wg_start) wg_start[n_ranges] = (int32_t)fin;
        *n_items = fin;
    }
}

__global__ __launch_bounds__(256) void merge_kernel(const int32_t* __restrict__ pair_start,
                                                    int64_t B, int32_t H, int64_t max_items,
                                                    const float* __restrict__ partials,
                                                    int64_t MD, float* __restrict__ sketch) {
    const int64_t p = blockIdx.x;  // head-major pair index h*B + b
    int64_t s0 = pair_start[p], s1 = pair_start[p + 1];
    s0 = s0 < 0 ? 0 : (s0 > max_items ? max_items : s0);
    s1 = s1 < s0 ? s0 : (s1 > max_items ? max_items : s1);
    if (s1 - s0 == 1) return;  // written directly by the forward kernel
    const int64_t idx = ((int64_t)blockIdx.y * 256 + threadIdx.x) * 4;
    if (idx >= MD) return;
    const int64_t h = p / B, b = p % B;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8   // several segments' loads in flight; the sum keeps segment order
    for (int64_t k = s0; k < s1; ++k) {
        const float4 v = *reinterpret_cast<const float4*>(partials + k * MD + idx);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    *reinterpret_cast<float4*>(sketch + (b * H + h) * MD + idx) = acc;
}

}  // namespace

hipError_t launch_worklist(const int64_t* offsets, int64_t B, int64_t T, int32_t H, int64_t C,
                           int64_t n_ranges, int32_t* items, int64_t max_items,
                           int32_t* wg_start, int32_t* pair_start, int64_t* n_items,
                           hipStream_t stream) {
    hipLaunchKernelGGL(worklist_kernel, dim3(1), dim3(kWorklistThreads), 0, stream, offsets, B,
                       T, H, C, n_ranges, items, max_items, wg_start, pair_start, n_items);
    return hipGetLastError();
}

hipError_t launch_merge(const int32_t* pair_start, int64_t B, int32_t H, int64_t max_items,
                        const float* partials, int64_t MD, float* sketch, hipStream_t stream) {
    const int64_t npairs = (int64_t)H * B;
    if (npairs == 0) return hipSuccess;
    // MD is a multiple of 4 (d is 64 or 128)
    dim3 grid((unsigned)npairs, (unsigned)((MD + 1023) / 1024));
    hipLaunchKernelGGL(merge_kernel, grid, dim3(256), 0, stream, pair_start, B, H, max_items,
                       partials, MD, sketch);
    return hipGetLastError();
}

}  // namespace sa

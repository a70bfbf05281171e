// Internal declarations shared by the host library and the kernel translation
// units of the SA sketching library (gfx950).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/sa_sketch.h"

namespace sa {

// ---------------------------------------------------------------------------
// work list item: 8 x int32 (see sa_build_worklist in sa_sketch.h)
// ---------------------------------------------------------------------------
enum : int { IT_B = 0, IT_H = 1, IT_T0 = 2, IT_T1 = 3, IT_RANGE = 4, IT_SPLIT = 5,
             IT_PAIR_FIRST = 6, IT_WORDS = 8 };

constexpr int kTileTokens = 32;     // tokens per MFMA tile (rows of the 32x32 output)
constexpr int kWorklistThreads = 1024;

// Brackets the launches made in its scope with HIP events on `stream` when
// kernel timing is enabled on the calling thread (sa_profile_enable).
class ProfScope {
  public:
    ProfScope(const char* name, hipStream_t stream);
    ~ProfScope();
    ProfScope(const ProfScope&) = delete;
    ProfScope& operator=(const ProfScope&) = delete;

  private:
    hipStream_t stream_;
    const char* name_ = nullptr;
    hipEvent_t start_ = nullptr, stop_ = nullptr;
    bool active_ = false;
};

// ---------------------------------------------------------------------------
// launchers (each returns hipSuccess or the launch error)
// ---------------------------------------------------------------------------

// Work list over the head-major (h, t) index space cut into ranges of C tokens.
// wg_start[n_ranges + 1] and pair_start[H*B + 1] may be null.
hipError_t launch_worklist(const int64_t* offsets, int64_t B, int64_t T, int32_t H,
                           int64_t C, int64_t n_ranges, int32_t* items, int64_t max_items,
                           int32_t* wg_start, int32_t* pair_start, int64_t* n_items,
                           hipStream_t stream);

// sketch[b,h] = sum of the partial sketches of a split (user, head) pair, in
// segment order; zero for empty pairs; untouched for single-segment pairs.
hipError_t launch_merge(const int32_t* pair_start, int64_t B, int32_t H, int64_t max_items,
                        const float* partials, int64_t MD, float* sketch, hipStream_t stream);

// Fused bf16 forward (matrix cores).  Returns hipErrorInvalidValue for a
// (d, M) it has no instance for.
struct FusedFwdArgs {
    const uint16_t* K;
    const uint16_t* V;
    const uint16_t* P;
    const int32_t* items;
    const int32_t* wg_start;
    int64_t n_ranges;
    int64_t max_items;
    int64_t T;
    int32_t B, H, M, d;
    float scale;
    float* sketch;
    float* lse;
    float* partials;
    bool p_user;   // P is [B,H,M,d], one prototype block per user (stacked layers)
};
bool fused_fwd_supported(int32_t M, int32_t d);
size_t fused_fwd_lds_bytes(int32_t M, int32_t d);
hipError_t fused_fwd_occupancy(int32_t M, int32_t d, int* blocks_per_cu);
hipError_t launch_fused_fwd(const FusedFwdArgs& a, hipStream_t stream);

// Fused bf16 backward (matrix cores): prep, token-side and prototype-side
// kernels plus the per-head sum of the dP partials.
struct FusedBwdArgs {
    const uint16_t* K;
    const uint16_t* V;
    const uint16_t* P;
    const float* dsketch;
    const float* lse;
    const int32_t* items;
    const int32_t* wg_start;
    const int32_t* pair_start;
    int64_t n_ranges;
    int64_t max_items;
    int64_t B, T;
    int32_t H, M, d, R;
    float scale;
    uint16_t* Ymj;       // [B,H,M,d] bf16
    uint16_t* Yjm;       // [B,H,d,M] bf16, prototype index permuted within 16-groups
    uint16_t* Pjm;       // [H,d,M] bf16, likewise
    float* Dbuf;         // [T,H]
    float* partials;     // [max_items][M][d]
    float* dK;
    float* dV;
    float* dP;
    // When non-null, K and V are the same tensor X (the SA layer, whose value
    // is its history and whose key projection is absorbed into P): the token
    // side writes dX = dV + dK here instead of dK and dV.
    float* dX;
    // P (and Pjm) hold one prototype block per (user, head) and dP is [B,H,M,d],
    // each pair's gradient (stacked layers after the first)
    bool p_user;
    // with dX: add the gradient to dX instead of overwriting it
    bool dx_add = false;
};
bool fused_bwd_supported(int32_t M, int32_t d);
int32_t fused_bwd_part(int32_t M, int32_t d);
// token-side workgroups resident per CU (sizes the work-list ranges)
int32_t fused_bwd_ranges_per_cu();
hipError_t launch_fused_bwd(const FusedBwdArgs& a, hipStream_t stream);

// Token-wise normalised forward (sa_sketch_fwd_tokenwise).
bool tokenwise_fused_supported(int32_t M, int32_t d);
hipError_t launch_tokenwise_fused(const int32_t* items, const int32_t* wg_start, int64_t n_ranges,
                                  int64_t max_items, const void* K, const void* V, const void* P,
                                  int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                                  float* sketch, float* lse_m, float* partials, float* stats,
                                  hipStream_t stream);
hipError_t launch_tokenwise_merge(const int32_t* pair_start, int64_t B, int32_t H, int32_t M, int32_t d,
                                  int64_t max_items, const float* partials, const float* stats,
                                  float* sketch, float* lse_m, hipStream_t stream);
hipError_t launch_tokenwise_generic(const void* K, const void* V, const void* P, const int64_t* offsets,
                                    int64_t B, int32_t H, int32_t M, int32_t d, float scale, bool bf16,
                                    float* sketch, float* lse_m, hipStream_t stream);

// Batched product for the projections and the FFN of the SA layers (fp32
// accumulation): C[z][r][c] = sum_k A[z](r, k) B[z % b_mod](k, c), r < R, c < N,
// k < Kd, z < H batches, C row-major [R][N] per batch, bf16 (rounded) or fp32.
// Operand element (i, j) of batch z sits at p[z * s_h + i * s_0 + j * s_1], so a
// transpose is a swap of strides; b_mod <= 0 means b_mod = H (one B per batch).
// With accumulate the product is added to C's values.
struct MatView {
    const void* p;
    bool bf16;
    int64_t s_h, s_0, s_1;
};
hipError_t launch_small_gemm(const MatView& a, const MatView& b, void* c, bool c_bf16, int32_t H, int32_t R,
                             int32_t N, int32_t Kd, hipStream_t stream, int32_t b_mod = 0,
                             bool accumulate = false);
// General batched product C[z](m, n) = alpha sum_k A[z](m, k) B[z](k, n) (+ C with
// accumulate), element (z, m, k) of A at A[z a_z + m a_m + k a_k], (z, k, n) of B at
// B[z b_z + k b_k + n b_n], (z, m, n) of C at C[z c_z + m c_m + n]; fp32 accumulation.
// bf16 operands contiguous along k or along m (n), with k a multiple of 64 and
// 16-byte aligned pieces, run on the matrix cores (gemm.hip); the rest on the
// register-tiled fp32 product (layer.hip).
struct GemmDesc {
    const void* A;
    bool a_bf16;
    int64_t a_z, a_m, a_k;
    const void* B;
    bool b_bf16;
    int64_t b_z, b_k, b_n;
    void* C;
    bool c_bf16;
    int64_t c_z, c_m;
    int32_t M, N, K, batch;
    float alpha;
    bool accumulate;
    int64_t b_mod = 0;        // > 0: B's batch index is z % b_mod (weights shared across users)
    bool round_bf16 = false;  // fp32 operands may be rounded to bf16 (matrix cores)
};
bool gemm_on_matrix_cores(const GemmDesc& d);
// number of compute units of the current device (read once per device)
int device_cus();
// The bf16-operand product on one given tile shape (0 .. gemm_tile_shapes() - 1,
// the largest first) instead of the one launch_gemm picks (shape < 0: as
// launch_gemm); hipErrorInvalidValue where that shape cannot take the product.
int gemm_tile_shapes();
hipError_t launch_gemm_tile_shape(const GemmDesc& d, int shape, hipStream_t stream);
hipError_t launch_gemm(const GemmDesc& d, hipStream_t stream);
hipError_t launch_small_gemm_general(const GemmDesc& d, hipStream_t stream);

// Reordered single-query STCA rows (stca.hip), over [rows][k] fp32 logits already
// scaled: lse and alpha = exp(s - lse) in bf16 or fp32; the backward writes
// ds = scale alpha (da - <alpha, da>).
hipError_t launch_stca_softmax(const void* S, bool s_bf16, int64_t rows, int32_t k, bool bf16, void* alpha,
                               float* lse, hipStream_t stream);
hipError_t launch_stca_softmax_bwd(const void* S, bool s_bf16, const float* lse, const float* dA, int64_t rows,
                                   int32_t k, float scale, bool bf16, void* ds, hipStream_t stream);
hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t stream);

// Stacked-SA refinement (block.hip).  add_ln: one row of d features per
// (user, head, prototype): out[r] = LN(x[r mod x_rows] + y[r]) * gamma[h] + beta[h],
// h = (r / M) % H; x fp32 or bf16 (the shared prototypes broadcast over users
// when x_rows = H * M), y fp32, gamma / beta [H][d] in the parameter dtype.
// With sum_out non-null the pre-norm sum x + y is also written there.
hipError_t launch_add_ln(const void* x, bool x_bf16, int64_t x_rows, const float* y, const void* gamma,
                         const void* beta, bool p_bf16, int64_t rows, int32_t H, int32_t M, int32_t d, float eps,
                         float* out, hipStream_t stream, float* sum_out = nullptr);
// g = silu(g) * u elementwise (n fp32 values, n a multiple of 4)
hipError_t launch_swiglu_gate(float* g, const float* u, int64_t n, hipStream_t stream);
// z = silu(g) * u, keeping g and u
hipError_t launch_swiglu_fwd(const float* g, const float* u, float* z, int64_t n, hipStream_t stream);
// backward of z = silu(g) * u: dz_dg holds dz on entry and dg on exit; du written
hipError_t launch_swiglu_bwd(float* dz_dg, const float* g, const float* u, float* du, int64_t n,
                             hipStream_t stream);
// Backward of out = LN(y) * gamma[h] + beta[h] over the B * H * M rows of [B,H,M,d]
// (fp32): with dout = dy1 + dy2 (dy2 may be null), writes dx (aliasing neither),
// the per-row (mean, rstd) into stats [rows], and the gamma / beta gradients,
// [H][d] each, to dgamma_dbeta and dgamma_dbeta + ostride.  The column sums run
// over nch chunks of the (user, prototype) rows of each head into colpart
// [nch][H][2][d], then over the chunks in order (deterministic).
hipError_t launch_ln_bwd(const float* dy1, const float* dy2, const float* y, const void* gamma, bool p_bf16,
                         int64_t B, int32_t H, int32_t M, int32_t d, float eps, float* dx, float2* stats,
                         float* colpart, int64_t nch, float* dgamma_dbeta, int64_t ostride, hipStream_t stream);
// p[i] = v for i < n (fp32)
hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t stream);
// out[h][i] = sum over b, in order, of part[b * H + h][i], i < n (fp32)
hipError_t launch_sum_users(const float* part, int64_t B, int32_t H, int64_t n, float* out, hipStream_t stream);

// out = a + b elementwise (n fp32 values, n a multiple of 4, 16-byte aligned)
hipError_t launch_add(const float* a, const float* b, float* out, int64_t n, hipStream_t stream);

// Plain fp32-arithmetic path (fp32 or bf16 inputs).
// Work list of the plain forward's aggregation (the fused forward's format:
// items and per-range starts from launch_worklist) and the partial sketches of
// (user, head) pairs split across ranges, merged by launch_merge.
struct GenericFwdItems {
    const int32_t* items = nullptr;
    const int32_t* wg_start = nullptr;
    int64_t n_ranges = 0, max_items = 0;
    float* partials = nullptr;
};
hipError_t launch_generic_fwd(const void* K, const void* V, const void* P, const int64_t* off, int64_t B,
                              int64_t T, int32_t H, int32_t M, int32_t d, float scale, bool bf16, float* sketch,
                              float* lse_out, const GenericFwdItems& w, hipStream_t stream, bool p_user);

// dY[b,h] = sum_r dsketch[b,r,h]  (fp32, [B,H,M,d])
hipError_t launch_dy_reduce(const float* dsketch, int64_t B, int32_t R, int32_t H, int64_t MD,
                            float* dY, hipStream_t stream);

hipError_t launch_generic_bwd(const void* K, const void* V, const void* P,
                              const int64_t* offsets, int64_t B, int64_t T, int32_t H,
                              int32_t M, int32_t d, float scale, bool bf16, const float* dY,
                              const float* lse, float* Dbuf, float* dK, float* dV, float* dP,
                              float* dp_partials, int32_t n_chunks, hipStream_t stream,
                              bool p_user = false);

// number of token chunks the generic dP kernel uses (sizes its partial buffer)
int32_t generic_dp_chunks(int64_t T, int32_t H, int32_t M);

}  // namespace sa

/*
 * sa_sketch.h -- C ABI of the Sketch Attention (SA) sketching step on one
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (SequenceO1, section 3.1 "Sketch Attention", equations for the
 * affinities S, the prototype-wise softmax A and the sketch; Appendix B steps
 * 1-3; section 4.4 "FlashSA" for the fused, streaming evaluation with softmax
 * statistics kept instead of the k x n scores):
 *
 *   for every user b, head h and token t of user b:
 *     s[t,m]   = scale * <K[t,h,:], P[h,m,:]>                  m = 0..M-1
 *     A[t,m]   = exp(s[t,m]) / sum_m' exp(s[t,m'])             normalised over the
 *                                                              M prototypes, per token
 *     sketch[b,h,m,:] = sum_{t in user b} A[t,m] * V[t,h,:]
 *     lse[t,h] = log sum_m exp(s[t,m])
 *
 * K and P are the already projected keys (X W_K) and prototypes (P W_Q) of the
 * paper; V is the tensor aggregated into the slots (the paper's X).  Heads are
 * independent SA instances, each with its own P[h]; H = 1 is exactly the
 * paper's single-head SA.  An empty user (no tokens) gets a zero sketch.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Every pointer argument except the scalar ones is DEVICE memory owned by
 *    the caller.  The library keeps no pointer after the call returns and
 *    allocates no device memory of its own: scratch space is the caller's
 *    `workspace` buffer, sized by the matching *_workspace_size() call.
 *  * Work is enqueued on `stream` (a hipStream_t passed as void*; NULL = the
 *    default stream) without any host synchronisation, except in the
 *    validation mode described below.
 *  * Layouts are row-major and token-major, packed without padding:
 *        K, V     [T, H, d]        bf16 (SA_BF16) or fp32 (SA_FP32)
 *        P        [H, M, d]        same dtype as K and V
 *        offsets  [B + 1]          int64 CSR offsets: offsets[0] = 0,
 *                                  non-decreasing, offsets[B] = T; user b owns
 *                                  tokens offsets[b] .. offsets[b+1]-1
 *        sketch   [B, H, M, d]     fp32
 *        lse      [T, H]           fp32
 *        dsketch  [B, R, H, M, d]  fp32
 *        dK, dV   [T, H, d]        fp32
 *        dP       [H, M, d]        fp32
 *    Base addresses must be 16-byte aligned.
 *  * Errors are returned as sa_status codes; nothing is thrown across the ABI.
 *    Argument checks happen on the host before anything is enqueued.  Offsets
 *    live on the device and are not read by the host: malformed offsets give
 *    unspecified values but never an out-of-bounds access.  With the
 *    environment variable SA_DEBUG_VALIDATE=1 the library copies the offsets to
 *    the host (synchronising `stream`) and returns SA_ERR_BAD_OFFSETS for
 *    malformed ones.
 *  * Calls on different streams with disjoint outputs and workspaces may run
 *    concurrently; the library holds no mutable global state besides
 *    per-device constants (CU count) read once.
 *  * Results are deterministic: the same inputs, shapes and device give
 *    bit-identical outputs (fixed reduction orders, no floating-point atomics).
 */
#ifndef SA_SKETCH_H
#define SA_SKETCH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SA_OK = 0,
    SA_ERR_INVALID_ARG = 1, /* null pointer, negative size, misaligned pointer, bad scale */
    SA_ERR_UNSUPPORTED = 2, /* a shape or dtype this build does not handle */
    SA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than *_workspace_size() */
    SA_ERR_BAD_OFFSETS = 4, /* only with SA_DEBUG_VALIDATE=1 */
    SA_ERR_HIP = 5          /* a HIP runtime or launch error */
} sa_status;

typedef enum {
    SA_BF16 = 0, /* K, V, P in bfloat16; logits and accumulation in fp32 */
    SA_FP32 = 1  /* K, V, P in fp32; no sub-fp32 rounding anywhere */
} sa_dtype;

/*
 * Supported shapes (SA_ERR_UNSUPPORTED otherwise): 1 <= H, 1 <= M <= 4096,
 * d in {64, 128}, T < 2^31, B >= 0.  bf16 with d = 64 and M a multiple of 128
 * up to 1024, or d = 128 and M a multiple of 128 up to 512, runs the fused
 * matrix-core kernels; other supported shapes and SA_FP32 run a plain fp32
 * path with the same ABI and the same results up to rounding.
 */

/* Bytes of workspace that sa_sketch_fwd needs for this shape (0 is possible). */
size_t sa_sketch_fwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M,
                                    int32_t d, sa_dtype dtype);

/*
 * Forward: sketch (and optionally lse) of every user.
 *
 * Section 3.1 (S, A, sketch) and section 4.4 (streaming evaluation that keeps
 * the per-token softmax statistics instead of the scores).
 *
 *   K, V, P, offsets  inputs as above
 *   B, T, H, M, d     sizes; B = 0 is a no-op returning SA_OK
 *   scale             logit scale, normally 1/sqrt(d); finite and >= 0
 *   dtype             SA_BF16 or SA_FP32 (K, V and P share it)
 *   sketch            output [B,H,M,d] fp32, fully overwritten (zeros for an
 *                     empty user)
 *   lse               output [T,H] fp32 log-sum-exp of each token's scaled
 *                     logits over the M prototypes, or NULL if not wanted
 *                     (sa_sketch_bwd needs it)
 *   workspace         device scratch of at least workspace_bytes; may be NULL
 *                     when the size query returned 0
 */
sa_status sa_sketch_fwd(const void* K, const void* V, const void* P,
                        const int64_t* offsets, int64_t B, int64_t T, int32_t H,
                        int32_t M, int32_t d, float scale, sa_dtype dtype,
                        float* sketch, float* lse, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * sa_sketch_fwd without a workspace argument and without any allocation, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Same operation,
 * arguments, kernels, results (bit for bit) and errors as sa_sketch_fwd, with
 * these differences:
 *  * the work list, the per-range partial sketches and (plain path, lse = NULL)
 *    the lse scratch live in a device array of SA_NOALLOC_SCRATCH_BYTES that the
 *    library holds on every device it runs on until the process ends (looked up
 *    once per device, on the first call with that device current);
 *  * a shape whose scratch exceeds that size returns SA_ERR_WORKSPACE (the
 *    ragged 100K batch at H = 4, d = 128, M = 512 needs about 100 MB and fits);
 *  * every call on one device shares that device's array: calls that overlap
 *    in time on one device (other streams, other host threads) race and give
 *    wrong results.  Calls on one stream are ordered and safe.  Nothing in the
 *    array needs to start at zero (every kernel writes what it later reads);
 *  * it records no per-launch timing (sa_profile_enable) and ignores
 *    SA_DEBUG_VALIDATE (which would synchronise the stream).
 */
#define SA_NOALLOC_SCRATCH_BYTES (128u << 20)
sa_status sa_sketch_fwd_noalloc(const void* K, const void* V, const void* P, const int64_t* offsets,
                                int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                                sa_dtype dtype, float* sketch, float* lse, void* stream);

/* Bytes of workspace that sa_sketch_fwd_tokenwise needs for this shape. */
size_t sa_sketch_fwd_tokenwise_workspace_size(int64_t B, int64_t T, int32_t H,
                                              int32_t M, int32_t d, sa_dtype dtype);

/*
 * Forward of the token-wise normalised variant: the normalisation the paper
 * compares SA's prototype-wise one with (appendix on prototype-wise
 * normalisation; Table 1 baseline).  For each user b, head h and prototype m
 * the weights are normalised over the user's tokens:
 *
 *   s_t            = scale * K[t,h] . P[h,m]           t over the user's tokens
 *   sketch[b,h,m]  = sum_t exp(s_t) V[t,h] / sum_t exp(s_t)
 *   lse_m[b,h,m]   = log sum_t exp(s_t)                  (-inf for an empty user)
 *
 * i.e. attention with the prototypes as queries over each user's tokens.
 * Arguments, layouts, supported shapes and error behaviour are those of
 * sa_sketch_fwd except:
 *   lse_m     output [B,H,M] fp32 per-prototype log-sum-exp, or NULL
 * An empty user gets a zero sketch (and lse_m = -inf).  bf16 with d in {64,128}
 * and M a multiple of 128 runs the matrix-core kernel (online softmax over token
 * tiles, users cut across ranges merged by log-sum-exp); other shapes and
 * SA_FP32 run a plain fp32 path.
 */
sa_status sa_sketch_fwd_tokenwise(const void* K, const void* V, const void* P,
                                  const int64_t* offsets, int64_t B, int64_t T,
                                  int32_t H, int32_t M, int32_t d, float scale,
                                  sa_dtype dtype, float* sketch, float* lse_m,
                                  void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Bytes of workspace that sa_sketch_bwd needs for this shape. */
size_t sa_sketch_bwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M,
                                    int32_t d, sa_dtype dtype, int32_t R);

/*
 * Backward of the forward above (the paper trains the sketch end to end,
 * section 3.1; the gradients follow by the chain rule):
 *
 *   dY[b,h]  = sum_{r<R} dsketch[b,r,h]   one user's sketch reused by R target
 *                                         instances receives the sum of their
 *                                         gradients (section 4.2, MRLB)
 *   dV[t,h]  = sum_m A[t,m] dY[b,h,m,:]
 *   dS[t,m]  = A[t,m] (<V[t,h],dY[b,h,m]> - sum_m' A[t,m'] <V[t,h],dY[b,h,m']>)
 *   dK[t,h]  = scale * sum_m dS[t,m] P[h,m,:]
 *   dP[h,m]  = scale * sum over every user and token of dS[t,m] K[t,h,:]
 *
 *   lse       the lse written by sa_sketch_fwd for the same inputs (required)
 *   dsketch   [B,R,H,M,d] fp32, R >= 1 target instances per user
 *   dK, dV    outputs [T,H,d] fp32, overwritten (tokens outside every user get 0)
 *   dP        output [H,M,d] fp32, overwritten (not accumulated into)
 */
sa_status sa_sketch_bwd(const void* K, const void* V, const void* P,
                        const int64_t* offsets, int64_t B, int64_t T, int32_t H,
                        int32_t M, int32_t d, float scale, sa_dtype dtype,
                        const float* dsketch, int32_t R, const float* lse,
                        float* dK, float* dV, float* dP, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Bytes of workspace that sa_layer_fwd needs for this shape. */
size_t sa_layer_fwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M,
                                   int32_t d, sa_dtype dtype);

/*
 * Forward of one SA layer with its projections (Appendix G.3; section 3.1):
 *
 *   Q = P W_Q,  K = X W_K,  S = scale Q K^T,  A = softmax over prototypes,
 *   sketch = A X      (the history X itself is aggregated, as in section 3.1)
 *
 * per user and per head (heads are independent SA instances with their own
 * P[h], W_Q[h], W_K[h]; H = 1 is the paper's single-head SA).  The key
 * projection is folded into the prototypes, S = scale (P W_Q W_K^T) X^T (the
 * reordering the paper uses for single-query STCA, Appendix G.2): no key tensor
 * is formed and X is read once.  In bf16 mode P' = P W_Q W_K^T is computed with
 * fp32 accumulation and rounded once to bf16.
 *
 *   X         [T,H,d] history, dtype
 *   P         [H,M,d] prototypes P^(0), dtype
 *   Wq, Wk    [H,d,d] row-major, K[t,h,j] = sum_i X[t,h,i] Wk[h,i,j]; dtype
 *   sketch    output [B,H,M,d] fp32; lse output [T,H] fp32 or NULL (as sa_sketch_fwd)
 *
 * Offsets, sizes, supported shapes, errors, ownership and streams are those of
 * sa_sketch_fwd; the workspace is required (at least the per-head products).
 */
sa_status sa_layer_fwd(const void* X, const void* P, const void* Wq, const void* Wk,
                       const int64_t* offsets, int64_t B, int64_t T, int32_t H, int32_t M,
                       int32_t d, float scale, sa_dtype dtype, float* sketch, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace that sa_layer_bwd needs for this shape. */
size_t sa_layer_bwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M,
                                   int32_t d, sa_dtype dtype, int32_t R);

/*
 * Backward of sa_layer_fwd, by the chain rule (dY = sum over the R target
 * instances, section 4.2):
 *
 *   dX  = A^T dY + dK W_K^T         (X is both the value and the key input)
 *   dW_K = sum over users of X^T dK,  dK = scale dS^T Q
 *   dQ  = scale sum over users of dS K,  dW_Q = P^T dQ,  dP = dQ W_Q^T
 *
 * with dS the prototype-softmax gradient of sa_sketch_bwd.  Computed as the
 * sketching backward with K = V = X and prototypes P' = Q W_K^T, which yields
 * dX = dV + scale dS P' per token and dP', followed by dW_K = dP'^T Q,
 * dQ = dP' W_K, dW_Q = P^T dQ and dP = dQ W_Q^T per head.
 *
 *   lse             the lse written by sa_layer_fwd for the same inputs (required)
 *   dsketch         [B,R,H,M,d] fp32
 *   dX              output [T,H,d] fp32, overwritten
 *   dP              output [H,M,d] fp32; dWq, dWk outputs [H,d,d] fp32; overwritten
 */
sa_status sa_layer_bwd(const void* X, const void* P, const void* Wq, const void* Wk,
                       const int64_t* offsets, int64_t B, int64_t T, int32_t H, int32_t M,
                       int32_t d, float scale, sa_dtype dtype, const float* dsketch, int32_t R,
                       const float* lse, float* dX, float* dP, float* dWq, float* dWk,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace that sa_block_fwd needs for this shape. */
size_t sa_block_fwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   int32_t n_layers, sa_dtype dtype);

/*
 * Forward of stacked SA (section 3.3, stacked refinement) with n_layers layers.
 * Per user and head, starting from the shared prototypes Xt = P:
 *
 *   Xhat = sketch of X with queries Xt W_Q and keys X W_K   (as sa_layer_fwd; per
 *          user prototypes from the second layer on)
 *   Xbar = LN1(Xt + Xhat)
 *   Xt   = LN2(Xbar + FFN(Xbar)),   FFN(x) = (silu(x W1) * (x W3)) W2
 *
 * with LN(x) = (x - mean) / sqrt(var + eps) * gamma + beta over the d features
 * (biased variance) and a SwiGLU FFN of intermediate width 2d without biases.
 *
 *   X         [T,H,d] history; P [H,M,d] prototypes (dtype)
 *   Wq, Wk    [n_layers,H,d,d]; W1, W3 [n_layers,H,d,2d]; W2 [n_layers,H,2d,d] (dtype)
 *   ln        [n_layers,4,H,d]: gamma1, beta1, gamma2, beta2 (dtype)
 *   eps       layer-norm epsilon (> 0)
 *   out       output [B,H,M,d] fp32: the refined sketch
 *   lse       output [n_layers,T,H] fp32 (each layer's per-token log-sum-exp), or NULL
 *   saved     NULL (inference), or a device buffer of sa_block_saved_size bytes,
 *             16-byte aligned (training): every layer's intermediates are written
 *             there for sa_block_bwd, which then skips its replay of the forward.
 *             Its layout is private to the library; the caller owns it and keeps
 *             it unchanged between the two calls.
 *
 * A user without tokens has a zero Xhat in every layer, so its output is the
 * refinement of the prototypes alone.  The sketching steps run on the same
 * kernels as sa_layer_fwd; the projections and the FFN on a batched fp32
 * product.  Offsets, sizes, errors, ownership and streams as for sa_sketch_fwd;
 * n_layers < 1 or a non-positive eps is SA_ERR_INVALID_ARG, a saved buffer too
 * small or misaligned SA_ERR_WORKSPACE.
 */
sa_status sa_block_fwd(const void* X, const void* P, const void* Wq, const void* Wk, const void* ln,
                       const void* W1, const void* W3, const void* W2, const int64_t* offsets,
                       int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers,
                       float scale, float eps, sa_dtype dtype, float* out, float* lse,
                       void* saved, size_t saved_bytes, void* workspace, size_t workspace_bytes,
                       void* stream);

/* Bytes of the buffer of saved intermediates (sa_block_fwd's `saved`) for this
 * shape: per layer about (36 + 2 or 4 bytes per element of the dtype) B H M d
 * bytes plus 4 T H; 0 for invalid sizes. */
size_t sa_block_saved_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers,
                           sa_dtype dtype);

/* Intermediates that a training forward keeps in `saved`, for inspection by
 * the caller (the backward reads them itself).  Layer l's block of `saved`
 * holds, each at its own offset:
 *   SA_SAVED_STATE  [B,H,M,d] fp32   the layer's query state Xt (l >= 1 only;
 *                                    the first layer's state is P itself)
 *   SA_SAVED_Q      [B,H,M,d] fp32   Q = Xt W_Q  ([H,M,d] used for l = 0)
 *   SA_SAVED_PP     [B,H,M,d] dtype  P' = Q W_K^T as the sketch's prototypes
 *                                    (bf16: rounded once from fp32; [H,M,d] used
 *                                    for l = 0)
 *   SA_SAVED_LSE    [T,H] fp32       the layer's per-token log-sum-exp
 */
typedef enum { SA_SAVED_STATE = 0, SA_SAVED_Q = 1, SA_SAVED_PP = 2, SA_SAVED_LSE = 3 } sa_saved_item;

/* Byte offset of intermediate `item` of layer `layer` inside a `saved` buffer
 * of this shape (sa_block_saved_size bytes for n_layers layers); (size_t)-1 for
 * invalid sizes, a layer outside [0, n_layers), an unknown item, or the state of
 * layer 0. */
size_t sa_block_saved_offset(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers,
                             sa_dtype dtype, int32_t layer, int32_t item);

/* Bytes of workspace that sa_block_bwd needs for this shape; with_saved != 0
 * when it will be given a saved buffer (then the replay's region is left out). */
size_t sa_block_bwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   int32_t n_layers, sa_dtype dtype, int32_t with_saved);

/*
 * Backward of sa_block_fwd (section 3.3) by the chain rule: the gradients of
 * <dout, out> with respect to every input.  Each layer's intermediates come
 * from `saved` when the training forward wrote them there (same inputs, not
 * changed since); with saved = NULL the forward is replayed first, keeping them
 * in the workspace.  Both give bit-identical gradients.  Then, from the last
 * layer down: the second norm, the FFN (dW2 = Z^T dY2, the gate
 * silu'(g) = s (1 + g (1 - s)), dW1 = Xbar^T dG, dW3 = Xbar^T dU), the first
 * norm, the sketch (the sketching backward with dsketch = the gradient of Xhat,
 * one target instance, per-user prototypes from the second layer on) and the two
 * projections.  The first layer's state gradient is the prototypes' gradient,
 * summed over users; weight gradients are summed over users in user order.
 *
 *   dout      [B,H,M,d] fp32, the gradient of out
 *   dX        output [T,H,d] fp32;  dP output [H,M,d] fp32
 *   dWq, dWk  outputs [n_layers,H,d,d];  dW1, dW3 [n_layers,H,d,2d];  dW2 [n_layers,H,2d,d]
 *   dln       output [n_layers,4,H,d] (gamma1, beta1, gamma2, beta2)
 *
 * All outputs fp32 and overwritten.  Results are deterministic (fixed
 * summation orders).  Other arguments, errors, ownership and streams as for
 * sa_block_fwd; B = 0 is SA_ERR_INVALID_ARG here (no gradients to write) and
 * more than 65535 users SA_ERR_UNSUPPORTED.
 */
sa_status sa_block_bwd(const void* X, const void* P, const void* Wq, const void* Wk, const void* ln,
                       const void* W1, const void* W3, const void* W2, const int64_t* offsets,
                       int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers,
                       float scale, float eps, sa_dtype dtype, const float* dout, float* dX,
                       float* dP, float* dWq, float* dWk, float* dln, float* dW1, float* dW3,
                       float* dW2, const void* saved, size_t saved_bytes, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Bytes of workspace that sa_stca_fwd needs for this shape. */
size_t sa_stca_fwd_workspace_size(int64_t B, int32_t R, int32_t k, int32_t D, int32_t h,
                                  sa_dtype dtype);

/*
 * Single-query target-to-history cross attention over the adapted sketch, in
 * the reordered form of Appendix G.2 (STCA of section 2.1, applied over the
 * sketch in section 3.4).  Each of the B users has a sketch Xs [k, D] and R
 * targets (its MRLB group, section 4.2), each with one query q [D].  Per
 * target and head i (h heads of width d_h = D / h; W^(i) = columns
 * i*d_h .. (i+1)*d_h - 1 of W_Q, W_K, W_V):
 *
 *   u     = (q W_Q^(i)) W_K^(i)T
 *   alpha = softmax over the k sketch rows of scale * u Xs^T
 *   o^(i) = (alpha Xs) W_V^(i)
 *
 * which equals softmax(scale (q W_Q^(i))(Xs W_K^(i))^T)(Xs W_V^(i)) without the
 * length-k projections.  The output projection and the FFNs of a full STCA
 * layer are separate products.
 *
 *   Xs          [B,k,D] adapted sketches (dtype)
 *   q           [B,R,D] target queries (dtype)
 *   Wq, Wk, Wv  [D,D] (dtype), row = input feature
 *   scale       normally 1/sqrt(D/h), finite and > 0
 *   out         output [B,R,D] fp32: the heads' o^(i) side by side
 *   lse         output [B,R,h] fp32 log-sum-exp of the scaled logits, or NULL
 *
 * bf16 mode runs the products on the matrix cores with bf16 intermediates
 * (queries, logits' softmax weights, aggregates) and fp32 accumulation; fp32
 * mode keeps every value in fp32.  D must be a multiple of h; B = 0 is a no-op.
 * Errors, ownership and streams as for sa_sketch_fwd.
 */
sa_status sa_stca_fwd(const void* Xs, const void* q, const void* Wq, const void* Wk, const void* Wv,
                      int64_t B, int32_t R, int32_t k, int32_t D, int32_t h, float scale,
                      sa_dtype dtype, float* out, float* lse, void* workspace,
                      size_t workspace_bytes, void* stream);

/* Bytes of workspace that sa_stca_bwd needs for this shape. */
size_t sa_stca_bwd_workspace_size(int64_t B, int32_t R, int32_t k, int32_t D, int32_t h,
                                  sa_dtype dtype);

/*
 * Backward of sa_stca_fwd by the chain rule: gradients of <dout, out>.  The
 * forward is replayed in the workspace; then, with c = alpha Xs:
 * dc = do^(i) W_V^(i)T and dW_V^(i) = sum c^T do^(i); dalpha = dc Xs^T;
 * ds = scale alpha (dalpha - <alpha, dalpha>); dXs = sum alpha^T dc + ds^T u;
 * du = ds Xs; with p = q W_Q^(i): dp = du W_K^(i), dW_K^(i) = sum du^T p,
 * dq = dp W_Q^T (summed over heads), dW_Q = sum q^T dp.  Sums run over every
 * user and target.
 *
 *   dout                    [B,R,D] fp32
 *   dXs                     output [B,k,D] fp32
 *   dq                      output [B,R,D] fp32
 *   dWq, dWk, dWv           outputs [D,D] fp32
 *
 * All outputs are overwritten.  B = 0 is SA_ERR_INVALID_ARG (nothing to write);
 * other arguments as for sa_stca_fwd.
 */
sa_status sa_stca_bwd(const void* Xs, const void* q, const void* Wq, const void* Wk, const void* Wv,
                      int64_t B, int32_t R, int32_t k, int32_t D, int32_t h, float scale,
                      sa_dtype dtype, const float* dout, float* dXs, float* dq, float* dWq,
                      float* dWk, float* dWv, void* workspace, size_t workspace_bytes,
                      void* stream);

/*
 * Work list used by the fused forward, exposed for exact testing.
 *
 * The (head, token) pairs are laid out head-major in one index space of
 * length H*T, cut into n_ranges = ceil(H*T / chunk_tokens) equal ranges (one
 * per workgroup).  Each (user, head) pair with at least one token is cut at
 * the range boundaries into segments; segments are listed in (head, user,
 * range) order.  Every token of every user is covered exactly once.
 *
 * Each item is 8 int32: {b, h, t0, t1, range, split, pair_first, 0}, where
 * [t0, t1) are token indices, `range` is the workgroup range that processes
 * the segment, split = 1 when the user's tokens span more than one range (its
 * partial sketches are summed by the split-L merge), and pair_first is the
 * index of the first segment of the same (user, head) pair.
 *
 *   offsets        device int64 [B+1]
 *   chunk_tokens   range length, > 0
 *   items          device int32 [max_items * 8]
 *   max_items      capacity; at most ceil(H*T/chunk_tokens) + H*B items are produced
 *   n_items        device int64 [1]: number of items written
 */
sa_status sa_build_worklist(const int64_t* offsets, int64_t B, int64_t T,
                            int32_t H, int64_t chunk_tokens, int32_t* items,
                            int64_t max_items, int64_t* n_items, void* stream);

/* Tokens per workgroup range that sa_sketch_fwd uses for this shape. */
int64_t sa_sketch_fwd_chunk_tokens(int64_t B, int64_t T, int32_t H, int32_t M,
                                   int32_t d, sa_dtype dtype);

/*
 * The library's batched product on the matrix cores, for tests of each of its
 * tile shapes (the STCA step and the layer and block gradients run on it):
 *
 *   C[z](m, n) = alpha sum_k A[z](m, k) B[z](k, n)  (+ C[z](m, n) when accumulate)
 *
 * with A[z](m, k) = A[z a_z + m a_m + k a_k] and B[z](k, n) = B[(z mod b_mod, or
 * z when b_mod = 0) b_z + k b_k + n b_n] bf16 (device pointers, strides in
 * elements), C[z](m, n) = C[z c_z + m c_m + n] fp32 (c_bf16 = 0) or bf16, fp32
 * accumulation.  A is contiguous along k (a_k = 1) or along m (a_m = 1), B along k
 * (b_k = 1) or along n (b_n = 1).  tile_shape < 0 lets the library pick the
 * shape (as it does for its own products, including the register-tiled fp32
 * product when the matrix cores cannot take it); 0 .. sa_gemm_tile_shapes() - 1
 * forces one shape and returns SA_ERR_UNSUPPORTED where that shape cannot take
 * the product (K not a multiple of 64, strides or bases not on 16 bytes, an
 * m-contiguous A on the 160-row shape, byte offsets beyond 32 bits).  Operands
 * and result are the caller's; asynchronous on `stream`.
 */
int32_t sa_gemm_tile_shapes(void);
sa_status sa_gemm_bf16(const void* A, int64_t a_z, int64_t a_m, int64_t a_k, const void* B, int64_t b_z,
                       int64_t b_k, int64_t b_n, int64_t b_mod, void* C, int32_t c_bf16, int64_t c_z, int64_t c_m,
                       int32_t M, int32_t N, int32_t K, int32_t batch, float alpha, int32_t accumulate,
                       int32_t tile_shape, void* stream);

/*
 * Kernel timing for benchmarks.  While enabled (on = 1) on the calling thread,
 * every kernel the library launches from that thread is bracketed by two HIP
 * events recorded on the launch stream.  sa_kernel_times() waits for those
 * events and returns, for up to max_kernels distinct kernels, the name (NUL
 * terminated, at most 47 characters, in names[i*48]), the number of launches
 * and the total device time in milliseconds since the previous collection, then
 * clears the record.  Returns the number of kernels written, or -1 on a HIP
 * error.  Disabled by default; costs two event records per launch when on.
 */
void sa_profile_enable(int32_t on);
int32_t sa_kernel_times(int32_t max_kernels, char* names, int64_t* launches, double* total_ms);

/* Static text of a status code. */
const char* sa_status_string(sa_status status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* sa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SA_SKETCH_H */

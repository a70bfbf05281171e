// Host side of the C ABI declared in include/sa_sketch.h: argument checks,
// launch plans, workspace carving and kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "sa_internal.h"

namespace {

thread_local char g_last_error[512] = "";

sa_status fail(sa_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}

sa_status hip_fail(hipError_t e, const char* what) {
    return fail(SA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

using sa::device_cus;
constexpr int kMaxDevices = 64;

// ---------------------------------------------------------------- kernel timing
struct ProfRec {
    const char* name;
    hipEvent_t start, stop;
};
thread_local bool g_prof_on = false;
thread_local std::vector<ProfRec> g_prof_recs;
thread_local std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
    if (!g_prof_pool.empty()) {
        hipEvent_t e = g_prof_pool.back();
        g_prof_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

bool debug_validate() {
    const char* v = getenv("SA_DEBUG_VALIDATE");
    return v && v[0] && strcmp(v, "0") != 0;
}

sa_status check_common(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                       sa_dtype dtype) {
    if (B < 0 || T < 0 || H < 1 || M < 1 || d < 1)
        return fail(SA_ERR_INVALID_ARG, "bad sizes B=%lld T=%lld H=%d M=%d d=%d", (long long)B,
                    (long long)T, H, M, d);
    if (!(std::isfinite(scale) && scale >= 0.f))
        return fail(SA_ERR_INVALID_ARG, "scale must be finite and >= 0 (got %g)", (double)scale);
    if (dtype != SA_BF16 && dtype != SA_FP32)
        return fail(SA_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
    if (d != 64 && d != 128) return fail(SA_ERR_UNSUPPORTED, "d must be 64 or 128 (got %d)", d);
    if (M > 4096) return fail(SA_ERR_UNSUPPORTED, "M must be <= 4096 (got %d)", M);
    if (T >= (int64_t(1) << 31)) return fail(SA_ERR_UNSUPPORTED, "T must be < 2^31");
    if ((int64_t)H * B >= (int64_t(1) << 31))
        return fail(SA_ERR_UNSUPPORTED, "H*B must be < 2^31");
    return SA_OK;
}

sa_status validate_offsets(const int64_t* offsets, int64_t B, int64_t T, hipStream_t stream) {
    std::vector<int64_t> h((size_t)B + 1);
    hipError_t e = hipMemcpyAsync(h.data(), offsets, sizeof(int64_t) * (B + 1),
                                  hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "copying offsets for validation");
    if (h[0] != 0) return fail(SA_ERR_BAD_OFFSETS, "offsets[0] = %lld, expected 0", (long long)h[0]);
    for (int64_t b = 0; b < B; ++b)
        if (h[b + 1] < h[b])
            return fail(SA_ERR_BAD_OFFSETS, "offsets decrease at user %lld", (long long)b);
    if (h[B] != T)
        return fail(SA_ERR_BAD_OFFSETS, "offsets[B] = %lld, expected T = %lld", (long long)h[B],
                    (long long)T);
    return SA_OK;
}

// ---------------------------------------------------------------- forward plan
struct FwdPlan {
    bool fused = false;
    int64_t C = 0;         // tokens per workgroup range
    int64_t n_ranges = 0;  // workgroups
    int64_t max_items = 0;
    // workspace offsets (bytes)
    size_t off_nitems = 0, off_wgstart = 0, off_pairstart = 0, off_items = 0, off_partials = 0,
           off_lse = 0, total = 0;
};

int64_t fused_chunk_tokens(int64_t T, int32_t H, int32_t M, int32_t d) {
    int per_cu = 1;
    if (sa::fused_fwd_occupancy(M, d, &per_cu) != hipSuccess || per_cu < 1) per_cu = 1;
    const int64_t target = (int64_t)device_cus() * per_cu;
    const int64_t HT = (int64_t)H * T;
    int64_t C = (HT + target - 1) / target;
    C = (C + sa::kTileTokens - 1) / sa::kTileTokens * sa::kTileTokens;
    if (C < sa::kTileTokens) C = sa::kTileTokens;
    return C;
}

FwdPlan plan_fwd(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, sa_dtype dtype,
                 bool need_lse_scratch) {
    FwdPlan p;
    p.fused = dtype == SA_BF16 && sa::fused_fwd_supported(M, d);
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    // both paths cut the head-major token space into equal ranges (a work list
    // of (user, head) segments, split pairs merged in segment order): the fused
    // kernel runs one range per workgroup slot, the plain aggregation one range
    // per 64 prototypes and about four workgroups per CU
    const int64_t HT = (int64_t)H * T;
    if (p.fused) {
        p.C = fused_chunk_tokens(T, H, M, d);
    } else {
        const int64_t target = 4 * (int64_t)device_cus();
        int64_t C = (HT + target - 1) / target;
        C = (C + sa::kTileTokens - 1) / sa::kTileTokens * sa::kTileTokens;
        p.C = C < sa::kTileTokens ? sa::kTileTokens : C;
    }
    p.n_ranges = (HT + p.C - 1) / p.C;
    p.max_items = p.n_ranges + (int64_t)H * B;
    p.off_nitems = carve(sizeof(int64_t));
    p.off_wgstart = carve(sizeof(int32_t) * (p.n_ranges + 1));
    p.off_pairstart = carve(sizeof(int32_t) * ((int64_t)H * B + 1));
    p.off_items = carve(sizeof(int32_t) * sa::IT_WORDS * p.max_items);
    p.off_partials = carve(sizeof(float) * (size_t)p.max_items * M * d);
    if (!p.fused && need_lse_scratch) p.off_lse = carve(sizeof(float) * (size_t)T * H);
    p.total = off;
    return p;
}

// ---------------------------------------------------------------- token-wise plan
struct TwPlan {
    bool fused = false;
    int64_t C = 0, n_ranges = 0, max_items = 0;
    size_t off_nitems = 0, off_wgstart = 0, off_pairstart = 0, off_items = 0, off_partials = 0,
           off_stats = 0, total = 0;
};

TwPlan plan_tokenwise(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, sa_dtype dtype) {
    TwPlan p;
    p.fused = dtype == SA_BF16 && sa::tokenwise_fused_supported(M, d);
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    if (p.fused) {
        // one range per CU; each range runs M / (prototypes per workgroup) workgroups
        const int64_t HT = (int64_t)H * T;
        const int64_t target = device_cus();
        int64_t C = (HT + target - 1) / target;
        C = (C + sa::kTileTokens - 1) / sa::kTileTokens * sa::kTileTokens;
        if (C < sa::kTileTokens) C = sa::kTileTokens;
        p.C = C;
        p.n_ranges = (HT + C - 1) / C;
        p.max_items = p.n_ranges + (int64_t)H * B;
        p.off_nitems = carve(sizeof(int64_t));
        p.off_wgstart = carve(sizeof(int32_t) * (p.n_ranges + 1));
        p.off_pairstart = carve(sizeof(int32_t) * ((int64_t)H * B + 1));
        p.off_items = carve(sizeof(int32_t) * sa::IT_WORDS * p.max_items);
        p.off_partials = carve(sizeof(float) * (size_t)p.max_items * M * d);
        p.off_stats = carve(sizeof(float) * (size_t)p.max_items * M * 2);
    }
    p.total = off;
    return p;
}

// ---------------------------------------------------------------- backward plan
struct BwdPlan {
    bool fused = false;
    int32_t n_chunks = 1;
    int64_t C = 0, n_ranges = 0, max_items = 0;
    size_t off_dY = 0, off_D = 0, off_part = 0;
    size_t off_nitems = 0, off_wgstart = 0, off_pairstart = 0, off_items = 0, off_ymj = 0,
           off_yjm = 0, off_pjm = 0, total = 0;
};

BwdPlan plan_bwd(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, sa_dtype dtype,
                 bool p_user = false) {
    BwdPlan p;
    p.fused = dtype == SA_BF16 && sa::fused_bwd_supported(M, d);
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    if (p.fused) {
        // token-side workgroup ranges: as many as fit on the CUs at once; the dP
        // kernel runs M / part workgroups per range
        const int64_t HT = (int64_t)H * T;
        const int64_t target = (int64_t)device_cus() * sa::fused_bwd_ranges_per_cu();
        int64_t C = (HT + target - 1) / target;
        C = (C + 127) / 128 * 128;
        if (C < 128) C = 128;
        p.C = C;
        p.n_ranges = (HT + C - 1) / C;
        p.max_items = p.n_ranges + (int64_t)H * B;
        p.off_nitems = carve(sizeof(int64_t));
        p.off_wgstart = carve(sizeof(int32_t) * (p.n_ranges + 1));
        p.off_pairstart = carve(sizeof(int32_t) * ((int64_t)H * B + 1));
        p.off_items = carve(sizeof(int32_t) * sa::IT_WORDS * p.max_items);
        p.off_ymj = carve(sizeof(uint16_t) * (size_t)B * H * M * d);
        p.off_yjm = carve(sizeof(uint16_t) * (size_t)B * H * M * d);
        p.off_pjm = carve(sizeof(uint16_t) * (size_t)(p_user ? B * H : H) * M * d);
        p.off_D = carve(sizeof(float) * (size_t)T * H);
        p.off_part = carve(sizeof(float) * (size_t)p.max_items * M * d);
    } else {
        p.n_chunks = sa::generic_dp_chunks(T, H, M);
        p.off_dY = carve(sizeof(float) * (size_t)B * H * M * d);
        p.off_D = carve(sizeof(float) * (size_t)T * H);
        p.off_part = carve(sizeof(float) * (size_t)p.n_chunks * H * M * d);
    }
    p.total = off;
    return p;
}

// ---------------------------------------------------------------- SA layer plan
// [Q fp32 | P' = Q W_K^T in the input dtype | (bwd) dP' fp32 | dQ fp32 |
//  (bwd, plain path) dK, dV fp32 | workspace of the sketching call]
struct LayerPlan {
    size_t off_q = 0, off_pp = 0, off_dpp = 0, off_dq = 0, off_dk = 0, off_dv = 0, off_base = 0;
    size_t total = 0;
};

LayerPlan plan_layer(int64_t T, int32_t H, int32_t M, int32_t d, sa_dtype dtype, bool bwd,
                     bool plain_bwd, size_t base_bytes) {
    LayerPlan p;
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t hmd = (size_t)H * M * d;
    p.off_q = carve(sizeof(float) * hmd);
    p.off_pp = carve((dtype == SA_BF16 ? 2 : 4) * hmd);
    if (bwd) {
        p.off_dpp = carve(sizeof(float) * hmd);
        p.off_dq = carve(sizeof(float) * hmd);
        if (plain_bwd) {
            p.off_dk = carve(sizeof(float) * (size_t)T * H * d);
            p.off_dv = carve(sizeof(float) * (size_t)T * H * d);
        }
    }
    p.off_base = carve(base_bytes);
    p.total = off;
    return p;
}

// Q = P W_Q (fp32) and P' = Q W_K^T (input dtype), per head
sa_status layer_prototypes(const void* P, const void* Wq, const void* Wk, int32_t H, int32_t M,
                           int32_t d, sa_dtype dtype, float* Q, void* Pp, hipStream_t stream) {
    const bool bf = dtype == SA_BF16;
    const int64_t md = (int64_t)M * d, dd = (int64_t)d * d;
    sa::ProfScope ps("layer_proto_proj", stream);
    hipError_t e = sa::launch_small_gemm({P, bf, md, d, 1}, {Wq, bf, dd, d, 1}, Q, false, H, M, d, d,
                                         stream);
    if (e == hipSuccess)
        e = sa::launch_small_gemm({Q, false, md, d, 1}, {Wk, bf, dd, 1, d}, Pp, bf, H, M, d, d, stream);
    if (e != hipSuccess) return hip_fail(e, "prototype projection launch");
    return SA_OK;
}

// ---------------------------------------------------------------- stacked block plan
// [state | Q | P' (input dtype) | Xhat (also the FFN output) | Xbar | gate | up |
//  lse scratch | workspace of the sketching call]; state, Q, P', Xhat, Xbar are
// [B,H,M,d] fp32 (P' in the input dtype), gate and up [B,H,M,2d] fp32.
struct BlockPlan {
    FwdPlan base;
    size_t off_state = 0, off_q = 0, off_pp = 0, off_xhat = 0, off_xbar = 0, off_g = 0, off_u = 0, off_lse = 0,
           off_base = 0, total = 0;
};

BlockPlan plan_block(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, sa_dtype dtype) {
    BlockPlan p;
    p.base = plan_fwd(B, T, H, M, d, dtype, false);
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t rows = (size_t)B * H * M;
    p.off_state = carve(sizeof(float) * rows * d);
    p.off_q = carve(sizeof(float) * rows * d);
    p.off_pp = carve((dtype == SA_BF16 ? 2 : 4) * rows * d);
    p.off_xhat = carve(sizeof(float) * rows * d);
    p.off_xbar = carve(sizeof(float) * rows * d);
    p.off_g = carve(sizeof(float) * rows * 2 * d);
    p.off_u = carve(sizeof(float) * rows * 2 * d);
    p.off_lse = carve(sizeof(float) * (size_t)T * H);
    p.off_base = carve(p.base.total);
    p.total = off;
    return p;
}

// ---------------------------------------------------------------- stacked block: saved intermediates
// Per layer l a region [state_l (l >= 1) | Q_l | P'_l | lse_l | Y1_l | Xbar_l | G_l | U_l | Y2_l]
// holding the forward's intermediates (Y1 = Xt + Xhat, Y2 = Xbar + FFN: the
// inputs of the two norms).  The training forward writes them to the caller's
// `saved` buffer; without one, the backward replays the forward into its workspace.
struct BlockSaved {
    size_t l_state = 0, l_q = 0, l_pp = 0, l_lse = 0, l_y1 = 0, l_xbar = 0, l_g = 0, l_u = 0, l_y2 = 0,
           l_stride = 0;
};

BlockSaved saved_layout(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, sa_dtype dtype) {
    BlockSaved p;
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t rd = (size_t)B * H * M * d, f = sizeof(float);
    p.l_state = carve(f * rd);
    p.l_q = carve(f * rd);
    p.l_pp = carve((dtype == SA_BF16 ? 2 : 4) * rd);
    p.l_lse = carve(f * (size_t)T * H);
    p.l_y1 = carve(f * rd);
    p.l_xbar = carve(f * rd);
    p.l_g = carve(f * 2 * rd);
    p.l_u = carve(f * 2 * rd);
    p.l_y2 = carve(f * rd);
    p.l_stride = off;
    return p;
}

// ---------------------------------------------------------------- stacked block backward plan
// [per-layer intermediates (when no saved buffer is given) | the backward's
//  scratch | one region shared by the sketching forward and backward calls]
struct BlockBwdPlan : BlockSaved {
    FwdPlan fwd;
    BwdPlan bshared, buser;
    size_t off_layers = 0, off_xhat = 0, off_z = 0, off_du = 0, off_dy2 = 0, off_dy1 = 0, off_dpp = 0,
           off_dq = 0, off_stats = 0, off_colpart = 0, off_wpart = 0, off_dk = 0, off_dv = 0,
           off_out = 0, off_base = 0, total = 0;
    int64_t nch = 1;
};

BlockBwdPlan plan_block_bwd(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t L, sa_dtype dtype,
                            bool with_saved) {
    BlockBwdPlan p;
    static_cast<BlockSaved&>(p) = saved_layout(B, T, H, M, d, dtype);
    p.fwd = plan_fwd(B, T, H, M, d, dtype, false);
    p.bshared = plan_bwd(B, T, H, M, d, dtype, false);
    p.buser = plan_bwd(B, T, H, M, d, dtype, true);
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t rd = (size_t)B * H * M * d, f = sizeof(float);
    p.off_layers = carve(with_saved ? 0 : p.l_stride * (size_t)L);
    p.off_xhat = carve(f * rd);
    p.off_z = carve(f * 2 * rd);
    p.off_du = carve(f * 2 * rd);
    p.off_dy2 = carve(f * rd);
    p.off_dy1 = carve(f * rd);
    p.off_dpp = carve(f * rd);
    p.off_dq = carve(f * rd);
    p.off_stats = carve(sizeof(float) * 2 * (size_t)B * H * M);
    // column-sum chunks of the norms' gamma / beta gradients: about 1024 workgroups
    p.nch = std::max<int64_t>(1, std::min<int64_t>(B * M, (1024 + H - 1) / H));
    p.off_colpart = carve(f * (size_t)p.nch * H * 2 * d);
    p.off_wpart = carve(f * (size_t)B * H * 2 * d * d);
    if (!p.bshared.fused) {
        p.off_dk = carve(f * (size_t)T * H * d);
        p.off_dv = carve(f * (size_t)T * H * d);
    }
    p.off_out = carve(f * rd);
    p.off_base = carve(std::max({p.fwd.total, p.bshared.total, p.buser.total}));
    p.total = off;
    return p;
}

// parameters of the stacked block, sliced per layer
struct BlockParams {
    const void *Wq, *Wk, *ln, *W1, *W3, *W2;
    int32_t H, d;
    size_t el;
    const void* at(const void* base, size_t per_layer, int32_t l) const {
        return reinterpret_cast<const uint8_t*>(base) + el * per_layer * (size_t)l;
    }
    const void* wq(int32_t l) const { return at(Wq, (size_t)H * d * d, l); }
    const void* wk(int32_t l) const { return at(Wk, (size_t)H * d * d, l); }
    const void* w1(int32_t l) const { return at(W1, (size_t)H * d * 2 * d, l); }
    const void* w3(int32_t l) const { return at(W3, (size_t)H * d * 2 * d, l); }
    const void* w2(int32_t l) const { return at(W2, (size_t)H * 2 * d * d, l); }
    // k = 0: gamma1, 1: beta1, 2: gamma2, 3: beta2
    const void* ln_(int32_t l, int k) const { return at(ln, (size_t)H * d, 4 * l + k); }
};

// Buffers of one layer of the stacked forward.  xt is the layer's state: the
// shared prototypes (input dtype, H * M rows) for the first layer, else fp32
// [B,H,M,d].  Y1, Y2 and Z may be null: without Z the gate is applied to G in place.
struct BlockLayerIo {
    const void* xt;
    bool first;
    float *Q, *lse, *Xhat, *Y1, *Xbar, *G, *U, *Z, *Y2, *out;
    void* Pp;
};

sa_status run_fwd(const void* K, const void* V, const void* P, const int64_t* offsets, int64_t B,
                  int64_t T, int32_t H, int32_t M, int32_t d, float scale, sa_dtype dtype,
                  float* sketch, float* lse, uint8_t* ws, const FwdPlan& plan, hipStream_t stream,
                  bool p_user);

// Batched product of the backward, C[z] (=, or += with accumulate) A[z] B[z'] with
// z' = z % b_mod when b_mod > 0 (per-head weights shared by the users), in the
// layout of launch_small_gemm (C dense [batch][M][N] fp32).  In bf16 mode its fp32
// operands are rounded to bf16 and it runs on the matrix cores when the shapes
// allow; otherwise (and always in fp32 mode) on the fp32 product.
hipError_t grad_gemm(bool bf16_mode, const sa::MatView& a, const sa::MatView& b, float* c, int32_t batch,
                     int32_t M, int32_t N, int32_t K, hipStream_t stream, int32_t b_mod = 0,
                     bool accumulate = false) {
    sa::GemmDesc g{a.p, a.bf16, a.s_h, a.s_0, a.s_1, b.p, b.bf16, b.s_h, b.s_0, b.s_1, c, false,
                   (int64_t)M * N, N, M, N, K, batch, 1.0f, accumulate};
    g.b_mod = b_mod > 0 ? b_mod : 0;
    g.round_bf16 = bf16_mode;
    return sa::launch_gemm(g, stream);
}

// Layer l's intermediates inside a saved region (layout s, L layers); its state
// output is the next layer's state, or `last` for the last layer.  Xhat and Z
// are scratch the caller sets.
BlockLayerIo saved_io(uint8_t* base, const BlockSaved& s, int32_t l, int32_t L, const void* P, float* last) {
    uint8_t* r = base + s.l_stride * (size_t)l;
    BlockLayerIo io{};
    io.first = l == 0;
    io.xt = io.first ? P : reinterpret_cast<const void*>(r + s.l_state);
    io.Q = reinterpret_cast<float*>(r + s.l_q);
    io.Pp = r + s.l_pp;
    io.lse = reinterpret_cast<float*>(r + s.l_lse);
    io.Y1 = reinterpret_cast<float*>(r + s.l_y1);
    io.Xbar = reinterpret_cast<float*>(r + s.l_xbar);
    io.G = reinterpret_cast<float*>(r + s.l_g);
    io.U = reinterpret_cast<float*>(r + s.l_u);
    io.Y2 = reinterpret_cast<float*>(r + s.l_y2);
    io.out = l + 1 < L ? reinterpret_cast<float*>(base + s.l_stride * (size_t)(l + 1) + s.l_state) : last;
    return io;
}

sa_status block_layer_fwd(const void* X, const int64_t* offsets, int64_t B, int64_t T, int32_t H, int32_t M,
                          int32_t d, int32_t l, float scale, float eps, sa_dtype dtype, const BlockParams& w,
                          const BlockLayerIo& io, uint8_t* base_ws, const FwdPlan& base, hipStream_t stream) {
    const bool bf = dtype == SA_BF16;
    const int64_t md = (int64_t)M * d, dd = (int64_t)d * d, d2 = 2 * (int64_t)d;
    const int64_t BH = B * H, rows = BH * M;
    // queries of this layer: the shared prototypes first, then each user's state
    const int64_t nq = io.first ? H : BH;
    hipError_t e;
    {
        sa::ProfScope ps("block_proj", stream);
        const sa::MatView xt{io.xt, io.first && bf, md, d, 1};
        e = sa::launch_small_gemm(xt, {w.wq(l), bf, dd, d, 1}, io.Q, false, (int32_t)nq, M, d, d, stream, H);
        if (e == hipSuccess)
            e = sa::launch_small_gemm({io.Q, false, md, d, 1}, {w.wk(l), bf, dd, 1, d}, io.Pp, bf, (int32_t)nq, M,
                                      d, d, stream, H);
        if (e != hipSuccess) return hip_fail(e, "block projection launch");
    }
    sa_status st = run_fwd(X, X, io.Pp, offsets, B, T, H, M, d, scale, dtype, io.Xhat, io.lse, base_ws, base,
                           stream, !io.first);
    if (st != SA_OK) return st;
    sa::ProfScope ps("block_refine", stream);
    // Xbar = LN1(Xt + Xhat)
    e = sa::launch_add_ln(io.xt, io.first && bf, io.first ? (int64_t)H * M : rows, io.Xhat, w.ln_(l, 0),
                          w.ln_(l, 1), bf, rows, H, M, d, eps, io.Xbar, stream, io.Y1);
    // FFN(Xbar) = (silu(Xbar W1) * (Xbar W3)) W2, into the Xhat buffer
    if (e == hipSuccess)
        e = grad_gemm(bf, {io.Xbar, false, md, d, 1}, {w.w1(l), bf, d * d2, d2, 1}, io.G, (int32_t)BH, M,
                      (int32_t)d2, d, stream, H);
    if (e == hipSuccess)
        e = grad_gemm(bf, {io.Xbar, false, md, d, 1}, {w.w3(l), bf, d * d2, d2, 1}, io.U, (int32_t)BH, M,
                      (int32_t)d2, d, stream, H);
    float* Z = io.Z ? io.Z : io.G;
    if (e == hipSuccess)
        e = io.Z ? sa::launch_swiglu_fwd(io.G, io.U, io.Z, rows * d2, stream)
                 : sa::launch_swiglu_gate(io.G, io.U, rows * d2, stream);
    if (e == hipSuccess)
        e = grad_gemm(bf, {Z, false, M * d2, d2, 1}, {w.w2(l), bf, d2 * d, d, 1}, io.Xhat, (int32_t)BH, M, d,
                      (int32_t)d2, stream, H);
    // Xt' = LN2(Xbar + FFN)
    if (e == hipSuccess)
        e = sa::launch_add_ln(io.Xbar, false, rows, io.Xhat, w.ln_(l, 2), w.ln_(l, 3), bf, rows, H, M, d, eps,
                              io.out, stream, io.Y2);
    if (e != hipSuccess) return hip_fail(e, "block refinement launch");
    return SA_OK;
}

// ---------------------------------------------------------------- STCA over the sketch
// [Qp | U | S | alpha | C | lse (fp32) | (bwd) dout in the operand dtype | dC |
//  dalpha (fp32) | ds | dU | dQp]; operand buffers in the input dtype.  Per user b,
// target r and head i: Qp = q W_Q [B,R,D]; U = per-head (Qp W_K^T) [B,R,h,D]; S =
// scale U Xs^T [B,R h,k]; alpha = softmax rows; C = alpha Xs [B,R,h,D].
struct StcaPlan {
    size_t off_qp = 0, off_u = 0, off_s = 0, off_al = 0, off_c = 0, off_lse = 0, off_dob = 0, off_dc = 0,
           off_da = 0, off_ds = 0, off_du = 0, off_dqp = 0, total = 0;
};

StcaPlan plan_stca(int64_t B, int32_t R, int32_t k, int32_t D, int32_t h, sa_dtype dtype, bool bwd) {
    StcaPlan p;
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t el = dtype == SA_BF16 ? 2 : 4;
    const size_t BR = (size_t)B * R, rows = BR * h;
    p.off_qp = carve(el * BR * D);
    p.off_u = carve(el * rows * D);
    p.off_s = carve(el * rows * k);
    p.off_al = carve(el * rows * k);
    p.off_c = carve(el * rows * D);
    p.off_lse = carve(4 * rows);
    if (bwd) {
        p.off_dob = carve(dtype == SA_BF16 ? el * BR * D : 0);
        p.off_dc = carve(el * rows * D);
        p.off_da = carve(4 * rows * k);
        p.off_ds = carve(el * rows * k);
        p.off_du = carve(el * rows * D);
        p.off_dqp = carve(el * BR * D);
    }
    p.total = off;
    return p;
}

sa_status check_stca(int64_t B, int32_t R, int32_t k, int32_t D, int32_t h, float scale, sa_dtype dtype) {
    if (dtype != SA_BF16 && dtype != SA_FP32) return fail(SA_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    if (B < 0 || R < 1 || k < 1 || D < 1 || h < 1)
        return fail(SA_ERR_INVALID_ARG, "bad sizes B=%lld R=%d k=%d D=%d h=%d", (long long)B, R, k, D, h);
    if (D % h != 0) return fail(SA_ERR_INVALID_ARG, "D=%d is not a multiple of h=%d", D, h);
    if (!(std::isfinite(scale) && scale > 0.f)) return fail(SA_ERR_INVALID_ARG, "scale must be finite and > 0");
    if (B > 65535 || B * R * (int64_t)h >= (int64_t(1) << 31) || (int64_t)R * h * k >= (int64_t(1) << 31))
        return fail(SA_ERR_UNSUPPORTED, "sizes beyond the supported range");
    return SA_OK;
}

sa_status stca_forward(const void* Xs, const void* q, const void* Wq, const void* Wk, const void* Wv, int64_t B,
                       int32_t R, int32_t k, int32_t D, int32_t h, float scale, sa_dtype dtype, float* out,
                       float* lse, uint8_t* ws, const StcaPlan& p, hipStream_t stream) {
    const bool bf = dtype == SA_BF16;
    const int32_t BR = (int32_t)(B * R), dh = D / h, Rh = R * h;
    const int64_t kD = (int64_t)k * D, RhD = (int64_t)Rh * D, Rhk = (int64_t)Rh * k;
    void* Qp = ws + p.off_qp;
    void* U = ws + p.off_u;
    void* S = ws + p.off_s;   // logits, in the operand dtype
    void* Al = ws + p.off_al;
    void* Cc = ws + p.off_c;
    hipError_t e;
    {
        sa::ProfScope ps("stca_query_proj", stream);
        // Qp = q W_Q;  U[., i] = Qp[., head i] W_K^(i)T
        e = sa::launch_gemm({q, bf, 0, D, 1, Wq, bf, 0, D, 1, Qp, bf, 0, D, BR, D, D, 1, 1.f, false}, stream);
        if (e == hipSuccess)
            e = sa::launch_gemm({Qp, bf, dh, D, 1, Wk, bf, dh, 1, D, U, bf, D, (int64_t)h * D, BR, D, dh, h, 1.f,
                                 false}, stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_logits", stream);   // S = scale U Xs^T per user
        e = sa::launch_gemm({U, bf, RhD, D, 1, Xs, bf, kD, 1, D, S, bf, Rhk, k, Rh, k, D, (int32_t)B, scale, false},
                            stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_softmax", stream);
        e = sa::launch_stca_softmax(S, bf, (int64_t)BR * h, k, bf, Al, lse, stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_aggregate", stream);   // C = alpha Xs per user
        e = sa::launch_gemm({Al, bf, Rhk, k, 1, Xs, bf, kD, D, 1, Cc, bf, RhD, D, Rh, D, k, (int32_t)B, 1.f, false},
                            stream);
    }
    if (e == hipSuccess && out) {
        sa::ProfScope ps("stca_value_proj", stream);   // out[., head i] = C[., i] W_V^(i)
        e = sa::launch_gemm({Cc, bf, D, (int64_t)h * D, 1, Wv, bf, dh, D, 1, out, false, dh, D, BR, dh, D, h, 1.f,
                             false}, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "STCA forward launch");
    return SA_OK;
}

// forward on a checked plan and workspace (shared by sa_sketch_fwd and sa_layer_fwd)
sa_status run_fwd(const void* K, const void* V, const void* P, const int64_t* offsets, int64_t B,
                  int64_t T, int32_t H, int32_t M, int32_t d, float scale, sa_dtype dtype,
                  float* sketch, float* lse, uint8_t* ws, const FwdPlan& plan, hipStream_t stream,
                  bool p_user) {
    hipError_t e;
    int32_t* items = reinterpret_cast<int32_t*>(ws + plan.off_items);
    int32_t* wg_start = reinterpret_cast<int32_t*>(ws + plan.off_wgstart);
    int32_t* pair_start = reinterpret_cast<int32_t*>(ws + plan.off_pairstart);
    int64_t* n_items = reinterpret_cast<int64_t*>(ws + plan.off_nitems);
    float* partials = reinterpret_cast<float*>(ws + plan.off_partials);
    {
        sa::ProfScope ps("worklist", stream);
        e = sa::launch_worklist(offsets, B, T, H, plan.C, plan.n_ranges, items, plan.max_items, wg_start,
                                pair_start, n_items, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "work list launch");
    if (plan.fused) {
        sa::FusedFwdArgs a;
        a.K = reinterpret_cast<const uint16_t*>(K);
        a.V = reinterpret_cast<const uint16_t*>(V);
        a.P = reinterpret_cast<const uint16_t*>(P);
        a.items = items;
        a.wg_start = wg_start;
        a.n_ranges = plan.n_ranges;
        a.max_items = plan.max_items;
        a.T = T;
        a.B = (int32_t)B;
        a.H = H;
        a.M = M;
        a.d = d;
        a.scale = scale;
        a.sketch = sketch;
        a.lse = lse;
        a.partials = partials;
        a.p_user = p_user;
        {
            sa::ProfScope ps("fused_fwd", stream);
            e = sa::launch_fused_fwd(a, stream);
        }
        if (e != hipSuccess) return hip_fail(e, "fused forward launch");
        {
            sa::ProfScope ps("splitL_merge", stream);
            e = sa::launch_merge(pair_start, B, H, plan.max_items, partials, (int64_t)M * d,
                                 sketch, stream);
        }
        if (e != hipSuccess) return hip_fail(e, "split-L merge launch");
        return SA_OK;
    }
    float* lse_out = lse ? lse : reinterpret_cast<float*>(ws + plan.off_lse);
    {
        sa::ProfScope ps("plain_fwd", stream);
        sa::GenericFwdItems wi;
        wi.items = items;
        wi.wg_start = wg_start;
        wi.n_ranges = plan.n_ranges;
        wi.max_items = plan.max_items;
        wi.partials = partials;
        e = sa::launch_generic_fwd(K, V, P, offsets, B, T, H, M, d, scale, dtype == SA_BF16, sketch, lse_out, wi,
                                   stream, p_user);
    }
    if (e != hipSuccess) return hip_fail(e, "fp32 forward launch");
    {
        sa::ProfScope ps("splitL_merge", stream);
        e = sa::launch_merge(pair_start, B, H, plan.max_items, partials, (int64_t)M * d, sketch, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "split-L merge launch");
    return SA_OK;
}


// backward on a checked plan and workspace.  With dX non-null, K and V are the
// same tensor X and the gradient w.r.t. it, dX = dK + dV, is written (added to dX
// with dx_add) instead of dK and dV (the plain path still needs dK and dV as
// scratch).
sa_status run_bwd(const void* K, const void* V, const void* P, const int64_t* offsets, int64_t B,
                  int64_t T, int32_t H, int32_t M, int32_t d, float scale, sa_dtype dtype,
                  const float* dsketch, int32_t R, const float* lse, float* dK, float* dV,
                  float* dP, float* dX, uint8_t* ws, const BwdPlan& plan, hipStream_t stream,
                  bool p_user = false, bool dx_add = false) {
    float* dY = reinterpret_cast<float*>(ws + plan.off_dY);
    float* Dbuf = reinterpret_cast<float*>(ws + plan.off_D);
    float* part = reinterpret_cast<float*>(ws + plan.off_part);
    hipError_t e;
    if (plan.fused) {
        sa::FusedBwdArgs f;
        f.K = reinterpret_cast<const uint16_t*>(K);
        f.V = reinterpret_cast<const uint16_t*>(V);
        f.P = reinterpret_cast<const uint16_t*>(P);
        f.dsketch = dsketch;
        f.lse = lse;
        f.items = reinterpret_cast<int32_t*>(ws + plan.off_items);
        f.wg_start = reinterpret_cast<int32_t*>(ws + plan.off_wgstart);
        f.pair_start = reinterpret_cast<int32_t*>(ws + plan.off_pairstart);
        f.n_ranges = plan.n_ranges;
        f.max_items = plan.max_items;
        f.B = B;
        f.T = T;
        f.H = H;
        f.M = M;
        f.d = d;
        f.R = R;
        f.scale = scale;
        f.Ymj = reinterpret_cast<uint16_t*>(ws + plan.off_ymj);
        f.Yjm = reinterpret_cast<uint16_t*>(ws + plan.off_yjm);
        f.Pjm = reinterpret_cast<uint16_t*>(ws + plan.off_pjm);
        f.Dbuf = Dbuf;
        f.partials = part;
        f.dK = dK;
        f.dV = dV;
        f.dP = dP;
        f.dX = dX;
        f.p_user = p_user;
        f.dx_add = dx_add;
        {
            sa::ProfScope ps("bwd_worklist", stream);
            e = sa::launch_worklist(offsets, B, T, H, plan.C, plan.n_ranges,
                                    const_cast<int32_t*>(f.items), plan.max_items,
                                    const_cast<int32_t*>(f.wg_start),
                                    const_cast<int32_t*>(f.pair_start),
                                    reinterpret_cast<int64_t*>(ws + plan.off_nitems), stream);
        }
        if (e != hipSuccess) return hip_fail(e, "work list launch");
        e = sa::launch_fused_bwd(f, stream);
        if (e != hipSuccess) return hip_fail(e, "fused backward launch");
        return SA_OK;
    }
    {
        sa::ProfScope ps("dY_reduce", stream);
        e = sa::launch_dy_reduce(dsketch, B, R, H, (int64_t)M * d, dY, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "dY reduce launch");
    {
        sa::ProfScope ps("plain_bwd", stream);
        e = sa::launch_generic_bwd(K, V, P, offsets, B, T, H, M, d, scale, dtype == SA_BF16, dY,
                                   lse, Dbuf, dK, dV, dP, part, plan.n_chunks, stream, p_user);
    }
    if (e != hipSuccess) return hip_fail(e, "backward launch");
    if (dX) {
        sa::ProfScope ps("dX_sum", stream);
        e = sa::launch_add(dK, dV, dx_add ? dK : dX, T * H * d, stream);
        if (e == hipSuccess && dx_add) e = sa::launch_add(dX, dK, dX, T * H * d, stream);
        if (e != hipSuccess) return hip_fail(e, "dX sum launch");
    }
    return SA_OK;
}


}  // namespace

namespace sa {

// per-device constant: number of compute units (read once per device)
static constexpr int kMaxCuDevices = 64;
static std::once_flag g_cu_once[kMaxCuDevices];
static int g_cu_count[kMaxCuDevices];

int device_cus() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxCuDevices) return 256;
    std::call_once(g_cu_once[dev], [dev] {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        g_cu_count[dev] = n;
    });
    return g_cu_count[dev];
}

ProfScope::ProfScope(const char* name, hipStream_t stream) : stream_(stream) {
    if (!g_prof_on) return;
    name_ = name;
    start_ = prof_event();
    stop_ = prof_event();
    if (start_ && stop_ && hipEventRecord(start_, stream_) == hipSuccess) active_ = true;
}

ProfScope::~ProfScope() {
    if (!active_) return;
    if (hipEventRecord(stop_, stream_) == hipSuccess) g_prof_recs.push_back({name_, start_, stop_});
}

}  // namespace sa

extern "C" {

const char* sa_status_string(sa_status s) {
    switch (s) {
        case SA_OK: return "SA_OK";
        case SA_ERR_INVALID_ARG: return "SA_ERR_INVALID_ARG";
        case SA_ERR_UNSUPPORTED: return "SA_ERR_UNSUPPORTED";
        case SA_ERR_WORKSPACE: return "SA_ERR_WORKSPACE";
        case SA_ERR_BAD_OFFSETS: return "SA_ERR_BAD_OFFSETS";
        case SA_ERR_HIP: return "SA_ERR_HIP";
    }
    return "SA_ERR_UNKNOWN";
}

const char* sa_last_error(void) { return g_last_error; }

size_t sa_sketch_fwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                    sa_dtype dtype) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK) return 0;
    // the plain path needs lse scratch only when the caller passes lse = NULL;
    // size for that case so one query serves both
    return plan_fwd(B, T, H, M, d, dtype, true).total;
}

int64_t sa_sketch_fwd_chunk_tokens(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   sa_dtype dtype) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK) return 0;
    return plan_fwd(B, T, H, M, d, dtype, false).C;
}

sa_status sa_sketch_fwd(const void* K, const void* V, const void* P, const int64_t* offsets,
                        int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                        sa_dtype dtype, float* sketch, float* lse, void* workspace,
                        size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (B == 0) return SA_OK;
    if (!offsets || !sketch || !P || (T > 0 && (!K || !V)))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(K) || !aligned16(V) || !aligned16(P) || !aligned16(sketch) ||
        !aligned16(lse))
        return fail(SA_ERR_INVALID_ARG, "K, V, P, sketch and lse must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const FwdPlan plan = plan_fwd(B, T, H, M, d, dtype, lse == nullptr);
    if (plan.total > 0 && (!workspace || workspace_bytes < plan.total))
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (debug_validate()) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    return run_fwd(K, V, P, offsets, B, T, H, M, d, scale, dtype, sketch, lse,
                   reinterpret_cast<uint8_t*>(workspace), plan, stream, false);
}

}  // extern "C"

namespace {

// Scratch space of sa_sketch_fwd_noalloc: one array per device, alive until the
// process ends.  Host code never passes `scratch` itself to a kernel (on the
// host the name stands for a host-side shadow, not a device address): each
// device's address is looked up once, with that device current, and kept.
__device__ __align__(256) uint8_t scratch[SA_NOALLOC_SCRATCH_BYTES];

std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// device address of this device's scratch array, or null (error in *err)
uint8_t* device_scratch(hipError_t* err) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        *err = e != hipSuccess ? e : hipErrorInvalidDevice;
        return nullptr;
    }
    std::call_once(g_scratch_once[dev], [dev] {
        void* ptr = nullptr;
        g_scratch_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? ptr : nullptr;
    });
    *err = g_scratch_err[dev];
    return reinterpret_cast<uint8_t*>(g_scratch_ptr[dev]);
}

}  // namespace

extern "C" {

sa_status sa_sketch_fwd_noalloc(const void* K, const void* V, const void* P, const int64_t* offsets,
                                int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                                sa_dtype dtype, float* sketch, float* lse, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (B == 0) return SA_OK;
    if (!offsets || !sketch || !P || (T > 0 && (!K || !V)))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(K) || !aligned16(V) || !aligned16(P) || !aligned16(sketch) ||
        !aligned16(lse))
        return fail(SA_ERR_INVALID_ARG, "K, V, P, sketch and lse must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const FwdPlan plan = plan_fwd(B, T, H, M, d, dtype, lse == nullptr);
    if (plan.total > (size_t)SA_NOALLOC_SCRATCH_BYTES)
        return fail(SA_ERR_WORKSPACE,
                    "this shape needs %zu bytes of scratch; the no-allocation forward holds %zu "
                    "(use sa_sketch_fwd with a workspace)",
                    plan.total, (size_t)SA_NOALLOC_SCRATCH_BYTES);
    hipError_t e = hipSuccess;
    uint8_t* ws = device_scratch(&e);
    if (!ws) return hip_fail(e, "looking up the device scratch array");
    // no per-launch timing events here (creating them is an allocation)
    const bool prof = g_prof_on;
    g_prof_on = false;
    st = run_fwd(K, V, P, offsets, B, T, H, M, d, scale, dtype, sketch, lse, ws, plan, stream, false);
    g_prof_on = prof;
    return st;
}

size_t sa_sketch_fwd_tokenwise_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M,
                                              int32_t d, sa_dtype dtype) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK) return 0;
    return plan_tokenwise(B, T, H, M, d, dtype).total;
}

sa_status sa_sketch_fwd_tokenwise(const void* K, const void* V, const void* P,
                                  const int64_t* offsets, int64_t B, int64_t T, int32_t H,
                                  int32_t M, int32_t d, float scale, sa_dtype dtype, float* sketch,
                                  float* lse_m, void* workspace, size_t workspace_bytes,
                                  void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (B == 0) return SA_OK;
    if (!offsets || !sketch || !P || (T > 0 && (!K || !V)))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(K) || !aligned16(V) || !aligned16(P) || !aligned16(sketch) ||
        !aligned16(lse_m))
        return fail(SA_ERR_INVALID_ARG, "K, V, P, sketch and lse_m must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const TwPlan plan = plan_tokenwise(B, T, H, M, d, dtype);
    if (plan.total > 0 && (!workspace || workspace_bytes < plan.total))
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (debug_validate()) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    hipError_t e;
    if (plan.fused) {
        uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
        int32_t* items = reinterpret_cast<int32_t*>(ws + plan.off_items);
        int32_t* wg_start = reinterpret_cast<int32_t*>(ws + plan.off_wgstart);
        int32_t* pair_start = reinterpret_cast<int32_t*>(ws + plan.off_pairstart);
        int64_t* n_items = reinterpret_cast<int64_t*>(ws + plan.off_nitems);
        float* partials = reinterpret_cast<float*>(ws + plan.off_partials);
        float* stats = reinterpret_cast<float*>(ws + plan.off_stats);
        {
            sa::ProfScope ps("worklist", stream);
            e = sa::launch_worklist(offsets, B, T, H, plan.C, plan.n_ranges, items,
                                    plan.max_items, wg_start, pair_start, n_items, stream);
        }
        if (e != hipSuccess) return hip_fail(e, "work list launch");
        {
            sa::ProfScope ps("tokenwise_fwd", stream);
            e = sa::launch_tokenwise_fused(items, wg_start, plan.n_ranges, plan.max_items, K, V, P,
                                           B, T, H, M, d, scale, sketch, lse_m, partials, stats,
                                           stream);
        }
        if (e != hipSuccess) return hip_fail(e, "token-wise forward launch");
        {
            sa::ProfScope ps("tokenwise_merge", stream);
            e = sa::launch_tokenwise_merge(pair_start, B, H, M, d, plan.max_items, partials, stats,
                                           sketch, lse_m, stream);
        }
        if (e != hipSuccess) return hip_fail(e, "token-wise merge launch");
        return SA_OK;
    }
    {
        sa::ProfScope ps("tokenwise_plain", stream);
        e = sa::launch_tokenwise_generic(K, V, P, offsets, B, H, M, d, scale, dtype == SA_BF16,
                                         sketch, lse_m, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "token-wise plain launch");
    return SA_OK;
}

size_t sa_sketch_bwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                    sa_dtype dtype, int32_t R) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK || R < 1) return 0;
    return plan_bwd(B, T, H, M, d, dtype).total;
}

sa_status sa_sketch_bwd(const void* K, const void* V, const void* P, const int64_t* offsets,
                        int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, float scale,
                        sa_dtype dtype, const float* dsketch, int32_t R, const float* lse,
                        float* dK, float* dV, float* dP, void* workspace,
                        size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (R < 1) return fail(SA_ERR_INVALID_ARG, "R must be >= 1 (got %d)", R);
    if (!offsets || !P || !dP || (B > 0 && !dsketch) ||
        (T > 0 && (!K || !V || !lse || !dK || !dV)))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(K) || !aligned16(V) || !aligned16(P) || !aligned16(dsketch) ||
        !aligned16(lse) || !aligned16(dK) || !aligned16(dV) || !aligned16(dP))
        return fail(SA_ERR_INVALID_ARG, "tensor arguments must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const BwdPlan plan = plan_bwd(B, T, H, M, d, dtype);
    if (plan.total > 0 && (!workspace || workspace_bytes < plan.total))
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (debug_validate() && B > 0) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    return run_bwd(K, V, P, offsets, B, T, H, M, d, scale, dtype, dsketch, R, lse, dK, dV, dP,
                   nullptr, reinterpret_cast<uint8_t*>(workspace), plan, stream);
}

size_t sa_layer_fwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   sa_dtype dtype) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK) return 0;
    return plan_layer(T, H, M, d, dtype, false, false, plan_fwd(B, T, H, M, d, dtype, true).total)
        .total;
}

sa_status sa_layer_fwd(const void* X, const void* P, const void* Wq, const void* Wk,
                       const int64_t* offsets, int64_t B, int64_t T, int32_t H, int32_t M,
                       int32_t d, float scale, sa_dtype dtype, float* sketch, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (B == 0) return SA_OK;
    if (!offsets || !sketch || !P || !Wq || !Wk || (T > 0 && !X))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(X) || !aligned16(P) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(sketch) ||
        !aligned16(lse))
        return fail(SA_ERR_INVALID_ARG, "X, P, W_Q, W_K, sketch and lse must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const FwdPlan base = plan_fwd(B, T, H, M, d, dtype, lse == nullptr);
    const LayerPlan plan = plan_layer(T, H, M, d, dtype, false, false, base.total);
    if (!workspace || workspace_bytes < plan.total)
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (debug_validate()) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    float* Q = reinterpret_cast<float*>(ws + plan.off_q);
    void* Pp = ws + plan.off_pp;
    st = layer_prototypes(P, Wq, Wk, H, M, d, dtype, Q, Pp, stream);
    if (st != SA_OK) return st;
    return run_fwd(X, X, Pp, offsets, B, T, H, M, d, scale, dtype, sketch, lse, ws + plan.off_base,
                   base, stream, false);
}

size_t sa_layer_bwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   sa_dtype dtype, int32_t R) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK || R < 1) return 0;
    const BwdPlan base = plan_bwd(B, T, H, M, d, dtype);
    return plan_layer(T, H, M, d, dtype, true, !base.fused, base.total).total;
}

sa_status sa_layer_bwd(const void* X, const void* P, const void* Wq, const void* Wk,
                       const int64_t* offsets, int64_t B, int64_t T, int32_t H, int32_t M,
                       int32_t d, float scale, sa_dtype dtype, const float* dsketch, int32_t R,
                       const float* lse, float* dX, float* dP, float* dWq, float* dWk,
                       void* workspace, size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (R < 1) return fail(SA_ERR_INVALID_ARG, "R must be >= 1 (got %d)", R);
    if (!offsets || !P || !Wq || !Wk || !dP || !dWq || !dWk || (B > 0 && !dsketch) ||
        (T > 0 && (!X || !lse || !dX)))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(X) || !aligned16(P) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(dsketch) ||
        !aligned16(lse) || !aligned16(dX) || !aligned16(dP) || !aligned16(dWq) || !aligned16(dWk))
        return fail(SA_ERR_INVALID_ARG, "tensor arguments must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const BwdPlan base = plan_bwd(B, T, H, M, d, dtype);
    const LayerPlan plan = plan_layer(T, H, M, d, dtype, true, !base.fused, base.total);
    if (!workspace || workspace_bytes < plan.total)
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (debug_validate() && B > 0) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    float* Q = reinterpret_cast<float*>(ws + plan.off_q);
    void* Pp = ws + plan.off_pp;
    float* dPp = reinterpret_cast<float*>(ws + plan.off_dpp);
    float* dQ = reinterpret_cast<float*>(ws + plan.off_dq);
    st = layer_prototypes(P, Wq, Wk, H, M, d, dtype, Q, Pp, stream);
    if (st != SA_OK) return st;
    float* dKs = base.fused ? nullptr : reinterpret_cast<float*>(ws + plan.off_dk);
    float* dVs = base.fused ? nullptr : reinterpret_cast<float*>(ws + plan.off_dv);
    st = run_bwd(X, X, Pp, offsets, B, T, H, M, d, scale, dtype, dsketch, R, lse, dKs, dVs, dPp, dX,
                 ws + plan.off_base, base, stream);
    if (st != SA_OK) return st;
    // dW_K = dP'^T Q, dQ = dP' W_K, dW_Q = P^T dQ, dP = dQ W_Q^T
    const bool bf = dtype == SA_BF16;
    const int64_t md = (int64_t)M * d, dd = (int64_t)d * d;
    sa::ProfScope ps("layer_proj_grads", stream);
    // (fp32 products: with identity projections dP equals the sketching step's dP
    // bit for bit)
    hipError_t e = sa::launch_small_gemm({dPp, false, md, 1, d}, {Q, false, md, d, 1}, dWk, false, H, d,
                                         d, M, stream);
    if (e == hipSuccess)
        e = sa::launch_small_gemm({dPp, false, md, d, 1}, {Wk, bf, dd, d, 1}, dQ, false, H, M, d, d, stream);
    if (e == hipSuccess)
        e = sa::launch_small_gemm({P, bf, md, 1, d}, {dQ, false, md, d, 1}, dWq, false, H, d, d, M, stream);
    if (e == hipSuccess)
        e = sa::launch_small_gemm({dQ, false, md, d, 1}, {Wq, bf, dd, 1, d}, dP, false, H, M, d, d, stream);
    if (e != hipSuccess) return hip_fail(e, "projection gradient launch");
    return SA_OK;
}

size_t sa_block_fwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   int32_t n_layers, sa_dtype dtype) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK || n_layers < 1) return 0;
    return plan_block(B, T, H, M, d, dtype).total;
}

size_t sa_block_saved_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers,
                           sa_dtype dtype) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK || n_layers < 1) return 0;
    return saved_layout(B, T, H, M, d, dtype).l_stride * (size_t)n_layers;
}

size_t sa_block_saved_offset(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers,
                             sa_dtype dtype, int32_t layer, int32_t item) {
    const size_t bad = ~(size_t)0;
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK || n_layers < 1 || layer < 0 || layer >= n_layers)
        return bad;
    const BlockSaved s = saved_layout(B, T, H, M, d, dtype);
    const size_t base = s.l_stride * (size_t)layer;
    switch (item) {
        case SA_SAVED_STATE: return layer == 0 ? bad : base + s.l_state;
        case SA_SAVED_Q: return base + s.l_q;
        case SA_SAVED_PP: return base + s.l_pp;
        case SA_SAVED_LSE: return base + s.l_lse;
        default: return bad;
    }
}

sa_status sa_block_fwd(const void* X, const void* P, const void* Wq, const void* Wk, const void* ln,
                       const void* W1, const void* W3, const void* W2, const int64_t* offsets, int64_t B,
                       int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers, float scale, float eps,
                       sa_dtype dtype, float* out, float* lse, void* saved, size_t saved_bytes, void* workspace,
                       size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (n_layers < 1) return fail(SA_ERR_INVALID_ARG, "n_layers must be >= 1 (got %d)", n_layers);
    if (!(std::isfinite(eps) && eps > 0.f)) return fail(SA_ERR_INVALID_ARG, "eps must be finite and > 0");
    if (B == 0) return SA_OK;
    if (!offsets || !out || !P || !Wq || !Wk || !ln || !W1 || !W3 || !W2 || (T > 0 && !X))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(X) || !aligned16(P) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(ln) || !aligned16(W1) ||
        !aligned16(W3) || !aligned16(W2) || !aligned16(out) || !aligned16(lse))
        return fail(SA_ERR_INVALID_ARG, "tensor arguments must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const BlockPlan plan = plan_block(B, T, H, M, d, dtype);
    if (!workspace || workspace_bytes < plan.total)
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    const BlockSaved sl = saved_layout(B, T, H, M, d, dtype);
    if (saved && (saved_bytes < sl.l_stride * (size_t)n_layers || !aligned16(saved)))
        return fail(SA_ERR_WORKSPACE, "saved buffer of %zu bytes (16-byte aligned) needed, %zu given",
                    sl.l_stride * (size_t)n_layers, saved_bytes);
    if (debug_validate()) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    float* state = reinterpret_cast<float*>(ws + plan.off_state);
    const BlockParams w{Wq, Wk, ln, W1, W3, W2, H, d, (size_t)(dtype == SA_BF16 ? 2 : 4)};
    if (saved) {
        // training forward: every layer's intermediates stay in `saved` for the
        // backward (the gate output goes to scratch so that G is kept)
        for (int32_t l = 0; l < n_layers; ++l) {
            BlockLayerIo io = saved_io(reinterpret_cast<uint8_t*>(saved), sl, l, n_layers, P, out);
            io.Xhat = reinterpret_cast<float*>(ws + plan.off_xhat);
            io.Z = reinterpret_cast<float*>(ws + plan.off_g);
            st = block_layer_fwd(X, offsets, B, T, H, M, d, l, scale, eps, dtype, w, io, ws + plan.off_base,
                                 plan.base, stream);
            if (st != SA_OK) return st;
            if (lse && T > 0) {
                const hipError_t e = hipMemcpyAsync(lse + (size_t)l * T * H, io.lse, sizeof(float) * (size_t)T * H,
                                                    hipMemcpyDeviceToDevice, stream);
                if (e != hipSuccess) return hip_fail(e, "lse copy");
            }
        }
        return SA_OK;
    }
    for (int32_t l = 0; l < n_layers; ++l) {
        BlockLayerIo io{};
        io.first = l == 0;
        io.xt = io.first ? P : state;
        io.Q = reinterpret_cast<float*>(ws + plan.off_q);
        io.Pp = ws + plan.off_pp;
        io.lse = lse ? lse + (size_t)l * T * H : reinterpret_cast<float*>(ws + plan.off_lse);
        io.Xhat = reinterpret_cast<float*>(ws + plan.off_xhat);
        io.Xbar = reinterpret_cast<float*>(ws + plan.off_xbar);
        io.G = reinterpret_cast<float*>(ws + plan.off_g);
        io.U = reinterpret_cast<float*>(ws + plan.off_u);
        io.out = l == n_layers - 1 ? out : state;
        st = block_layer_fwd(X, offsets, B, T, H, M, d, l, scale, eps, dtype, w, io, ws + plan.off_base, plan.base,
                             stream);
        if (st != SA_OK) return st;
    }
    return SA_OK;
}

size_t sa_block_bwd_workspace_size(int64_t B, int64_t T, int32_t H, int32_t M, int32_t d,
                                   int32_t n_layers, sa_dtype dtype, int32_t with_saved) {
    if (check_common(B, T, H, M, d, 1.0f, dtype) != SA_OK || n_layers < 1) return 0;
    return plan_block_bwd(B, T, H, M, d, n_layers, dtype, with_saved != 0).total;
}

sa_status sa_block_bwd(const void* X, const void* P, const void* Wq, const void* Wk, const void* ln,
                       const void* W1, const void* W3, const void* W2, const int64_t* offsets, int64_t B,
                       int64_t T, int32_t H, int32_t M, int32_t d, int32_t n_layers, float scale, float eps,
                       sa_dtype dtype, const float* dout, float* dX, float* dP, float* dWq, float* dWk,
                       float* dln, float* dW1, float* dW3, float* dW2, const void* saved, size_t saved_bytes,
                       void* workspace, size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_common(B, T, H, M, d, scale, dtype);
    if (st != SA_OK) return st;
    if (n_layers < 1) return fail(SA_ERR_INVALID_ARG, "n_layers must be >= 1 (got %d)", n_layers);
    if (!(std::isfinite(eps) && eps > 0.f)) return fail(SA_ERR_INVALID_ARG, "eps must be finite and > 0");
    if (B < 1) return fail(SA_ERR_INVALID_ARG, "B must be >= 1 for the backward (got %lld)", (long long)B);
    if (B > 65535) return fail(SA_ERR_UNSUPPORTED, "more than 65535 users");
    if (!offsets || !P || !Wq || !Wk || !ln || !W1 || !W3 || !W2 || !dout || !dP || !dWq || !dWk || !dln ||
        !dW1 || !dW3 || !dW2 || (T > 0 && (!X || !dX)))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(X) || !aligned16(P) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(ln) || !aligned16(W1) ||
        !aligned16(W3) || !aligned16(W2) || !aligned16(dout) || !aligned16(dX) || !aligned16(dP) ||
        !aligned16(dWq) || !aligned16(dWk) || !aligned16(dln) || !aligned16(dW1) || !aligned16(dW3) ||
        !aligned16(dW2))
        return fail(SA_ERR_INVALID_ARG, "tensor arguments must be 16-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const BlockBwdPlan plan = plan_block_bwd(B, T, H, M, d, n_layers, dtype, saved != nullptr);
    if (!workspace || workspace_bytes < plan.total)
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (saved && (saved_bytes < plan.l_stride * (size_t)n_layers || !aligned16(saved)))
        return fail(SA_ERR_WORKSPACE, "saved buffer of %zu bytes (16-byte aligned) needed, %zu given",
                    plan.l_stride * (size_t)n_layers, saved_bytes);
    if (debug_validate()) {
        st = validate_offsets(offsets, B, T, stream);
        if (st != SA_OK) return st;
    }
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    auto F = [&](size_t o) { return reinterpret_cast<float*>(ws + o); };
    const BlockParams w{Wq, Wk, ln, W1, W3, W2, H, d, (size_t)(dtype == SA_BF16 ? 2 : 4)};
    const bool bf = dtype == SA_BF16;
    const int64_t md = (int64_t)M * d, dd = (int64_t)d * d, d2 = 2 * (int64_t)d;
    const int64_t BH = B * H, rows = BH * M;
    // the intermediates: the caller's saved buffer (read only), or the workspace
    uint8_t* layers = saved ? reinterpret_cast<uint8_t*>(const_cast<void*>(saved)) : ws + plan.off_layers;
    auto layer_io = [&](int32_t l) {
        BlockLayerIo io = saved_io(layers, plan, l, n_layers, P, F(plan.off_out));
        io.Xhat = F(plan.off_xhat);
        io.Z = F(plan.off_z);
        return io;
    };
    // without a saved buffer: forward replay keeping every layer's intermediates
    for (int32_t l = 0; !saved && l < n_layers; ++l) {
        st = block_layer_fwd(X, offsets, B, T, H, M, d, l, scale, eps, dtype, w, layer_io(l), ws + plan.off_base,
                             plan.fwd, stream);
        if (st != SA_OK) return st;
    }
    float* Zb = F(plan.off_z);     // Z, then dZ, then dG
    float* dU = F(plan.off_du);
    float* dY2 = F(plan.off_dy2);
    float* dY1 = F(plan.off_dy1);  // the state gradient of the layer below
    float* dXbar = F(plan.off_xhat);
    float* dPp = F(plan.off_dpp);
    float* dQ = F(plan.off_dq);
    float* wpart = F(plan.off_wpart);
    float2* stats = reinterpret_cast<float2*>(ws + plan.off_stats);
    float* colpart = F(plan.off_colpart);
    const float* dXt = dout;
    hipError_t e = hipSuccess;
    for (int32_t l = n_layers - 1; l >= 0; --l) {
        const BlockLayerIo io = layer_io(l);
        const int64_t nq = io.first ? H : BH;
        float* dlnl = dln + (size_t)4 * l * H * d;
        {
            sa::ProfScope ps("block_refine_bwd", stream);
            // LN2: dY2, dgamma2, dbeta2
            e = sa::launch_ln_bwd(dXt, nullptr, io.Y2, w.ln_(l, 2), bf, B, H, M, d, eps, dY2, stats, colpart,
                                  plan.nch, dlnl + 2 * (size_t)H * d, (int64_t)H * d, stream);
            // dW2 = sum over users of Z^T dY2, dZ = dY2 W2^T
            if (e == hipSuccess) e = sa::launch_swiglu_fwd(io.G, io.U, Zb, rows * d2, stream);
            if (e == hipSuccess)
                e = grad_gemm(bf, {Zb, false, M * d2, 1, d2}, {dY2, false, md, d, 1}, wpart,
                              (int32_t)BH, (int32_t)d2, d, M, stream);
            if (e == hipSuccess)
                e = sa::launch_sum_users(wpart, B, H, d2 * d, dW2 + (size_t)l * H * d2 * d, stream);
            if (e == hipSuccess)
                e = grad_gemm(bf, {dY2, false, md, d, 1}, {w.w2(l), bf, d2 * d, 1, d}, Zb,
                              (int32_t)BH, M, (int32_t)d2, d, stream, H);
            // through the gate: dG (over dZ), dU
            if (e == hipSuccess) e = sa::launch_swiglu_bwd(Zb, io.G, io.U, dU, rows * d2, stream);
            // dW1 = sum Xbar^T dG, dW3 = sum Xbar^T dU
            if (e == hipSuccess)
                e = grad_gemm(bf, {io.Xbar, false, md, 1, d}, {Zb, false, M * d2, d2, 1}, wpart,
                              (int32_t)BH, d, (int32_t)d2, M, stream);
            if (e == hipSuccess)
                e = sa::launch_sum_users(wpart, B, H, d * d2, dW1 + (size_t)l * H * d * d2, stream);
            if (e == hipSuccess)
                e = grad_gemm(bf, {io.Xbar, false, md, 1, d}, {dU, false, M * d2, d2, 1}, wpart,
                              (int32_t)BH, d, (int32_t)d2, M, stream);
            if (e == hipSuccess)
                e = sa::launch_sum_users(wpart, B, H, d * d2, dW3 + (size_t)l * H * d * d2, stream);
            // dXbar = dY2 + dG W1^T + dU W3^T (dY2 enters through the norm's second input)
            if (e == hipSuccess)
                e = grad_gemm(bf, {Zb, false, M * d2, d2, 1}, {w.w1(l), bf, d * d2, 1, d2}, dXbar,
                              (int32_t)BH, M, d, (int32_t)d2, stream, H);
            if (e == hipSuccess)
                e = grad_gemm(bf, {dU, false, M * d2, d2, 1}, {w.w3(l), bf, d * d2, 1, d2}, dXbar,
                              (int32_t)BH, M, d, (int32_t)d2, stream, H, true);
            // LN1: dY1 = gradient of Xt + Xhat
            if (e == hipSuccess)
                e = sa::launch_ln_bwd(dXbar, dY2, io.Y1, w.ln_(l, 0), bf, B, H, M, d, eps, dY1, stats, colpart,
                                      plan.nch, dlnl, (int64_t)H * d, stream);
            if (e != hipSuccess) return hip_fail(e, "block refinement backward launch");
        }
        // the sketch (dsketch = dY1, one target instance): dX of this layer (the
        // last layer writes dX, the others add to it) and dP'
        if (T > 0) {
            float* dKs = plan.bshared.fused ? nullptr : F(plan.off_dk);
            float* dVs = plan.bshared.fused ? nullptr : F(plan.off_dv);
            st = run_bwd(X, X, io.Pp, offsets, B, T, H, M, d, scale, dtype, dY1, 1, io.lse, dKs, dVs, dPp, dX,
                         ws + plan.off_base, io.first ? plan.bshared : plan.buser, stream, !io.first,
                         l != n_layers - 1);
            if (st != SA_OK) return st;
        } else {
            e = sa::launch_fill(dPp, nq * md, 0.f, stream);
            if (e != hipSuccess) return hip_fail(e, "fill launch");
        }
        sa::ProfScope ps("block_proj_grads", stream);
        // P' = Q W_K^T, Q = Xt W_Q:  dW_K = sum dP'^T Q, dQ = dP' W_K, dW_Q = sum Xt^T dQ,
        // and the state gradient dXt = dY1 + dQ W_Q^T
        float* dwk = dWk + (size_t)l * H * dd;
        float* dwq = dWq + (size_t)l * H * dd;
        e = grad_gemm(bf, {dPp, false, md, 1, d}, {io.Q, false, md, d, 1}, io.first ? dwk : wpart,
                      (int32_t)nq, d, d, M, stream);
        if (e == hipSuccess && !io.first) e = sa::launch_sum_users(wpart, B, H, dd, dwk, stream);
        if (e == hipSuccess)
            e = grad_gemm(bf, {dPp, false, md, d, 1}, {w.wk(l), bf, dd, d, 1}, dQ, (int32_t)nq, M, d,
                          d, stream, H);
        if (e == hipSuccess)
            e = grad_gemm(bf, {io.xt, io.first && bf, md, 1, d}, {dQ, false, md, d, 1}, io.first ? dwq : wpart,
                          (int32_t)nq, d, d, M, stream);
        if (e == hipSuccess && !io.first) e = sa::launch_sum_users(wpart, B, H, dd, dwq, stream);
        if (e == hipSuccess) {
            if (io.first) {
                // the shared prototypes: dP = sum over users of dY1, plus dQ W_Q^T
                e = sa::launch_sum_users(dY1, B, H, md, dP, stream);
                if (e == hipSuccess)
                    e = grad_gemm(bf, {dQ, false, md, d, 1}, {w.wq(l), bf, dd, 1, d}, dP, H, M, d, d,
                                  stream, H, true);
            } else {
                e = grad_gemm(bf, {dQ, false, md, d, 1}, {w.wq(l), bf, dd, 1, d}, dY1, (int32_t)BH,
                              M, d, d, stream, H, true);
            }
        }
        if (e != hipSuccess) return hip_fail(e, "block projection gradient launch");
        dXt = dY1;
    }
    return SA_OK;
}

size_t sa_stca_fwd_workspace_size(int64_t B, int32_t R, int32_t k, int32_t D, int32_t h, sa_dtype dtype) {
    if (check_stca(B, R, k, D, h, 1.0f, dtype) != SA_OK) return 0;
    return plan_stca(B, R, k, D, h, dtype, false).total;
}

sa_status sa_stca_fwd(const void* Xs, const void* q, const void* Wq, const void* Wk, const void* Wv, int64_t B,
                      int32_t R, int32_t k, int32_t D, int32_t h, float scale, sa_dtype dtype, float* out, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_stca(B, R, k, D, h, scale, dtype);
    if (st != SA_OK) return st;
    if (B == 0) return SA_OK;
    if (!Xs || !q || !Wq || !Wk || !Wv || !out) return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(Xs) || !aligned16(q) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(Wv) || !aligned16(out) ||
        !aligned16(lse))
        return fail(SA_ERR_INVALID_ARG, "tensor arguments must be 16-byte aligned");
    const StcaPlan plan = plan_stca(B, R, k, D, h, dtype, false);
    if (!workspace || workspace_bytes < plan.total)
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                    workspace ? workspace_bytes : (size_t)0);
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    return stca_forward(Xs, q, Wq, Wk, Wv, B, R, k, D, h, scale, dtype, out,
                        lse ? lse : reinterpret_cast<float*>(ws + plan.off_lse), ws, plan,
                        reinterpret_cast<hipStream_t>(stream_));
}

size_t sa_stca_bwd_workspace_size(int64_t B, int32_t R, int32_t k, int32_t D, int32_t h, sa_dtype dtype) {
    if (check_stca(B, R, k, D, h, 1.0f, dtype) != SA_OK) return 0;
    return plan_stca(B, R, k, D, h, dtype, true).total;
}

sa_status sa_stca_bwd(const void* Xs, const void* q, const void* Wq, const void* Wk, const void* Wv, int64_t B,
                      int32_t R, int32_t k, int32_t D, int32_t h, float scale, sa_dtype dtype, const float* dout,
                      float* dXs, float* dq, float* dWq, float* dWk, float* dWv, void* workspace,
                      size_t workspace_bytes, void* stream_) {
    g_last_error[0] = 0;
    sa_status st = check_stca(B, R, k, D, h, scale, dtype);
    if (st != SA_OK) return st;
    if (B < 1) return fail(SA_ERR_INVALID_ARG, "B must be >= 1 for the backward");
    if (!Xs || !q || !Wq || !Wk || !Wv || !dout || !dXs || !dq || !dWq || !dWk || !dWv)
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!aligned16(Xs) || !aligned16(q) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(Wv) || !aligned16(dout) ||
        !aligned16(dXs) || !aligned16(dq) || !aligned16(dWq) || !aligned16(dWk) || !aligned16(dWv))
        return fail(SA_ERR_INVALID_ARG, "tensor arguments must be 16-byte aligned");
    const StcaPlan p = plan_stca(B, R, k, D, h, dtype, true);
    if (!workspace || workspace_bytes < p.total)
        return fail(SA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", p.total,
                    workspace ? workspace_bytes : (size_t)0);
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    float* lse = reinterpret_cast<float*>(ws + p.off_lse);
    // forward replay: Qp, U, S, lse, alpha, C
    st = stca_forward(Xs, q, Wq, Wk, Wv, B, R, k, D, h, scale, dtype, nullptr, lse, ws, p, stream);
    if (st != SA_OK) return st;
    const bool bf = dtype == SA_BF16;
    const int32_t BR = (int32_t)(B * R), dh = D / h, Rh = R * h;
    const int64_t kD = (int64_t)k * D, RhD = (int64_t)Rh * D, Rhk = (int64_t)Rh * k, hD = (int64_t)h * D;
    void* Qp = ws + p.off_qp;
    void* U = ws + p.off_u;
    const void* S = ws + p.off_s;
    void* Al = ws + p.off_al;
    void* Cc = ws + p.off_c;
    void* dC = ws + p.off_dc;
    float* dA = reinterpret_cast<float*>(ws + p.off_da);
    void* ds = ws + p.off_ds;
    void* dU = ws + p.off_du;
    void* dQp = ws + p.off_dqp;
    const void* dob = dout;
    hipError_t e = hipSuccess;
    if (bf) {
        dob = ws + p.off_dob;
        e = sa::launch_to_bf16(dout, reinterpret_cast<uint16_t*>(ws + p.off_dob), (int64_t)BR * D, stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_value_grads", stream);
        // dC[., i] = dout[., head i] W_V^(i)T;  dW_V^(i) = sum over targets of C[., i]^T dout[., head i]
        e = sa::launch_gemm({dob, bf, dh, D, 1, Wv, bf, dh, 1, D, dC, bf, D, hD, BR, D, dh, h, 1.f, false}, stream);
        if (e == hipSuccess)
            e = sa::launch_gemm({Cc, bf, D, 1, hD, dob, bf, dh, D, 1, dWv, false, dh, D, D, dh, BR, h, 1.f, false},
                                stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_dalpha", stream);   // dalpha = dC Xs^T per user
        e = sa::launch_gemm({dC, bf, RhD, D, 1, Xs, bf, kD, 1, D, dA, false, Rhk, k, Rh, k, D, (int32_t)B, 1.f, false},
                            stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_softmax_bwd", stream);
        e = sa::launch_stca_softmax_bwd(S, bf, lse, dA, (int64_t)BR * h, k, scale, bf, ds, stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_sketch_grads", stream);
        // dXs = alpha^T dC + (scale ds)^T U per user;  dU = (scale ds) Xs
        e = sa::launch_gemm({Al, bf, Rhk, 1, k, dC, bf, RhD, D, 1, dXs, false, kD, D, k, D, Rh, (int32_t)B, 1.f, false},
                            stream);
        if (e == hipSuccess)
            e = sa::launch_gemm({ds, bf, Rhk, 1, k, U, bf, RhD, D, 1, dXs, false, kD, D, k, D, Rh, (int32_t)B, 1.f,
                                 true}, stream);
        if (e == hipSuccess)
            e = sa::launch_gemm({ds, bf, Rhk, k, 1, Xs, bf, kD, D, 1, dU, bf, RhD, D, Rh, D, k, (int32_t)B, 1.f, false},
                                stream);
    }
    if (e == hipSuccess) {
        sa::ProfScope ps("stca_query_grads", stream);
        // dQp[., head i] = dU[., i] W_K^(i);  dW_K^(i) = sum dU[., i]^T Qp[., head i]
        e = sa::launch_gemm({dU, bf, D, hD, 1, Wk, bf, dh, D, 1, dQp, bf, dh, D, BR, dh, D, h, 1.f, false}, stream);
        if (e == hipSuccess)
            e = sa::launch_gemm({dU, bf, D, 1, hD, Qp, bf, dh, D, 1, dWk, false, dh, D, D, dh, BR, h, 1.f, false},
                                stream);
        // dq = dQp W_Q^T;  dW_Q = q^T dQp
        if (e == hipSuccess)
            e = sa::launch_gemm({dQp, bf, 0, D, 1, Wq, bf, 0, 1, D, dq, false, 0, D, BR, D, D, 1, 1.f, false}, stream);
        if (e == hipSuccess)
            e = sa::launch_gemm({q, bf, 0, 1, D, dQp, bf, 0, D, 1, dWq, false, 0, D, D, D, BR, 1, 1.f, false}, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "STCA backward launch");
    return SA_OK;
}

void sa_profile_enable(int32_t on) { g_prof_on = on != 0; }

int32_t sa_kernel_times(int32_t max_kernels, char* names, int64_t* launches, double* total_ms) {
    struct Acc {
        const char* name;
        int64_t n;
        double ms;
    };
    std::vector<Acc> acc;
    bool ok = true;
    for (const ProfRec& r : g_prof_recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
            ok = false;
        size_t i = 0;
        while (i < acc.size() && strcmp(acc[i].name, r.name) != 0) ++i;
        if (i == acc.size()) acc.push_back({r.name, 0, 0.0});
        acc[i].n += 1;
        acc[i].ms += ms;
        g_prof_pool.push_back(r.start);
        g_prof_pool.push_back(r.stop);
    }
    g_prof_recs.clear();
    if (!ok) return -1;
    int32_t n = 0;
    for (const Acc& a : acc) {
        if (n >= max_kernels) break;
        if (names) {
            strncpy(names + (size_t)n * 48, a.name, 47);
            names[(size_t)n * 48 + 47] = 0;
        }
        if (launches) launches[n] = a.n;
        if (total_ms) total_ms[n] = a.ms;
        ++n;
    }
    return n;
}

sa_status sa_build_worklist(const int64_t* offsets, int64_t B, int64_t T, int32_t H,
                            int64_t chunk_tokens, int32_t* items, int64_t max_items,
                            int64_t* n_items, void* stream_) {
    g_last_error[0] = 0;
    if (B < 0 || T < 0 || H < 1 || chunk_tokens < 1 || max_items < 0)
        return fail(SA_ERR_INVALID_ARG, "bad sizes");
    if (!offsets || !n_items || (max_items > 0 && !items))
        return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (T >= (int64_t(1) << 31) || (int64_t)H * B >= (int64_t(1) << 31))
        return fail(SA_ERR_UNSUPPORTED, "sizes beyond int32 indexing");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const int64_t n_ranges = ((int64_t)H * T + chunk_tokens - 1) / chunk_tokens;
    hipError_t e = sa::launch_worklist(offsets, B, T, H, chunk_tokens, n_ranges, items, max_items,
                                       nullptr, nullptr, n_items, stream);
    if (e != hipSuccess) return hip_fail(e, "work list launch");
    return SA_OK;
}

int32_t sa_gemm_tile_shapes(void) { return sa::gemm_tile_shapes(); }

sa_status sa_gemm_bf16(const void* A, int64_t a_z, int64_t a_m, int64_t a_k, const void* B, int64_t b_z,
                       int64_t b_k, int64_t b_n, int64_t b_mod, void* C, int32_t c_bf16, int64_t c_z, int64_t c_m,
                       int32_t M, int32_t N, int32_t K, int32_t batch, float alpha, int32_t accumulate,
                       int32_t tile_shape, void* stream_) {
    g_last_error[0] = 0;
    if (M < 0 || N < 0 || K < 1 || batch < 0 || b_mod < 0 || tile_shape >= sa::gemm_tile_shapes())
        return fail(SA_ERR_INVALID_ARG, "bad sizes or tile shape");
    if (M == 0 || N == 0 || batch == 0) return SA_OK;
    if (!A || !B || !C) return fail(SA_ERR_INVALID_ARG, "null pointer argument");
    if (!std::isfinite(alpha)) return fail(SA_ERR_INVALID_ARG, "alpha must be finite");
    sa::GemmDesc d{A, true, a_z, a_m, a_k, B, true, b_z, b_k, b_n, C, c_bf16 != 0, c_z, c_m,
                   M, N, K, batch, alpha, accumulate != 0, b_mod, false};
    if (tile_shape >= 0 && !sa::gemm_on_matrix_cores(d))
        return fail(SA_ERR_UNSUPPORTED, "this product does not run on the matrix cores (layout, alignment or K)");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    const hipError_t e = sa::launch_gemm_tile_shape(d, tile_shape, stream);
    if (e == hipErrorInvalidValue) return fail(SA_ERR_UNSUPPORTED, "tile shape %d cannot take this product", tile_shape);
    if (e != hipSuccess) return hip_fail(e, "product launch");
    return SA_OK;
}

}  // extern "C"

/*
 * Plain CPU oracle of the Sketch Attention (SA) sketching step, in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  It is called by the tests, by the smoke check and
 * by the benchmark's CPU-baseline leg, never by the library: the GPU path does
 * not link, load or call anything here, and nothing here is shared with it.
 *
 * What it computes (SequenceO1, section 3.1 "Sketch Attention", Eqs. for S, A
 * and the sketch; Appendix B steps 1-3; Appendix G.3 with Q = P W_Q, K = X W_K):
 *
 *   for every user b, head h, token t in [offsets[b], offsets[b+1]):
 *     s_m    = scale * sum_j K[t,h,j] * P[h,m,j]             (affinities, m < M)
 *     a_m    = exp(s_m) / sum_m' exp(s_m')                     (prototype-wise softmax;
 *                                                               normalised over m, per token)
 *     sketch[b,h,m,:] += a_m * V[t,h,:]                        (sketch = A X)
 *     lse[t,h] = log sum_m exp(s_m)                             (softmax statistic, section 4.4)
 *
 * The softmax is evaluated in the usual stable form exp(s_m - mu)/z with
 * mu = max_m s_m and z = sum_m exp(s_m - mu); lse = mu + log z.  Everything is
 * fp64 on the exact fp32 values of the inputs (bf16 inputs are upcast exactly
 * by the caller).  The sum over tokens runs in token order.
 *
 * Backward (the paper states the sketch is differentiable and trained end to
 * end but prints no gradients; these follow from the forward by the chain rule):
 *   dY       = sum_r dsketch[b,r,h]                (a user's sketch reused by R targets,
 *                                                   section 4.2 MRLB: gradients add)
 *   dV[t,h]  = sum_m a_m dY_m
 *   g_m      = V[t,h] . dY_m
 *   dS_m     = a_m (g_m - sum_m' a_m' g_m')        (softmax Jacobian)
 *   dK[t,h]  = scale * sum_m dS_m P[h,m]
 *   dP[h,m] += scale * dS_m K[t,h]                 (P is shared by all users: summed over
 *                                                   every user and token of the call)
 *
 * Heads are independent SA instances, each with its own P[h] (the paper's SA is
 * single-head; H = 1 is exactly the paper).  An empty user (L_b = 0) has a zero
 * sketch.
 *
 * Token-wise ("vanilla") normalisation, the alternative the paper compares SA
 * against (Appendix "Why prototype-wise normalization"; Table 1 baseline):
 * the weights are normalised over the tokens of a user for each prototype,
 * p(i | j) instead of p(j | i):
 *   for every user b, head h, prototype m:
 *     s_t        = scale * K[t,h] . P[h,m]            (t over the user's tokens)
 *     w_t        = exp(s_t) / sum_t' exp(s_t')
 *     sketch[b,h,m,:] = sum_t w_t V[t,h,:]
 *     lse_m[b,h,m]    = log sum_t exp(s_t)              (-inf for an empty user)
 * evaluated in two passes: the maximum over tokens, then the shifted sums.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL 1
#define ORACLE_ENOMEM 2

static int check_offsets(const int64_t* offsets, int64_t B) {
    if (offsets[0] != 0) return ORACLE_EINVAL;
    for (int64_t b = 0; b < B; ++b)
        if (offsets[b + 1] < offsets[b]) return ORACLE_EINVAL;
    return ORACLE_OK;
}

static void set_threads(int32_t nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int sa_oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Logits of one token against all prototypes of head h: s[m], m < M. */
static void logits(const float* Kt, const float* Ph, int32_t M, int32_t d,
                   double scale, double* s) {
    for (int32_t m = 0; m < M; ++m) {
        const float* p = Ph + (int64_t)m * d;
        double acc = 0.0;
        for (int32_t j = 0; j < d; ++j) acc += (double)Kt[j] * (double)p[j];
        s[m] = scale * acc;
    }
}

/* Prototype-wise softmax of s[0..M) into a[], returns log sum_m exp(s_m). */
static double softmax_proto(const double* s, int32_t M, double* a) {
    double mu = s[0];
    for (int32_t m = 1; m < M; ++m)
        if (s[m] > mu) mu = s[m];
    double z = 0.0;
    for (int32_t m = 0; m < M; ++m) {
        a[m] = exp(s[m] - mu);
        z += a[m];
    }
    for (int32_t m = 0; m < M; ++m) a[m] /= z;
    return mu + log(z);
}

/*
 * Allocation weights A[t,h,m] for every token (no users needed): used by the
 * tests that check the per-token conservation sum_m A = 1.
 */
int sa_oracle_weights(const float* K, const float* P, int64_t T, int32_t H,
                      int32_t M, int32_t d, double scale, double* A, double* lse) {
    if (T < 0 || H < 1 || M < 1 || d < 1) return ORACLE_EINVAL;
    double* s = (double*)malloc(sizeof(double) * (size_t)M);
    if (!s) return ORACLE_ENOMEM;
    for (int64_t t = 0; t < T; ++t)
        for (int32_t h = 0; h < H; ++h) {
            logits(K + (t * H + h) * (int64_t)d, P + (int64_t)h * M * d, M, d, scale, s);
            double l = softmax_proto(s, M, A + (t * H + h) * (int64_t)M);
            if (lse) lse[t * H + h] = l;
        }
    free(s);
    return ORACLE_OK;
}

/*
 * Forward.  sketch: [B,H,M,d] (overwritten); lse: [T,H] or NULL.
 * nthreads <= 0 keeps the OpenMP default.
 */
int sa_oracle_fwd(const float* K, const float* V, const float* P,
                  const int64_t* offsets, int64_t B, int32_t H, int32_t M,
                  int32_t d, double scale, double* sketch, double* lse,
                  int32_t nthreads) {
    if (B < 0 || H < 1 || M < 1 || d < 1) return ORACLE_EINVAL;
    if (check_offsets(offsets, B)) return ORACLE_EINVAL;
    set_threads(nthreads);
    const int64_t npairs = B * (int64_t)H;
    int err = ORACLE_OK;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)M);
        double* a = (double*)malloc(sizeof(double) * (size_t)M);
        if (!s || !a) {
#pragma omp atomic write
            err = ORACLE_ENOMEM;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t p = 0; p < npairs; ++p) {
            if (!s || !a) continue;
            const int64_t b = p / H;
            const int32_t h = (int32_t)(p % H);
            const float* Ph = P + (int64_t)h * M * d;
            double* out = sketch + p * (int64_t)M * d; /* [b][h] block */
            memset(out, 0, sizeof(double) * (size_t)M * (size_t)d);
            for (int64_t t = offsets[b]; t < offsets[b + 1]; ++t) {
                const float* Kt = K + (t * H + h) * (int64_t)d;
                const float* Vt = V + (t * H + h) * (int64_t)d;
                logits(Kt, Ph, M, d, scale, s);
                double l = softmax_proto(s, M, a);
                if (lse) lse[t * H + h] = l;
                for (int32_t m = 0; m < M; ++m) {
                    double* row = out + (int64_t)m * d;
                    const double am = a[m];
                    for (int32_t j = 0; j < d; ++j) row[j] += am * (double)Vt[j];
                }
            }
        }
        free(s);
        free(a);
    }
    return err;
}

/*
 * Token-wise normalised forward.  sketch: [B,H,M,d] (overwritten); lse_m:
 * [B,H,M] or NULL.  Two passes over the user's tokens per (user, head): the
 * per-prototype maximum of the logits, then exp(s - max) summed into the
 * normaliser and, weighted, into the sketch rows.
 */
int sa_oracle_fwd_tokenwise(const float* K, const float* V, const float* P,
                            const int64_t* offsets, int64_t B, int32_t H, int32_t M,
                            int32_t d, double scale, double* sketch, double* lse_m,
                            int32_t nthreads) {
    if (B < 0 || H < 1 || M < 1 || d < 1) return ORACLE_EINVAL;
    if (check_offsets(offsets, B)) return ORACLE_EINVAL;
    set_threads(nthreads);
    const int64_t npairs = B * (int64_t)H;
    int err = ORACLE_OK;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)M);
        double* mu = (double*)malloc(sizeof(double) * (size_t)M);
        double* z = (double*)malloc(sizeof(double) * (size_t)M);
        if (!s || !mu || !z) {
#pragma omp atomic write
            err = ORACLE_ENOMEM;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t p = 0; p < npairs; ++p) {
            if (!s || !mu || !z) continue;
            const int64_t b = p / H;
            const int32_t h = (int32_t)(p % H);
            const float* Ph = P + (int64_t)h * M * d;
            double* out = sketch + p * (int64_t)M * d;
            memset(out, 0, sizeof(double) * (size_t)M * (size_t)d);
            for (int32_t m = 0; m < M; ++m) {
                mu[m] = -INFINITY;
                z[m] = 0.0;
            }
            /* pass 1: max over the user's tokens, per prototype */
            for (int64_t t = offsets[b]; t < offsets[b + 1]; ++t) {
                logits(K + (t * H + h) * (int64_t)d, Ph, M, d, scale, s);
                for (int32_t m = 0; m < M; ++m)
                    if (s[m] > mu[m]) mu[m] = s[m];
            }
            /* pass 2: shifted exponentials into the normaliser and the sketch */
            for (int64_t t = offsets[b]; t < offsets[b + 1]; ++t) {
                const float* Vt = V + (t * H + h) * (int64_t)d;
                logits(K + (t * H + h) * (int64_t)d, Ph, M, d, scale, s);
                for (int32_t m = 0; m < M; ++m) {
                    const double e = exp(s[m] - mu[m]);
                    z[m] += e;
                    double* row = out + (int64_t)m * d;
                    for (int32_t j = 0; j < d; ++j) row[j] += e * (double)Vt[j];
                }
            }
            for (int32_t m = 0; m < M; ++m) {
                if (z[m] > 0.0) {
                    double* row = out + (int64_t)m * d;
                    for (int32_t j = 0; j < d; ++j) row[j] /= z[m];
                }
                if (lse_m) lse_m[p * M + m] = z[m] > 0.0 ? mu[m] + log(z[m]) : -INFINITY;
            }
        }
        free(s);
        free(mu);
        free(z);
    }
    return err;
}

/*
 * Backward.  dsketch: [B,R,H,M,d]; dK, dV: [T,H,d]; dP: [H,M,d] (all
 * overwritten).  The per-user contributions to dP are added in user order.
 */
int sa_oracle_bwd(const float* K, const float* V, const float* P,
                  const int64_t* offsets, int64_t B, int32_t H, int32_t M,
                  int32_t d, double scale, const float* dsketch, int32_t R,
                  double* dK, double* dV, double* dP, int32_t nthreads) {
    if (B < 0 || H < 1 || M < 1 || d < 1 || R < 1) return ORACLE_EINVAL;
    if (check_offsets(offsets, B)) return ORACLE_EINVAL;
    set_threads(nthreads);
    const int64_t npairs = B * (int64_t)H;
    const size_t md = (size_t)M * (size_t)d;
    double* dP_user = (double*)calloc(npairs ? (size_t)npairs * md : 1, sizeof(double));
    if (!dP_user) return ORACLE_ENOMEM;
    int err = ORACLE_OK;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)M);
        double* a = (double*)malloc(sizeof(double) * (size_t)M);
        double* g = (double*)malloc(sizeof(double) * (size_t)M);
        double* dY = (double*)malloc(sizeof(double) * md);
        if (!s || !a || !g || !dY) {
#pragma omp atomic write
            err = ORACLE_ENOMEM;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t p = 0; p < npairs; ++p) {
            if (!s || !a || !g || !dY) continue;
            const int64_t b = p / H;
            const int32_t h = (int32_t)(p % H);
            const float* Ph = P + (int64_t)h * M * d;
            double* dPp = dP_user + p * (int64_t)md;
            /* dY = sum over the R target instances that reused this sketch */
            for (size_t i = 0; i < md; ++i) dY[i] = 0.0;
            for (int32_t r = 0; r < R; ++r) {
                const float* src = dsketch + (((b * R + r) * H + h) * (int64_t)md);
                for (size_t i = 0; i < md; ++i) dY[i] += (double)src[i];
            }
            for (int64_t t = offsets[b]; t < offsets[b + 1]; ++t) {
                const float* Kt = K + (t * H + h) * (int64_t)d;
                const float* Vt = V + (t * H + h) * (int64_t)d;
                double* dKt = dK + (t * H + h) * (int64_t)d;
                double* dVt = dV + (t * H + h) * (int64_t)d;
                logits(Kt, Ph, M, d, scale, s);
                softmax_proto(s, M, a);
                /* dV_t = sum_m a_m dY_m ; g_m = V_t . dY_m */
                for (int32_t j = 0; j < d; ++j) dVt[j] = 0.0;
                double D = 0.0;
                for (int32_t m = 0; m < M; ++m) {
                    const double* y = dY + (int64_t)m * d;
                    double gm = 0.0;
                    for (int32_t j = 0; j < d; ++j) {
                        dVt[j] += a[m] * y[j];
                        gm += (double)Vt[j] * y[j];
                    }
                    g[m] = gm;
                    D += a[m] * gm;
                }
                /* dS_m = a_m (g_m - D); dK_t = scale sum_m dS_m P_m; dP_m += scale dS_m K_t */
                for (int32_t j = 0; j < d; ++j) dKt[j] = 0.0;
                for (int32_t m = 0; m < M; ++m) {
                    const double dS = a[m] * (g[m] - D);
                    const float* pm = Ph + (int64_t)m * d;
                    double* dpm = dPp + (int64_t)m * d;
                    for (int32_t j = 0; j < d; ++j) {
                        dKt[j] += scale * dS * (double)pm[j];
                        dpm[j] += scale * dS * (double)Kt[j];
                    }
                }
            }
        }
        free(s);
        free(a);
        free(g);
        free(dY);
    }
    if (err == ORACLE_OK) {
        for (int32_t h = 0; h < H; ++h) {
            double* out = dP + (int64_t)h * md;
            for (size_t i = 0; i < md; ++i) out[i] = 0.0;
            for (int64_t b = 0; b < B; ++b) {
                const double* src = dP_user + (b * H + h) * (int64_t)md;
                for (size_t i = 0; i < md; ++i) out[i] += src[i];
            }
        }
    }
    free(dP_user);
    return err;
}

/*
 * Multi-Head LatentMoE CPU oracle — TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain, slow, obviously-correct definition of what the
 * per-GPU hot path computes.  It exists so that tests, the smoke check and
 * the benchmark's CPU-baseline leg can check the HIP library against it.
 * Nothing on the product path may link, load or call it, and it shares no
 * code, header, table or helper with the HIP library.
 *
 * Paper: "Multi-Head LatentMoE" (arXiv 2602.04870).
 *   - Eq. (1)-(4), Sec. 2.2: Mixtral-style MoE, top-k softmax gate, linear
 *     router.
 *   - Sec. 2.2 / App. A: the router computes in FP32.
 *   - Eq. (5)-(6), Sec. 3.1: each head h is an independent MoE applied to the
 *     d_h-wide slice of the latent token.
 *   - Algorithm 1 / Sec. 3.3: bias added before top-k and removed after, so it
 *     steers selection but never the scores.
 *   - Algorithm 2 / Sec. 3.3: routing backward, gradients only for the k
 *     selected experts.
 *   - Sec. 3.4: token clustering (experts' tokens contiguous), dropless.
 *
 * Because the paper states its routing and expert computation are exact, this
 * oracle computes the plain definitions (dense logits, full sort, per-slot
 * expert evaluation) and never the blocked algorithms.
 *
 * Precision:
 *   - router logits: fp64 dot product of the given values, then rounded to
 *     fp32 (the paper fixes the router at FP32); the selection key
 *     s + b is formed in fp32 and the top-k decision is taken on fp32 keys,
 *     ties broken toward the lower expert index.
 *   - everything else (softmax gates, expert FFN, combine, backward): fp64.
 *
 * Expert FFN: SwiGLU, y = W2 (silu(W1 x) * (W3 x)), with W1 = gate proj,
 * W3 = up proj, W2 = down proj (Mixtral convention, which Sec. 2.2 follows).
 * The paper's own experiments use a two-matrix GELU expert (Sec. 3.4),
 * y = W_out gelu(W_in x) with the exact gelu(z) = z Phi(z); the *_gelu
 * entry points compute that form (W_in in W1's layout, W_out in W2's).
 *
 * Load balancing (Sec. 2.2): auxiliary-loss-free, i.e. the routing bias b
 * of Algorithm 1 is nudged after a batch by a fixed rate toward equal load,
 * b[h][e] += rate * sign(mean_e counts[h] - counts[h][e]) (the rule of the
 * aux-free method the paper adopts), computed in fp32 like the bias itself.
 *
 * Layouts (row-major):
 *   X        [T][Nh][dh]            W_router [Nh][Ne][dh]   bias [Nh][Ne]
 *   idx      [T][Nh][k] (int32)     gate     [T][Nh][k]     counts [Nh][Ne]
 *   offsets  [Nh][Ne+1]             perm     [Nh][T*k]  (slot id = t*k + j)
 *   W1, W3   [Nh][Ne][dff][dh]      W2       [Nh][Ne][dh][dff]
 *   Y, dY, dX [T][Nh][dh]
 *
 * Parity pins: see tests/test_oracle_pins.py (brute force, closed forms,
 * invariants, finite differences) and tests/test_oracle_mutants.py (planted
 * mistakes in this file must fail a pin).
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
#define ORACLE_ENAN 2
#define ORACLE_ENOMEM 3

/* Threads the oracle's parallel loops use (1 without OpenMP). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Router: Eq. (4) s = r(x), in FP32 (Sec. 2.2).                             */
/* ------------------------------------------------------------------------ */

/* s[e] = fl32( sum_i x[i] * w[e][i] ), the fp64 dot rounded once to fp32. */
static void router_logits(int dh, int Ne, const double *x, const double *w,
                          float *s)
{
    for (int e = 0; e < Ne; ++e) {
        double acc = 0.0;
        for (int i = 0; i < dh; ++i)
            acc += x[i] * w[(int64_t)e * dh + i];
        s[e] = (float)acc;
    }
}

/* Ordering used by the top-k of Eq. (3) with Algorithm 1's biased key:
 * larger key first; equal keys -> lower expert index first. */
typedef struct {
    float key;
    int e;
} key_entry;

static int key_desc_then_index(const void *pa, const void *pb)
{
    const key_entry *a = (const key_entry *)pa;
    const key_entry *b = (const key_entry *)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->e > b->e) - (a->e < b->e);
}

/*
 * Routing forward: Eq. (2)-(4) plus Algorithm 1's load-balancing bias.
 *
 *   key[e]  = fl32(s[e] + b[h][e])       (bias only steers the selection)
 *   idx     = the k experts with largest key, in descending key order
 *   gate[j] = exp(s[idx_j]) / sum_j' exp(s[idx_j'])   (unbiased scores)
 *   counts[h][e] = number of (t, j) with idx[t][h][j] == e
 *
 * Optional outputs:
 *   keys_sorted [T][Nh][nk], nk = min(k+1, Ne): the leading fp32 keys in
 *               selection order (used by tests for the near-tie rule);
 *   s_top       [T][Nh][k]: the unbiased fp32 scores of the selection.
 */
int oracle_route(int64_t T, int Nh, int dh, int Ne, int k,
                 const double *X, const double *W_router, const double *bias,
                 int32_t *idx, double *gate, int32_t *counts,
                 float *keys_sorted, float *s_top)
{
    if (T < 0 || Nh <= 0 || dh <= 0 || Ne <= 0 || k <= 0 || k > Ne)
        return ORACLE_EINVAL;
    const int nk = (k + 1 < Ne) ? k + 1 : Ne;
    int status = ORACLE_OK;

#pragma omp parallel
    {
        float *s = (float *)malloc(sizeof(float) * (size_t)Ne);
        key_entry *ent = (key_entry *)malloc(sizeof(key_entry) * (size_t)Ne);
        if (!s || !ent) {
#pragma omp atomic write
            status = ORACLE_ENOMEM;
        } else {
#pragma omp for schedule(static)
            for (int64_t th = 0; th < T * Nh; ++th) {
                const int64_t t = th / Nh;
                const int h = (int)(th % Nh);
                const double *x = X + (t * Nh + h) * (int64_t)dh;
                const double *w = W_router + (int64_t)h * Ne * dh;
                router_logits(dh, Ne, x, w, s);
                for (int e = 0; e < Ne; ++e) {
                    float key = s[e];
                    if (bias) key = s[e] + (float)bias[(int64_t)h * Ne + e];
                    if (isnan(key)) {
#pragma omp atomic write
                        status = ORACLE_ENAN;
                    }
                    ent[e].key = key;
                    ent[e].e = e;
                }
                qsort(ent, (size_t)Ne, sizeof(key_entry), key_desc_then_index);

                int32_t *id = idx + th * k;
                for (int j = 0; j < k; ++j) id[j] = ent[j].e;

                double m = -INFINITY;
                for (int j = 0; j < k; ++j)
                    if ((double)s[id[j]] > m) m = (double)s[id[j]];
                double z = 0.0;
                for (int j = 0; j < k; ++j) z += exp((double)s[id[j]] - m);
                for (int j = 0; j < k; ++j)
                    gate[th * k + j] = exp((double)s[id[j]] - m) / z;

                if (keys_sorted)
                    for (int j = 0; j < nk; ++j)
                        keys_sorted[th * nk + j] = ent[j].key;
                if (s_top)
                    for (int j = 0; j < k; ++j) s_top[th * k + j] = s[id[j]];
            }
        }
        free(s);
        free(ent);
    }
    if (status != ORACLE_OK) return status;

    if (counts) {
        memset(counts, 0, sizeof(int32_t) * (size_t)Nh * (size_t)Ne);
        for (int64_t t = 0; t < T; ++t)
            for (int h = 0; h < Nh; ++h)
                for (int j = 0; j < k; ++j)
                    counts[(int64_t)h * Ne + idx[(t * Nh + h) * k + j]] += 1;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Token clustering (Sec. 3.4, Fig. 2): a stable counting sort by expert.    */
/* ------------------------------------------------------------------------ */

/*
 * offsets[h][e] = sum_{e' < e} counts[h][e'], offsets[h][Ne] = T*k.
 * perm[h][offsets[h][e] + r] = the r-th slot id (t*k + j), in ascending
 * (t, j) order, whose expert in head h is e.
 */
int oracle_bucket(int64_t T, int Nh, int Ne, int k, const int32_t *idx,
                  int32_t *offsets, int32_t *perm)
{
    if (T < 0 || Nh <= 0 || Ne <= 0 || k <= 0) return ORACLE_EINVAL;
    const int64_t slots = T * k;
    int64_t *cursor = (int64_t *)malloc(sizeof(int64_t) * (size_t)(Ne + 1));
    if (!cursor) return ORACLE_ENOMEM;
    int status = ORACLE_OK;
    for (int h = 0; h < Nh && status == ORACLE_OK; ++h) {
        for (int e = 0; e <= Ne; ++e) cursor[e] = 0;
        for (int64_t t = 0; t < T; ++t)
            for (int j = 0; j < k; ++j) {
                int e = idx[(t * Nh + h) * k + j];
                if (e < 0 || e >= Ne) { status = ORACLE_EINVAL; break; }
                cursor[e + 1] += 1;
            }
        if (status != ORACLE_OK) break;
        for (int e = 0; e < Ne; ++e) cursor[e + 1] += cursor[e];
        for (int e = 0; e <= Ne; ++e)
            offsets[(int64_t)h * (Ne + 1) + e] = (int32_t)cursor[e];
        for (int64_t t = 0; t < T; ++t)
            for (int j = 0; j < k; ++j) {
                int e = idx[(t * Nh + h) * k + j];
                perm[(int64_t)h * slots + cursor[e]] = (int32_t)(t * k + j);
                cursor[e] += 1;
            }
    }
    free(cursor);
    return status;
}

/* ------------------------------------------------------------------------ */
/* Expert FFN (SwiGLU) and the gate-weighted combine, Eq. (1).               */
/* ------------------------------------------------------------------------ */

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* y = W2 (silu(W1 x) * (W3 x)); also returns a = W1 x, b = W3 x, u. */
static void swiglu_expert(int dh, int dff, const double *x, const double *w1,
                          const double *w3, const double *w2, double *a,
                          double *b, double *u, double *y)
{
    for (int f = 0; f < dff; ++f) {
        double sa = 0.0, sb = 0.0;
        for (int i = 0; i < dh; ++i) {
            sa += w1[(int64_t)f * dh + i] * x[i];
            sb += w3[(int64_t)f * dh + i] * x[i];
        }
        a[f] = sa;
        b[f] = sb;
        u[f] = silu(sa) * sb;
    }
    for (int i = 0; i < dh; ++i) {
        double acc = 0.0;
        for (int f = 0; f < dff; ++f) acc += w2[(int64_t)i * dff + f] * u[f];
        y[i] = acc;
    }
}

/* GELU with the Gaussian CDF written through erf: z Phi(z). */
static double gelu(double z) { return 0.5 * z * (1.0 + erf(z / sqrt(2.0))); }

/* d/dz [z Phi(z)] = Phi(z) + z phi(z), phi the standard normal density. */
static double gelu_grad(double z)
{
    const double pi = 3.14159265358979323846;
    return 0.5 * (1.0 + erf(z / sqrt(2.0))) + z * exp(-0.5 * z * z) / sqrt(2.0 * pi);
}

/* y = W_out gelu(W_in x) (Sec. 3.4's expert); also returns u = gelu(W_in x)
 * and (a non-NULL) a = W_in x. */
static void gelu_expert(int dh, int dff, const double *x, const double *w_in,
                        const double *w_out, double *a, double *u, double *y)
{
    for (int f = 0; f < dff; ++f) {
        double s = 0.0;
        for (int i = 0; i < dh; ++i) s += w_in[(int64_t)f * dh + i] * x[i];
        if (a) a[f] = s;
        u[f] = gelu(s);
    }
    for (int i = 0; i < dh; ++i) {
        double acc = 0.0;
        for (int f = 0; f < dff; ++f) acc += w_out[(int64_t)i * dff + f] * u[f];
        y[i] = acc;
    }
}

static int experts_impl(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                        const double *X, const int32_t *idx, const double *gate,
                        const double *W1, const double *W3, const double *W2,
                        double *Y, double *ys);

/*
 * Y[t][h] = sum_{j=0}^{k-1} gate[t][h][j] * E_{h, idx[t][h][j]}(x_{t,h}),
 * Eq. (1) restricted to the k experts with non-zero gate, summed in j order;
 * the per-head outputs sit side by side, which is Eq. (6)'s concat.
 * ys (optional) [T][Nh][k][dh] receives the unscaled expert outputs.
 */
int oracle_experts(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                   const double *X, const int32_t *idx, const double *gate,
                   const double *W1, const double *W3, const double *W2,
                   double *Y, double *ys)
{
    if (W3 == NULL) return ORACLE_EINVAL;
    return experts_impl(T, Nh, dh, Ne, k, dff, X, idx, gate, W1, W3, W2, Y, ys);
}

/* The same with the two-matrix GELU expert: W_in [Nh][Ne][dff][dh],
 * W_out [Nh][Ne][dh][dff]. */
int oracle_experts_gelu(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                        const double *X, const int32_t *idx, const double *gate,
                        const double *W_in, const double *W_out, double *Y,
                        double *ys)
{
    return experts_impl(T, Nh, dh, Ne, k, dff, X, idx, gate, W_in, NULL, W_out,
                        Y, ys);
}

/* W3 == NULL selects the GELU expert (W1 = W_in, W2 = W_out). */
static int experts_impl(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                        const double *X, const int32_t *idx, const double *gate,
                        const double *W1, const double *W3, const double *W2,
                        double *Y, double *ys)
{
    if (T < 0 || Nh <= 0 || dh <= 0 || Ne <= 0 || k <= 0 || dff <= 0)
        return ORACLE_EINVAL;
    int status = ORACLE_OK;
#pragma omp parallel
    {
        double *a = (double *)malloc(sizeof(double) * (size_t)dff);
        double *b = (double *)malloc(sizeof(double) * (size_t)dff);
        double *u = (double *)malloc(sizeof(double) * (size_t)dff);
        double *y = (double *)malloc(sizeof(double) * (size_t)dh);
        if (!a || !b || !u || !y) {
#pragma omp atomic write
            status = ORACLE_ENOMEM;
        } else {
#pragma omp for schedule(static)
            for (int64_t th = 0; th < T * Nh; ++th) {
                const int h = (int)(th % Nh);
                const double *x = X + th * dh;
                double *out = Y + th * dh;
                for (int i = 0; i < dh; ++i) out[i] = 0.0;
                for (int j = 0; j < k; ++j) {
                    const int e = idx[th * k + j];
                    if (e < 0 || e >= Ne) {
#pragma omp atomic write
                        status = ORACLE_EINVAL;
                        continue;
                    }
                    const int64_t he = (int64_t)h * Ne + e;
                    if (W3)
                        swiglu_expert(dh, dff, x, W1 + he * dff * dh,
                                      W3 + he * dff * dh, W2 + he * dh * dff, a,
                                      b, u, y);
                    else
                        gelu_expert(dh, dff, x, W1 + he * dff * dh,
                                    W2 + he * dh * dff, NULL, u, y);
                    const double g = gate[th * k + j];
                    for (int i = 0; i < dh; ++i) out[i] += g * y[i];
                    if (ys)
                        for (int i = 0; i < dh; ++i)
                            ys[(th * k + j) * dh + i] = y[i];
                }
            }
        }
        free(a);
        free(b);
        free(u);
        free(y);
    }
    return status;
}

/* The whole per-GPU layer: routing forward, then the experts and combine. */
int oracle_layer(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                 const double *X, const double *W_router, const double *bias,
                 const double *W1, const double *W3, const double *W2,
                 double *Y, int32_t *idx, double *gate, int32_t *counts)
{
    int st = oracle_route(T, Nh, dh, Ne, k, X, W_router, bias, idx, gate,
                          counts, NULL, NULL);
    if (st != ORACLE_OK) return st;
    return oracle_experts(T, Nh, dh, Ne, k, dff, X, idx, gate, W1, W3, W2, Y,
                          NULL);
}

/* The layer with the two-matrix GELU expert. */
int oracle_layer_gelu(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                      const double *X, const double *W_router,
                      const double *bias, const double *W_in,
                      const double *W_out, double *Y, int32_t *idx,
                      double *gate, int32_t *counts)
{
    int st = oracle_route(T, Nh, dh, Ne, k, X, W_router, bias, idx, gate,
                          counts, NULL, NULL);
    if (st != ORACLE_OK) return st;
    return oracle_experts_gelu(T, Nh, dh, Ne, k, dff, X, idx, gate, W_in,
                               W_out, Y, NULL);
}

/* Auxiliary-loss-free bias update (Sec. 2.2).  Each head is its own MoE:
 * with S = sum_e counts[h][e], expert e is under-loaded when
 * counts[h][e] < S / Ne, i.e. counts[h][e] * Ne < S (decided exactly in
 * integers), and its bias rises by rate; over-loaded experts drop by rate;
 * exactly balanced ones keep their bias.  The sum is one fp32 addition. */
int oracle_bias_update(int Nh, int Ne, const int32_t *counts, float rate,
                       float *bias)
{
    if (Nh <= 0 || Ne <= 0) return ORACLE_EINVAL;
    for (int h = 0; h < Nh; ++h) {
        int64_t S = 0;
        for (int e = 0; e < Ne; ++e) S += counts[(int64_t)h * Ne + e];
        for (int e = 0; e < Ne; ++e) {
            const int64_t c = counts[(int64_t)h * Ne + e];
            const int64_t d = S - c * Ne;  /* sign of mean - c */
            float *b = &bias[(int64_t)h * Ne + e];
            if (d > 0) *b = *b + rate;
            else if (d < 0) *b = *b - rate;
        }
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Backward: Algorithm 2 (router) and the gradient of Eq. (1)-(3) with the  */
/* SwiGLU expert.  No gradient flows through the selection or to the bias.   */
/* ------------------------------------------------------------------------ */

/*
 * Algorithm 2 on its own (Sec. 3.3): given the forward's idx and gate and the
 * gradient dgate [T][Nh][k] of a loss with respect to the gates,
 *   dS_j = g_j (dgate_j - sum_j' g_j' dgate_j')   (softmax over the k scores)
 *   dX[t][h] = sum_j dS_j W_router[h][e_j]
 *   dW_router[h][e] = sum over the (t, j) with e_j = e of dS_j x_{t,h}
 * The bias gets no gradient and neither does the selection.  dW_router is
 * overwritten; heads run in parallel, tokens in ascending order.  dS
 * (optional) [T][Nh][k] receives the score gradients.
 */
int oracle_route_backward(int64_t T, int Nh, int dh, int Ne, int k,
                          const double *X, const double *W_router,
                          const int32_t *idx, const double *gate,
                          const double *dgate, double *dX, double *dW_router,
                          double *dS)
{
    if (T < 0 || Nh <= 0 || dh <= 0 || Ne <= 0 || k <= 0) return ORACLE_EINVAL;
    memset(dW_router, 0, sizeof(double) * (size_t)Nh * Ne * dh);
    int status = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int h = 0; h < Nh; ++h) {
        for (int64_t t = 0; t < T; ++t) {
            const int64_t th = t * Nh + h;
            const int32_t *id = idx + th * k;
            const double *g = gate + th * k;
            const double *dg = dgate + th * k;
            const double *x = X + th * dh;
            double *dx = dX + th * dh;
            int bad = 0;
            for (int j = 0; j < k; ++j)
                if (id[j] < 0 || id[j] >= Ne) bad = 1;
            if (bad) {
#pragma omp atomic write
                status = ORACLE_EINVAL;
                break;
            }
            double gdg = 0.0;
            for (int j = 0; j < k; ++j) gdg += g[j] * dg[j];
            for (int i = 0; i < dh; ++i) dx[i] = 0.0;
            for (int j = 0; j < k; ++j) {
                const double ds = g[j] * (dg[j] - gdg);
                if (dS) dS[th * k + j] = ds;
                const int64_t he = (int64_t)h * Ne + id[j];
                const double *wr = W_router + he * dh;
                double *dwr = dW_router + he * dh;
                for (int i = 0; i < dh; ++i) {
                    dx[i] += ds * wr[i];
                    dwr[i] += ds * x[i];
                }
            }
        }
    }
    return status;
}

/*
 * Given the forward's saved idx and gate and the output gradient dY:
 *   y_j   = E_{e_j}(x)                      (recomputed)
 *   dg_j  = <dY, y_j>
 *   dS_j  = g_j (dg_j - sum_j' g_j' dg_j')   (softmax over the k scores)
 *   dX   += dS_j W_router[h][e_j]            (Algorithm 2, input gradient)
 *   dW_router[h][e_j] += dS_j x              (Algorithm 2, weight gradient)
 *   du    = g_j W2^T dY;  da = du * b * silu'(a);  db = du * silu(a)
 *   dX   += W1^T da + W3^T db
 *   dW1 += da x^T;  dW3 += db x^T;  dW2 += (g_j dY) u^T
 * Weight gradients are overwritten (not accumulated into).  Heads are
 * independent and processed in parallel; within a head tokens are visited in
 * ascending order, so the result is deterministic.
 * dS (optional) [T][Nh][k] receives the score gradients.
 *
 * With separate routing sub-tokens (Sec. 4.4, Eq. (9)) the router reads R
 * while the experts read X: the router terms above then use r in place of x
 * (dW_router += dS_j r) and go to dR (dR += dS_j W_router[h][e_j]) instead of
 * dX.  oracle_layer_backward is the case R = X, dR = dX.
 *
 * W3 == NULL selects the two-matrix GELU expert (Sec. 3.4, W1 = W_in,
 * W2 = W_out): u = gelu(a) with a = W_in x, and the expert terms become
 *   da = du * gelu'(a),  gelu'(z) = Phi(z) + z phi(z);  dX += W_in^T da
 *   dW_in += da x^T;  dW_out += (g_j dY) u^T
 * (no b, db or dW3).
 */
static int backward_impl(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                         const double *X, const double *R, const double *W_router,
                         const double *W1, const double *W3, const double *W2,
                         const int32_t *idx, const double *gate,
                         const double *dY, double *dX, double *dR, double *dW_router,
                         double *dW1, double *dW3, double *dW2, double *dS);

int oracle_layer_backward(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                          const double *X, const double *W_router,
                          const double *W1, const double *W3, const double *W2,
                          const int32_t *idx, const double *gate,
                          const double *dY, double *dX, double *dW_router,
                          double *dW1, double *dW3, double *dW2, double *dS)
{
    return backward_impl(T, Nh, dh, Ne, k, dff, X, X, W_router, W1, W3, W2, idx,
                         gate, dY, dX, dX, dW_router, dW1, dW3, dW2, dS);
}

/* The backward of oracle_layer_gelu (the two-matrix GELU expert). */
int oracle_layer_gelu_backward(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                               const double *X, const double *W_router,
                               const double *W_in, const double *W_out,
                               const int32_t *idx, const double *gate,
                               const double *dY, double *dX, double *dW_router,
                               double *dW_in, double *dW_out, double *dS)
{
    return backward_impl(T, Nh, dh, Ne, k, dff, X, X, W_router, W_in, NULL, W_out,
                         idx, gate, dY, dX, dX, dW_router, dW_in, NULL, dW_out, dS);
}

int oracle_layer_backward_routed(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                                 const double *X, const double *R,
                                 const double *W_router, const double *W1,
                                 const double *W3, const double *W2,
                                 const int32_t *idx, const double *gate,
                                 const double *dY, double *dX, double *dR,
                                 double *dW_router, double *dW1, double *dW3,
                                 double *dW2, double *dS)
{
    if (dR == dX) return ORACLE_EINVAL;
    return backward_impl(T, Nh, dh, Ne, k, dff, X, R, W_router, W1, W3, W2, idx,
                         gate, dY, dX, dR, dW_router, dW1, dW3, dW2, dS);
}

static int backward_impl(int64_t T, int Nh, int dh, int Ne, int k, int dff,
                         const double *X, const double *R, const double *W_router,
                         const double *W1, const double *W3, const double *W2,
                         const int32_t *idx, const double *gate,
                         const double *dY, double *dX, double *dR, double *dW_router,
                         double *dW1, double *dW3, double *dW2, double *dS)
{
    if (T < 0 || Nh <= 0 || dh <= 0 || Ne <= 0 || k <= 0 || dff <= 0)
        return ORACLE_EINVAL;
    memset(dW_router, 0, sizeof(double) * (size_t)Nh * Ne * dh);
    memset(dW1, 0, sizeof(double) * (size_t)Nh * Ne * dff * dh);
    if (dW3) memset(dW3, 0, sizeof(double) * (size_t)Nh * Ne * dff * dh);
    memset(dW2, 0, sizeof(double) * (size_t)Nh * Ne * dh * dff);
    int status = ORACLE_OK;

#pragma omp parallel for schedule(dynamic, 1)
    for (int h = 0; h < Nh; ++h) {
        double *a = (double *)malloc(sizeof(double) * (size_t)k * dff);
        double *b = (double *)malloc(sizeof(double) * (size_t)k * dff);
        double *u = (double *)malloc(sizeof(double) * (size_t)k * dff);
        double *y = (double *)malloc(sizeof(double) * (size_t)k * dh);
        double *dg = (double *)malloc(sizeof(double) * (size_t)k);
        double *du = (double *)malloc(sizeof(double) * (size_t)dff);
        if (!a || !b || !u || !y || !dg || !du) {
#pragma omp atomic write
            status = ORACLE_ENOMEM;
            free(a); free(b); free(u); free(y); free(dg); free(du);
            continue;
        }
        for (int64_t t = 0; t < T; ++t) {
            const int64_t th = t * Nh + h;
            const double *x = X + th * dh;
            const double *r = R + th * dh;
            const double *dy = dY + th * dh;
            const int32_t *id = idx + th * k;
            const double *g = gate + th * k;
            double *dx = dX + th * dh;
            double *dr = dR + th * dh;
            int bad = 0;
            for (int j = 0; j < k; ++j)
                if (id[j] < 0 || id[j] >= Ne) bad = 1;
            if (bad) {
#pragma omp atomic write
                status = ORACLE_EINVAL;
                break;
            }

            for (int j = 0; j < k; ++j) {
                const int64_t he = (int64_t)h * Ne + id[j];
                if (W3)
                    swiglu_expert(dh, dff, x, W1 + he * dff * dh,
                                  W3 + he * dff * dh, W2 + he * dh * dff,
                                  a + (int64_t)j * dff, b + (int64_t)j * dff,
                                  u + (int64_t)j * dff, y + (int64_t)j * dh);
                else
                    gelu_expert(dh, dff, x, W1 + he * dff * dh, W2 + he * dh * dff,
                                a + (int64_t)j * dff, u + (int64_t)j * dff,
                                y + (int64_t)j * dh);
                double acc = 0.0;
                for (int i = 0; i < dh; ++i) acc += dy[i] * y[(int64_t)j * dh + i];
                dg[j] = acc;
            }
            double gdg = 0.0;
            for (int j = 0; j < k; ++j) gdg += g[j] * dg[j];

            for (int i = 0; i < dh; ++i) dx[i] = 0.0;
            for (int i = 0; i < dh; ++i) dr[i] = 0.0;
            for (int j = 0; j < k; ++j) {
                const int64_t he = (int64_t)h * Ne + id[j];
                const double ds = g[j] * (dg[j] - gdg);
                if (dS) dS[th * k + j] = ds;

                /* Algorithm 2: router gradients for the selected expert. */
                const double *wr = W_router + he * dh;
                double *dwr = dW_router + he * dh;
                for (int i = 0; i < dh; ++i) {
                    dr[i] += ds * wr[i];
                    dwr[i] += ds * r[i];
                }

                /* Expert gradients. */
                const double *w1 = W1 + he * dff * dh;
                const double *w3 = W3 ? W3 + he * dff * dh : NULL;
                const double *w2 = W2 + he * dh * dff;
                double *dw1 = dW1 + he * dff * dh;
                double *dw3 = W3 ? dW3 + he * dff * dh : NULL;
                double *dw2 = dW2 + he * dh * dff;
                const double *aj = a + (int64_t)j * dff;
                const double *bj = b + (int64_t)j * dff;
                const double *uj = u + (int64_t)j * dff;
                for (int f = 0; f < dff; ++f) {
                    double acc = 0.0;
                    for (int i = 0; i < dh; ++i)
                        acc += w2[(int64_t)i * dff + f] * dy[i];
                    du[f] = g[j] * acc;
                }
                for (int i = 0; i < dh; ++i)
                    for (int f = 0; f < dff; ++f)
                        dw2[(int64_t)i * dff + f] += g[j] * dy[i] * uj[f];
                for (int f = 0; f < dff && !W3; ++f) {
                    const double da = du[f] * gelu_grad(aj[f]);
                    for (int i = 0; i < dh; ++i) {
                        dx[i] += da * w1[(int64_t)f * dh + i];
                        dw1[(int64_t)f * dh + i] += da * x[i];
                    }
                }
                for (int f = 0; f < dff && W3; ++f) {
                    const double sig = 1.0 / (1.0 + exp(-aj[f]));
                    const double dsilu = sig * (1.0 + aj[f] * (1.0 - sig));
                    const double da = du[f] * bj[f] * dsilu;
                    const double db = du[f] * aj[f] * sig;
                    for (int i = 0; i < dh; ++i) {
                        dx[i] += da * w1[(int64_t)f * dh + i] +
                                 db * w3[(int64_t)f * dh + i];
                        dw1[(int64_t)f * dh + i] += da * x[i];
                        dw3[(int64_t)f * dh + i] += db * x[i];
                    }
                }
            }
        }
        free(a); free(b); free(u); free(y); free(dg); free(du);
    }
    return status;
}

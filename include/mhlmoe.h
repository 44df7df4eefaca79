/*
 * libmhlmoe — the per-GPU hot path of Multi-Head LatentMoE on AMD MI355X
 * (gfx950): IO-aware routing and IO-aware expert computation.
 *
 * Paper: "Multi-Head LatentMoE" (arXiv 2602.04870).
 *
 * Each of the N_h heads is an independent Mixtral-style MoE (Eq. (1)-(4),
 * Sec. 2.2) applied to its d_h-wide slice of the latent token (Eq. (5)-(6),
 * Sec. 3.1).  The library computes, for every token t and head h:
 *
 *   s[e]    = X[t,h,:] . W_router[h,e,:]                     (FP32 router)
 *   key[e]  = s[e] + bias[h,e]                   (Algorithm 1, bias optional)
 *   idx     = the top_k experts by key, descending; ties -> lower index
 *   gate[j] = softmax_j( s[idx_j] )             (bias removed, Eq. (2)-(3))
 *   Y[t,h]  = sum_j gate[j] * W2 (silu(W1 x) * (W3 x)) with the weights of
 *             expert idx_j of head h                        (Eq. (1), SwiGLU)
 *
 * without writing the T x N_e score matrix or the d_ff-wide expert
 * intermediate to device memory (Sec. 3.3, Sec. 3.4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensor pointers are DEVICE pointers owned by the caller; the library
 *    never allocates device memory for tensors, frees or synchronises (the
 *    latent-layer entry points create a hipBLASLt handle once per device).  All work is enqueued on
 *    `stream` (a hipStream_t; NULL = the default stream) and the call returns
 *    without waiting.  Inputs must stay valid until that work completes.
 *  - Layouts are dense row-major; element (a,b,c) of [A][B][C] is at
 *    (a*B + b)*C + c.  Pointers must be 16-byte aligned.
 *  - `dtype` selects the element type of X, W1, W3, W2, Y, dY and dX:
 *    MHLMOE_F32 (float) or MHLMOE_BF16 (bfloat16 stored as uint16).
 *    W_router and bias are always float; idx, counts, offsets and perm are
 *    int32; gate is float; weight gradients are float.
 *  - Scratch memory comes from `workspace`, a device buffer of at least
 *    mhlmoe_workspace_size(...) bytes, 256-byte aligned, owned by the
 *    caller.  Its contents need no initialisation and are clobbered.
 *    Concurrent calls must use distinct workspaces.
 *  - Supported shapes: d_head in {64, 128}; d_ff a multiple of 32 in [32, 512];
 *    1 <= top_k <= 32; top_k <= n_experts <= 1024; 1 <= n_heads <= 1024;
 *    0 <= T and T * top_k < 2^31.  T = 0 is a valid no-op.
 *  - Errors: every call returns a mhlmoe_status; on failure nothing has
 *    been enqueued (argument errors) or a launch failed (MHLMOE_EHIP), and
 *    mhlmoe_last_error() gives a message for the calling thread.
 *  - Determinism: every forward output (idx, gate, counts, offsets, perm, Y)
 *    and every gradient is bitwise reproducible for identical inputs and
 *    shapes; no floating-point atomics are used.
 */
#ifndef MHLMOE_H
#define MHLMOE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum mhlmoe_status {
    MHLMOE_OK = 0,
    MHLMOE_EINVAL = 1,       /* bad pointer, shape or alignment; k > N_e    */
    MHLMOE_EUNSUPPORTED = 2, /* shape outside the compiled set              */
    MHLMOE_EWORKSPACE = 3,   /* workspace missing or smaller than required  */
    MHLMOE_EHIP = 4          /* a HIP launch or runtime call failed         */
} mhlmoe_status;

typedef enum mhlmoe_dtype {
    MHLMOE_F32 = 0,
    MHLMOE_BF16 = 1,
    /* widens the type to every non-negative int, so that a caller's
     * out-of-range value is a defined value the library rejects */
    MHLMOE_DTYPE_FORCE_INT32 = 0x7FFFFFFF
} mhlmoe_dtype;

typedef enum mhlmoe_op {
    MHLMOE_OP_ROUTE = 0,
    MHLMOE_OP_BUCKET = 1,
    MHLMOE_OP_EXPERTS = 2,
    MHLMOE_OP_LAYER = 3,
    MHLMOE_OP_LAYER_BACKWARD = 4,
    MHLMOE_OP_LATENT_LAYER = 5,
    MHLMOE_OP_LATENT_BACKWARD = 6,
    MHLMOE_OP_ROUTE_BACKWARD = 7,
    MHLMOE_OP_FORCE_INT32 = 0x7FFFFFFF /* as MHLMOE_DTYPE_FORCE_INT32 */
} mhlmoe_op;

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int mhlmoe_version(void);

/* Message describing the last failure on the calling thread ("" if none).
 * The pointer stays valid until the next libmhlmoe call on this thread. */
const char *mhlmoe_last_error(void);

/*
 * Workspace bytes that entry point `op` needs for this shape (d_ff and dtype
 * are ignored by MHLMOE_OP_ROUTE and MHLMOE_OP_BUCKET).  Writes *bytes and
 * returns MHLMOE_OK, or an error status for an invalid or unsupported shape.
 */
mhlmoe_status mhlmoe_workspace_size(mhlmoe_op op, int64_t T, int n_heads,
                                    int d_head, int n_experts, int top_k,
                                    int d_ff, mhlmoe_dtype dtype,
                                    size_t *bytes);

/*
 * IO-aware routing forward: Algorithm 1 (Sec. 3.3) with the gate of
 * Eq. (2)-(4) and the per-expert load counts.
 *
 *   X        [T][n_heads][d_head]        dtype          (in)
 *   W_router [n_heads][n_experts][d_head] float          (in)  — the paper's
 *            W_r[h] is d_head x n_experts; this is its transpose, so each
 *            expert's row is contiguous.
 *   bias     [n_heads][n_experts] float or NULL           (in)  — Algorithm
 *            1's load-balancing bias: added to the scores before the top-k,
 *            removed after, so it steers selection but never the gates.
 *   idx      [T][n_heads][top_k] int32                    (out) — selected
 *            experts in descending biased-score order, ties to the lower
 *            expert index.
 *   gate     [T][n_heads][top_k] float                    (out) — softmax
 *            over the k selected unbiased scores.
 *   counts   [n_heads][n_experts] int32                   (out) — number of
 *            (t, j) with idx[t][h][j] == e.
 * Scores are computed to fp32 accuracy (the paper's FP32 router) and never
 * leave the chip.  Non-finite scores give unspecified indices.
 */
mhlmoe_status mhlmoe_route(const void *X, const float *W_router,
                           const float *bias, int64_t T, int n_heads,
                           int d_head, int n_experts, int top_k,
                           mhlmoe_dtype dtype, int32_t *idx, float *gate,
                           int32_t *counts, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

/*
 * mhlmoe_route without a workspace, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Arguments, results and kernels are those of
 * mhlmoe_route; the scratch (per-block expert histograms, counts) lives in a
 * static device array of 32 MiB that the library holds on every device it
 * runs on until the process ends (its device address is looked up once per
 * device, on the first call there).  The call allocates nothing and frees
 * nothing.  Shapes needing more than 32 MiB of scratch (4 (n_heads *
 * ceil(T / 128) + 1) n_experts bytes, roughly; e.g. T = 65536, 8 heads,
 * 1024 experts needs 16 MiB) return MHLMOE_EWORKSPACE before anything is
 * enqueued.  Nothing in the scratch needs to start at zero.  All calls on
 * one device share its array: calls that overlap in time on one device
 * (other streams, other threads) race and must be ordered by the caller.
 */
mhlmoe_status mhlmoe_route_static(const void *X, const float *W_router,
                                  const float *bias, int64_t T, int n_heads,
                                  int d_head, int n_experts, int top_k,
                                  mhlmoe_dtype dtype, int32_t *idx,
                                  float *gate, int32_t *counts,
                                  hipStream_t stream);

/*
 * IO-aware routing backward, Algorithm 2 (Sec. 3.3) on its own: given the
 * forward's idx and gate and the gradient dgate of a loss with respect to
 * the gates,
 *   dS_j = g_j (dgate_j - sum_j' g_j' dgate_j')       (softmax backward)
 *   dX[t][h] = sum_j dS_j W_router[h][e_j]
 *   dW_router[h][e] = sum over the (t, j) with e_j = e of dS_j X[t][h]
 * Gradients reach only the k selected experts of each token (no T x N_e
 * matrix); none reaches the bias or the selection.
 *
 *   X, W_router, idx, gate    the forward's inputs and outputs      (in)
 *   dgate [T][n_heads][top_k] float                                (in)
 *   dX    [T][n_heads][d_head] dtype                               (out)
 *   dW_router [n_heads][n_experts][d_head] float (out, overwritten;
 *             experts that received no slot get exact zeros)
 * dW_router is a fixed-order segmented sum over the clustered slots, so the
 * results are bitwise reproducible.  idx entries must lie in [0, n_experts).
 * Workspace: MHLMOE_OP_ROUTE_BACKWARD (d_ff ignored).
 */
mhlmoe_status mhlmoe_route_backward(const void *X, const float *W_router,
                                    const int32_t *idx, const float *gate,
                                    const float *dgate, int64_t T, int n_heads,
                                    int d_head, int n_experts, int top_k,
                                    mhlmoe_dtype dtype, void *dX,
                                    float *dW_router, void *workspace,
                                    size_t workspace_bytes, hipStream_t stream);

/*
 * Token clustering (Sec. 3.4, Fig. 2): a stable counting sort of every
 * head's routed slots by expert, so each expert's tokens are contiguous.
 *
 *   idx     [T][n_heads][top_k] int32    (in)  values in [0, n_experts)
 *   counts  [n_heads][n_experts] int32   (out, may be NULL)
 *   offsets [n_heads][n_experts + 1]     (out) exclusive prefix sum of counts;
 *           offsets[h][n_experts] = T * top_k.
 *   perm    [n_heads][T * top_k] int32   (out) perm[h][offsets[h][e] + r] is
 *           the slot id t*top_k + j of the r-th slot, in ascending (t, j)
 *           order, routed to expert e in head h.
 * Out-of-range idx values give unspecified results (no fault).
 */
mhlmoe_status mhlmoe_bucket(const int32_t *idx, int64_t T, int n_heads,
                            int n_experts, int top_k, int32_t *counts,
                            int32_t *offsets, int32_t *perm, void *workspace,
                            size_t workspace_bytes, hipStream_t stream);

/*
 * IO-aware expert computation (Sec. 3.4), dropless, and the gate-weighted
 * combine of Eq. (1); the per-head outputs are laid side by side, which is
 * the concat of Eq. (6).
 *
 *   X    [T][n_heads][d_head]                 dtype   (in)
 *   idx  [T][n_heads][top_k] int32                    (in)
 *   gate [T][n_heads][top_k] float                    (in)
 *   W1   [n_heads][n_experts][d_ff][d_head]   dtype   (in) gate projection
 *   W3   [n_heads][n_experts][d_ff][d_head]   dtype   (in) up projection
 *   W2   [n_heads][n_experts][d_head][d_ff]   dtype   (in) down projection
 *   Y    [T][n_heads][d_head]                 dtype   (out)
 * Every slot is computed (no capacity limit); the d_ff-wide intermediate
 * stays on chip.  Accumulation is fp32; bf16 results are rounded to nearest
 * even once per output element.
 */
mhlmoe_status mhlmoe_experts(const void *X, const int32_t *idx,
                             const float *gate, const void *W1, const void *W3,
                             const void *W2, int64_t T, int n_heads,
                             int d_head, int n_experts, int top_k, int d_ff,
                             mhlmoe_dtype dtype, void *Y, void *workspace,
                             size_t workspace_bytes, hipStream_t stream);

/*
 * The whole per-GPU layer: mhlmoe_route then mhlmoe_experts, sharing the
 * routing kernel's per-block expert histograms with the clustering step.
 * Arguments as above.  idx, gate and counts are optional outputs (NULL keeps
 * them in the workspace); pass idx and gate to run mhlmoe_layer_backward.
 */
mhlmoe_status mhlmoe_layer(const void *X, const float *W_router,
                           const float *bias, const void *W1, const void *W3,
                           const void *W2, int64_t T, int n_heads, int d_head,
                           int n_experts, int top_k, int d_ff,
                           mhlmoe_dtype dtype, void *Y, int32_t *idx,
                           float *gate, int32_t *counts, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

/*
 * The paper's own expert form (Sec. 3.4): each expert is the two-matrix
 * GELU MLP  y = W_out gelu(W_in x),  gelu(z) = z Phi(z) (the exact, erf
 * form), which Sec. 3.4 evaluates as block-sparse attention with
 * score_mod(s) = log(gelu(s) + 1).  Everything else (routing, clustering,
 * the gate-weighted combine of Eq. (1)) is as in mhlmoe_experts and
 * mhlmoe_layer, with the same workspace sizes (MHLMOE_OP_EXPERTS and
 * MHLMOE_OP_LAYER).
 *
 *   W_in  [n_heads][n_experts][d_ff][d_head]  dtype   (W1's layout)  (in)
 *   W_out [n_heads][n_experts][d_head][d_ff]  dtype   (W2's layout)  (in)
 *
 * Supported: the shapes of mhlmoe_experts / mhlmoe_layer (dtype MHLMOE_BF16
 * or MHLMOE_F32, d_head 64 or 128, the paper's 16 x 64 and 8 x 128 head
 * configurations among them, d_ff a multiple of 32 in [32, 512]); other
 * shapes return MHLMOE_EUNSUPPORTED.  On the GPU Phi is a logistic function
 * of a fitted odd polynomial, Phi(z) ~ 1 / (1 + exp(-z P(z^2))) with P of
 * degree 4 (|Phi error| <= 1.6e-6), below the rounding of the intermediate
 * (bf16) and within the fp32 tolerance.
 */
mhlmoe_status mhlmoe_experts_gelu(const void *X, const int32_t *idx,
                                  const float *gate, const void *W_in,
                                  const void *W_out, int64_t T, int n_heads,
                                  int d_head, int n_experts, int top_k,
                                  int d_ff, mhlmoe_dtype dtype, void *Y,
                                  void *workspace, size_t workspace_bytes,
                                  hipStream_t stream);

mhlmoe_status mhlmoe_layer_gelu(const void *X, const float *W_router,
                                const float *bias, const void *W_in,
                                const void *W_out, int64_t T, int n_heads,
                                int d_head, int n_experts, int top_k, int d_ff,
                                mhlmoe_dtype dtype, void *Y, int32_t *idx,
                                float *gate, int32_t *counts, void *workspace,
                                size_t workspace_bytes, hipStream_t stream);

/*
 * Backward of mhlmoe_layer: Algorithm 2 (routing backward, gradients only
 * for the k selected experts, Sec. 3.3) and the gradient of Eq. (1)-(3) with
 * the SwiGLU expert, recomputing the expert intermediate instead of storing
 * it.  No gradient flows through the selection or to the bias.
 *
 *   X, W_router, W1, W3, W2   forward inputs                  (in)
 *   idx, gate                 the forward's outputs           (in)
 *   dY   [T][n_heads][d_head] dtype                           (in)
 *   dX   [T][n_heads][d_head] dtype                           (out)
 *   dW_router [n_heads][n_experts][d_head] float              (out)
 *   dW1, dW3  [n_heads][n_experts][d_ff][d_head] float        (out)
 *   dW2       [n_heads][n_experts][d_head][d_ff] float        (out)
 * Weight gradients are overwritten, not accumulated into; experts that
 * received no slot get exact zeros.  dtype must be MHLMOE_BF16 (activations,
 * dY, dX and expert weights bf16; MHLMOE_EUNSUPPORTED otherwise); gradients
 * are accumulated in fp32 and the sums are taken in a fixed order, so equal
 * inputs give bitwise equal outputs.  idx entries must lie in
 * [0, n_experts) (the forward guarantees it); other values are not
 * detected.  Same shape limits as mhlmoe_layer.
 */
mhlmoe_status mhlmoe_layer_backward(
    const void *X, const float *W_router, const void *W1, const void *W3,
    const void *W2, const int32_t *idx, const float *gate, const void *dY,
    int64_t T, int n_heads, int d_head, int n_experts, int top_k, int d_ff,
    mhlmoe_dtype dtype, void *dX, float *dW_router, float *dW1, float *dW3,
    float *dW2, void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Backward of mhlmoe_layer_gelu (the two-matrix GELU expert of Sec. 3.4):
 * as mhlmoe_layer_backward with u = gelu(a), a = W_in x, and
 *   da = (g W_out^T dY) * gelu'(a),  gelu'(z) = Phi(z) + z phi(z),
 *   dX_expert = W_in^T da,  dW_in = sum da x^T,  dW_out = sum (g dY) u^T.
 *   dW_in  [n_heads][n_experts][d_ff][d_head] float  (out)
 *   dW_out [n_heads][n_experts][d_head][d_ff] float  (out)
 * dtype MHLMOE_BF16 (fp32 returns MHLMOE_EUNSUPPORTED, as for
 * mhlmoe_layer_backward); d_head in {64, 128}, d_ff a multiple of 32 up to
 * 512.  On the GPU
 * Phi comes from the Abramowitz & Stegun 7.1.26 erf (|error| <= 1.5e-7) and
 * phi from the exponential it already evaluates; the recomputed gelu(a)
 * differs from the forward's by at most 1.6e-6 |a|.  Workspace:
 * MHLMOE_OP_LAYER_BACKWARD.
 */
mhlmoe_status mhlmoe_layer_gelu_backward(
    const void *X, const float *W_router, const void *W_in, const void *W_out,
    const int32_t *idx, const float *gate, const void *dY, int64_t T,
    int n_heads, int d_head, int n_experts, int top_k, int d_ff,
    mhlmoe_dtype dtype, void *dX, float *dW_router, float *dW_in,
    float *dW_out, void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Separate routing sub-tokens (Sec. 4.4, Eq. (9)): W_in x is split into
 * 2 n_heads sub-tokens, x_{t,i} for the experts and r_{t,i} for the router.
 * The layer routes head h of token t by R[t][h] and computes the experts on
 * X[t][h]; everything else is as in mhlmoe_layer.  W3 == NULL selects the
 * two-matrix GELU expert (W1 = W_in, W2 = W_out, with mhlmoe_layer_gelu's
 * shape limits).  With R == X the outputs equal mhlmoe_layer's (or
 * mhlmoe_layer_gelu's) bit for bit.  Workspace: MHLMOE_OP_LAYER.
 *
 *   R  [T][n_heads][d_head]  dtype  (in)  the routing sub-tokens
 */
mhlmoe_status mhlmoe_layer_routed(const void *X, const void *R,
                                  const float *W_router, const float *bias,
                                  const void *W1, const void *W3,
                                  const void *W2, int64_t T, int n_heads,
                                  int d_head, int n_experts, int top_k,
                                  int d_ff, mhlmoe_dtype dtype, void *Y,
                                  int32_t *idx, float *gate, int32_t *counts,
                                  void *workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/*
 * Backward of mhlmoe_layer_routed (bf16): as mhlmoe_layer_backward (W3 ==
 * NULL: as mhlmoe_layer_gelu_backward, dW3 unused), except that Algorithm
 * 2's router gradients are taken against R: dR receives
 * sum_j dS_j W_router[h][e_j] and dW_router sums dS_j R[t][h], while dX
 * holds the expert input gradient only.
 *
 *   R   [T][n_heads][d_head]  bf16  (in)
 *   dR  [T][n_heads][d_head]  bf16  (out) a buffer distinct from dX; may be
 *                                   NULL only when T == 0.
 * Workspace: MHLMOE_OP_LAYER_BACKWARD.  The expert weight gradients equal
 * mhlmoe_layer_backward's bit for bit at the same (X, idx, gate, dY).
 */
mhlmoe_status mhlmoe_layer_backward_routed(
    const void *X, const void *R, const float *W_router, const void *W1,
    const void *W3, const void *W2, const int32_t *idx, const float *gate,
    const void *dY, int64_t T, int n_heads, int d_head, int n_experts,
    int top_k, int d_ff, mhlmoe_dtype dtype, void *dX, void *dR,
    float *dW_router, float *dW1, float *dW3, float *dW2, void *workspace,
    size_t workspace_bytes, hipStream_t stream);

/*
 * The whole Multi-Head LatentMoE layer with its projections (Eq. (5)-(6),
 * Sec. 3.1), N = n_heads * d_head latent width:
 *
 *   X_lat = W_in x                 [T][N], read as [T][n_heads][d_head]: the
 *                                  split of Eq. (5) is a view, no copy
 *   Y_lat = the per-head MoEs of mhlmoe_layer on X_lat (idx, gate, counts
 *           as there; W3 == NULL selects the two-matrix GELU expert)
 *   out   = W_out concat(Y_lat)    [T][d_model] (Eq. (6))
 *
 * routing_tokens = 1 gives the separate routing sub-tokens of Sec. 4.4,
 * Eq. (9): W_in then has 2N rows, its first N produce X_lat and its last N
 * the routing sub-tokens R_lat, which the router reads instead of X_lat.
 *
 *   x      [T][d_model]                         dtype  (in)
 *   W_in   [(1 + routing_tokens) N][d_model]    dtype  (in)
 *   W_out  [d_model][N]                         dtype  (in)
 *   out    [T][d_model]                         dtype  (out)
 *   X_lat, R_lat, Y_lat [T][n_heads][d_head]    dtype  (out, optional: NULL
 *          keeps them in the workspace; keep X_lat, Y_lat (and R_lat) for
 *          mhlmoe_latent_layer_backward)
 * The projections are hipBLASLt GEMMs with fp32 accumulation, rounded once
 * to dtype; the library creates one hipBLASLt handle per device on first use
 * and caches a GEMM plan per shape (the only host-side allocations of the
 * library besides the timing events).  Their results are reproducible for a
 * given hipBLASLt build and shape.  1 <= d_model <= 65536.  Workspace:
 * MHLMOE_OP_LATENT_LAYER (d_model does not change its size).
 */
mhlmoe_status mhlmoe_latent_layer(const void *x, const void *W_in,
                                  const float *W_router, const float *bias,
                                  const void *W1, const void *W3,
                                  const void *W2, const void *W_out,
                                  int64_t T, int d_model, int n_heads,
                                  int d_head, int n_experts, int top_k,
                                  int d_ff, int routing_tokens,
                                  mhlmoe_dtype dtype, void *out, void *X_lat,
                                  void *R_lat, void *Y_lat, int32_t *idx,
                                  float *gate, int32_t *counts,
                                  void *workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/*
 * Backward of mhlmoe_latent_layer (bf16; W3 == NULL: the GELU expert, dW3
 * unused), given the
 * forward's x, X_lat, (R_lat), Y_lat, idx and gate and the output gradient
 * dout [T][d_model]:
 *
 *   dY_lat = dout W_out;  dW_out = dout^T Y_lat
 *   the heads' backward of mhlmoe_layer_backward (mhlmoe_layer_backward_routed
 *   with routing sub-tokens) on X_lat and dY_lat -> dX_lat (dR_lat) and
 *   dW_router, dW1, dW3, dW2
 *   dW_in = [dX_lat; dR_lat]^T x;  dx = dX_lat W_in_x (+ dR_lat W_in_r)
 *
 *   dx     [T][d_model]                        bf16   (out)
 *   dW_in  [(1 + routing_tokens) N][d_model]   float  (out)
 *   dW_out [d_model][N]                        float  (out)
 *   dW_router, dW1, dW3, dW2 as in mhlmoe_layer_backward (out)
 * dY_lat, dX_lat and dR_lat are rounded to bf16 in the workspace; with
 * routing sub-tokens dx is the bf16 sum of its two products (accumulated by
 * the second GEMM).  Workspace: MHLMOE_OP_LATENT_BACKWARD.
 */
mhlmoe_status mhlmoe_latent_layer_backward(
    const void *x, const void *W_in, const float *W_router, const void *W1,
    const void *W3, const void *W2, const void *W_out, const void *X_lat,
    const void *R_lat, const void *Y_lat, const int32_t *idx,
    const float *gate, const void *dout, int64_t T, int d_model, int n_heads,
    int d_head, int n_experts, int top_k, int d_ff, int routing_tokens,
    mhlmoe_dtype dtype, void *dx, float *dW_in, float *dW_router, float *dW1,
    float *dW3, float *dW2, float *dW_out, void *workspace,
    size_t workspace_bytes, hipStream_t stream);

/*
 * Auxiliary-loss-free load balancing (Sec. 2.2, after the aux-free method it
 * cites): after a batch, every head's routing bias (Algorithm 1's b) moves
 * toward equal expert load by a fixed rate,
 *
 *   bias[h][e] += rate * sign(mean_e' counts[h][e'] - counts[h][e]),
 *
 * with sign(0) = 0, the mean compared exactly in integers and each bias
 * changed by one fp32 addition (round to nearest even).
 *
 *   counts [n_heads][n_experts] int32  (in)  e.g. mhlmoe_layer's counts,
 *                                      summed over the batches of a step
 *   bias   [n_heads][n_experts] float  (in/out, updated in place)
 *   rate   the update rate u, finite and >= 0 (MHLMOE_EINVAL otherwise)
 * 1 <= n_heads <= 1024, 1 <= n_experts <= 1024; no workspace.  The call
 * enqueues one kernel on `stream`; calls that update the same bias must be
 * ordered by the caller.
 */
mhlmoe_status mhlmoe_bias_update(const int32_t *counts, float *bias,
                                 int n_heads, int n_experts, float rate,
                                 hipStream_t stream);

/*
 * Per-kernel timing (a measurement aid, off by default).  While enabled, each
 * kernel the library launches is bracketed by two HIP events recorded on the
 * caller's stream, so the measured interval is that kernel's execution on
 * the stream it actually runs on.  Kernel names: "route_fwd", "hist",
 * "count_scan", "scatter", "ffn", "combine", "bwd_dx", "bwd_combine",
 * "bwd_dw", "router_dw", "route_bwd", "bias_update", "proj_in", "proj_out" and
 * "proj_bwd" (the projection GEMMs of the latent layer).
 *
 * mhlmoe_timing_enable(on)   start (on != 0) or stop recording; records
 *                            already taken are kept.
 * mhlmoe_timing_query(name, total_ms, launches)
 *                            waits for the recorded events of kernel `name`
 *                            and returns the sum of their durations (ms) and
 *                            how many launches were recorded.
 * mhlmoe_timing_reset()      waits for and drops every record.
 * Events are created on first use and reused; enabling timing is the only
 * way the library creates HIP objects.
 */
mhlmoe_status mhlmoe_timing_enable(int on);
mhlmoe_status mhlmoe_timing_query(const char *kernel, double *total_ms,
                                  int64_t *launches);
mhlmoe_status mhlmoe_timing_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* MHLMOE_H */

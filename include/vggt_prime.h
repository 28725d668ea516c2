/*
 * vggt_prime.h -- C ABI of libvggtprime.so: the routed global-attention layer
 * of VGGT-Prime (a compute-adaptive mixture of heads) on AMD Instinct MI355X
 * (gfx950).
 *
 * The layer (Algorithm 1, step 2 "compute routed attention"; Sections 4.1-4.3):
 * for every attention head h with per-head Q_h, K_h, V_h in R^{N x d} over all
 * N = S * P tokens of all views,
 *   1. a router pools the queries with gated attention (Eq.1-2), lets the
 *      pooled query attend to all keys (routing vector r_h) and scores the
 *      head by its largest routing weight s_h = max r_h (Eq.3);
 *   2. each head is assigned one computation mode (Eq.4):
 *        FULL  (s_h >= tau_high): exact softmax attention over all tokens,
 *        SURR  (tau_low < s_h < tau_high): learned surrogate, Eq.5-7,
 *        MEAN  (s_h <= tau_low): broadcast of the mean value token;
 *   3. the head outputs are concatenated (Algorithm 1, step 3).
 *
 * Conventions for every entry point:
 *   - Tensor arguments are DEVICE pointers owned by the caller.  The library
 *     never allocates, frees or synchronises; each call only enqueues work on
 *     `stream` (a hipStream_t passed as void*; NULL = the default stream) and
 *     returns.  Calls are stateless and re-entrant.
 *   - Struct arguments (vp_shape, vp_router_weights, ...) are HOST memory,
 *     read during the call only; the pointers inside them are device pointers.
 *   - Arguments are validated on the host before anything is enqueued; on an
 *     error nothing is enqueued and a VP_ERR_* code is returned.  A HIP
 *     launch error after enqueueing returns VP_ERR_HIP; vp_last_error() then
 *     gives the message (thread-local).
 *   - Q, K, V, Y are [N, H, d] row-major (token-major; the d values of one
 *     head of one token are contiguous).  Supported: 1 <= H <= 16, d = 64,
 *     router/surrogate hidden size L = 64, dtype fp32 or bf16 (fp32
 *     accumulation everywhere).
 *   - Numeric anomalies never fail a call: a NaN routing score sends its head
 *     to FULL and sets bit 0 of the flags word of `buckets`.
 */
#ifndef VGGT_PRIME_H
#define VGGT_PRIME_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    VP_OK = 0,
    VP_ERR_INVALID_ARG = 1,  /* null pointer, bad size, misaligned pointer, bad enum */
    VP_ERR_UNSUPPORTED = 2,  /* valid but unsupported shape (d != 64, H > 16, L != 64) */
    VP_ERR_WORKSPACE = 3,    /* workspace smaller than vp_workspace_bytes() */
    VP_ERR_HIP = 4           /* a HIP runtime error while enqueueing */
} vp_status;

typedef enum { VP_F32 = 0, VP_BF16 = 1 } vp_dtype;

/* Computation modes, ordered by cost (Eq.4). */
enum { VP_MODE_MEAN = 0, VP_MODE_SURR = 1, VP_MODE_FULL = 2, VP_NUM_MODES = 3 };

typedef enum {
    VP_ASSIGN_THRESHOLD = 0,        /* Eq.4 on the saliency scores s_h */
    VP_ASSIGN_ARGMAX = 1,           /* first argmax over the three per-head logits */
    /* Binary routing of the compute-mode study (Section 5.3, Table 6): two modes
     * only, FULL and MEAN. */
    VP_ASSIGN_THRESHOLD_BINARY = 2, /* FULL if s_h >= tau_high, MEAN otherwise */
    VP_ASSIGN_ARGMAX_BINARY = 3     /* FULL if its logit beats MEAN's, MEAN otherwise */
} vp_assign_rule;

/* Query pooling of the router (component study, Section 5.3, Table 5). */
typedef enum {
    VP_POOL_GATED = 0, /* gated attention pooling, Eq.1-2 */
    VP_POOL_MEAN = 1   /* "mean query": q_pool = (1/N) sum_i q_i (W, U, w unused) */
} vp_pool;

/* How SURR heads are computed: Eq.5-7, or one of the ablations of the
 * component study (Section 5.3, Table 5) and of the compute-mode study (Table 6). */
typedef enum {
    VP_SURR_EQ7 = 0,          /* y_i = C_h + gamma_i (.) delta_i (Eq.5-7) */
    VP_SURR_MEAN_CONTEXT = 1, /* Eq.6-7 with C_h replaced by the value mean */
    VP_SURR_NO_RESIDUAL = 2,  /* y_i = C_h (MLP weights unused) */
    VP_SURR_ADD_IDENTITY = 3, /* y_i = v_{h,i} + C_h + gamma_i (.) delta_i */
    VP_SURR_LINEAR_ATTN = 4   /* linear attention with phi(x) = elu(x) + 1 over all
                                 N tokens: y_i = sum_j (phi(q_i).phi(k_j)) v_j /
                                 sum_j phi(q_i).phi(k_j) (MLP weights unused) */
} vp_surr_variant;

typedef enum { VP_ACT_GELU_ERF = 0, VP_ACT_RELU = 1 } vp_act;

#define VP_MAX_HEADS 16
#define VP_HEAD_DIM 64
#define VP_HIDDEN 64
/* Size in int32 of the `buckets` array: counts[3], head list[16], flags[1]. */
#define VP_BUCKETS_LEN (VP_NUM_MODES + VP_MAX_HEADS + 1)
#define VP_FLAG_NAN_SCORE 1u

/* N = S * P tokens: S views of P tokens each (all views attend jointly). */
typedef struct {
    int64_t S, P;
    int32_t H, d;
    vp_dtype dtype; /* storage type of Q, K, V and of every weight matrix */
} vp_shape;

/* Gated attention pooling parameters (Eq.1): W, U are [H, L, d], w is [H, L],
 * all in shape.dtype; no biases.  `scale` multiplies q_pool . k in the
 * single-query attention (1/sqrt(d) when 0 is passed).  With pool =
 * VP_POOL_MEAN, W, U and w are not read and may be NULL (L is still 64). */
typedef struct {
    const void *W, *U, *w;
    int32_t L;
    float scale;
    vp_pool pool;
} vp_router_weights;

/* Router outputs, device fp32, written by vp_router_score:
 *   q_pool [H, d]  pooled query (Eq.2)
 *   stats  [H, 2]  (m_h, l_h): m_h = max_j t_{h,j}, l_h = sum_j exp(t_{h,j} - m_h),
 *                  t_{h,j} = scale * q_pool_h . k_{h,j}
 *   score  [H]     s_h = max_j r_h(j) = 1 / l_h (Eq.3)
 *   ctx    [H, d]  C_h = r_h V_h (Eq.5)
 *   vmean  [H, d]  (1/N) sum_j v_{h,j} (Algorithm 1, mean branch) */
typedef struct {
    float *q_pool, *stats, *score, *ctx, *vmean;
} vp_router_state;

/* Surrogate MLPs (Eq.6), per head: Linear(2d -> L) -> act -> Linear(L -> d)
 * acting on z = [v_{h,i}; C_h].  *_w1 [H, L, 2d] and *_w2 [H, d, L] in
 * shape.dtype; biases *_b1 [H, L], *_b2 [H, d] fp32.  g_* is the gate MLP
 * (gamma = sigmoid(MLP_gamma(z))), d_* the correction MLP (delta).
 * `variant` selects Eq.5-7 or an ablation; the variants NO_RESIDUAL and
 * LINEAR_ATTN read no weight (the pointers may then be NULL). */
typedef struct {
    const void *g_w1, *g_w2, *d_w1, *d_w2;
    const float *g_b1, *g_b2, *d_b1, *d_b2;
    int32_t L;
    vp_act act;
    vp_surr_variant variant;
} vp_surrogate_weights;

/* Bytes of device workspace that vp_router_score, vp_routed_global_attention
 * and its stages need for `shape` (0 if the shape is invalid).  The workspace
 * holds router partial sums, the gathered keys and values of FULL heads, the
 * FULL kernel's partial results and the linear-attention sums; it must be 256-byte
 * aligned and may be reused across calls on one stream (calls on different
 * streams need separate workspaces). */
size_t vp_workspace_bytes(const vp_shape *shape);

/* Router (Section 4.1, Eq.1-3; context Eq.5; value mean, Algorithm 1).
 * Reads Q, K, V once each (HBM-bound); writes every field of `out`.
 * Deterministic: partial sums are combined in a fixed order. */
vp_status vp_router_score(const vp_shape *shape, const void *Q, const void *K, const void *V,
                          const vp_router_weights *rw, vp_router_state *out, void *ws,
                          size_t ws_bytes, void *stream);

/* vp_router_score for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same kernels and results, with the router's partial sums kept in a
 * static device array of the library (4.5 MiB, one per device, held until
 * the process ends) instead of a caller workspace.  It calls no allocating
 * routine.  Every shape the library accepts fits; a shape needing more than
 * the array returns VP_ERR_WORKSPACE (message in vp_last_error).  All calls
 * on one device share that device's array: calls that overlap on one device
 * (different streams, or host threads) race and must be serialised by the
 * caller.  The array's address is looked up once per device, on the first
 * call made with that device current. */
vp_status vp_router_score_noalloc(const vp_shape *shape, const void *Q, const void *K,
                                  const void *V, const vp_router_weights *rw,
                                  vp_router_state *out, void *stream);

/* Linear-logit mode router of the synthetic workloads (not a construct of the
 * paper): logits[r] = sum_c W_r[r, c] * u[c] + b_r[r] for r = h * M + m,
 * m in (MEAN, SURR, FULL).  u: fp32 [Din]; W_r: [H * M, Din] in w_dtype;
 * b_r: fp32 [H * M]; logits: fp32 [H, M].  1 <= Din <= 65536.  M is the number
 * of modes, which Eq.4 fixes at VP_NUM_MODES = 3; any other M returns
 * VP_ERR_UNSUPPORTED. */
vp_status vp_router_logits(const float *u, const void *W_r, const float *b_r, int32_t H,
                           int32_t Din, int32_t M, vp_dtype w_dtype, float *logits,
                           void *stream);

/* Mode assignment (Eq.4).  `scores` holds M values per head: M = 1 for the
 * threshold rules (s_h), M = VP_NUM_MODES = 3 for the argmax rules (logits);
 * any other M for the rule returns VP_ERR_UNSUPPORTED.
 * THRESHOLD: scores = s_h [H]; FULL if s >= tau_high,
 * MEAN if s <= tau_low, SURR otherwise (0 <= tau_low <= tau_high).  ARGMAX:
 * scores = logits [H, 3]; the first maximal mode.  THRESHOLD_BINARY: FULL if
 * s >= tau_high, else MEAN (tau_low is checked but unused).  ARGMAX_BINARY:
 * FULL if logit[FULL] > logit[MEAN], else MEAN (the SURR logit is ignored).
 * NaN (in a score or a compared logit) -> FULL + flag.
 * Writes modes [H] (uint8) and buckets [VP_BUCKETS_LEN] (int32):
 *   buckets[0..2]   number of heads in MEAN, SURR, FULL;
 *   buckets[3..3+H) head ids grouped by mode (MEAN, then SURR, then FULL),
 *                   ascending within a group;
 *   buckets[3+16]   flags (bit 0: a NaN score was seen). */
vp_status vp_assign_heads(const float *scores, int32_t H, int32_t M, vp_assign_rule rule,
                          float tau_low, float tau_high, uint8_t *modes, int32_t *buckets,
                          void *stream);

/* Routed global attention (Algorithm 1 step 2, Eq.5-7): writes Y [N, H, d] in
 * y_dtype, every head in the mode vp_assign_heads gave it.  `modes` [H] and
 * `buckets` are the device outputs of vp_assign_heads for the same call: the
 * MEAN and SURR kernels read modes[h], the FULL kernels take the FULL head
 * list from buckets; nothing is copied back to the host.
 *   FULL heads: softmax(Q_h K_h^T / sqrt(d)) V_h over all N tokens;
 *   SURR heads: C_h + gamma (.) delta with C_h = state->ctx (Eq.5-7), or
 *               the ablation surr->variant names;
 *   MEAN heads: every row = state->vmean[h].
 * `state` must hold the vp_router_score outputs for the same Q, K, V.
 * `surr` must be non-NULL (its weights are read only for SURR heads).
 * Every output element is written exactly once. */
vp_status vp_routed_global_attention(const vp_shape *shape, const void *Q, const void *K,
                                     const void *V, const uint8_t *modes,
                                     const int32_t *buckets, const vp_router_state *state,
                                     const vp_surrogate_weights *surr, void *Y,
                                     vp_dtype y_dtype, void *ws, size_t ws_bytes,
                                     void *stream);

/* The three stages of vp_routed_global_attention, in the order it runs them,
 * for callers that schedule or time them separately (same arguments and
 * requirements as vp_routed_global_attention; run all three, in this order,
 * on one stream, to obtain the same Y).
 *   vp_gather_full_heads:   packs V (tile-transposed, scaled by a power of
 *                           two per head, fp16) and K (fp16 tiles) of each
 *                           FULL head into the workspace (bf16 layers; no-op
 *                           for fp32) and records the largest key norm of
 *                           every 64-key tile;
 *   vp_full_head_attention: exact softmax attention of every FULL head
 *                           (Algorithm 1, first branch); reads the packed
 *                           tiles the gather left in `ws` (bf16) and keeps
 *                           the partial results of work split over compute
 *                           units there (both dtypes).  Results are
 *                           deterministic for a given device (the split of
 *                           work over its compute units is fixed);
 *   vp_linear_heads:        SURR (Eq.5-7, or surr->variant) and MEAN heads.
 *                           Q, K and ws are read only by the LINEAR_ATTN
 *                           variant (they may be NULL / 0 otherwise), which
 *                           keeps its per-head sums in ws. */
vp_status vp_gather_full_heads(const vp_shape *shape, const void *K, const void *V,
                               const int32_t *buckets, void *ws, size_t ws_bytes, void *stream);
vp_status vp_full_head_attention(const vp_shape *shape, const void *Q, const void *K,
                                 const void *V, const int32_t *buckets, void *Y,
                                 vp_dtype y_dtype, void *ws, size_t ws_bytes, void *stream);
vp_status vp_linear_heads(const vp_shape *shape, const void *Q, const void *K, const void *V,
                          const uint8_t *modes, const vp_router_state *state,
                          const vp_surrogate_weights *surr, void *Y, vp_dtype y_dtype,
                          void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * The dense block around the routed layer (Algorithm 1, steps 1, 3 and 4), for
 * bf16 layers with H = 16 heads of d = 64 (model width D = 1024):
 *   vp_block_qkv:  X~ = LN_1(X); (Q, K, V) = X~ W_qkv^T + b_qkv, then the 2D
 *                  rotary encoding of the token positions applied to Q and K
 *                  (the positional information P of QKV_h(X~, P));
 *   [vp_router_score, vp_assign_heads, vp_routed_global_attention: Y]
 *   vp_block_out:  X_attn = X + LS_1 (Y W_O^T + b_O);
 *                  X_out  = X_attn + LS_2 (GELU(LN_2(X_attn) W_fc1^T + b_fc1)
 *                           W_fc2^T + b_fc2).
 * LN: per token, (x - mean) / sqrt(var + eps) * gain + bias (biased variance).
 * Rotary encoding: in each head, features j and j + 16 of the first 32 form a
 * plane rotated by row * base^(-j/16), those of the last 32 by column *
 * base^(-j/16), j < 16.  GELU: x (1 + erf(x / sqrt 2)) / 2.
 * X, Y, X_out, Q, K, V: [N, D] bf16 (Q, K, V and Y are the [N, H, d] tensors
 * of the routed layer); pos: int32 [N, 2] (row, column) per token.  Weight
 * matrices bf16 [out, in] row-major; biases, LN gains and biases and LayerScale
 * vectors fp32.  Arithmetic in fp32, every output rounded once to bf16.
 * X_out may be the same buffer as X. */
typedef struct {
    const float *ln1_w, *ln1_b;   /* [D] */
    const void *w_qkv;            /* [3D, D]: rows 0..D-1 Q, D..2D-1 K, 2D..3D-1 V */
    const float *b_qkv;           /* [3D] */
    const void *w_o;              /* [D, D] */
    const float *b_o, *ls1;       /* [D] */
    const float *ln2_w, *ln2_b;   /* [D] */
    const void *w_fc1;            /* [4D, D] */
    const float *b_fc1;           /* [4D] */
    const void *w_fc2;            /* [D, 4D] */
    const float *b_fc2, *ls2;     /* [D] */
    float ln_eps;                 /* 1e-6 when 0 */
    float rope_base;              /* 100 when 0 */
} vp_block_weights;

/* Bytes of device workspace vp_block_qkv and vp_block_out need for `shape`
 * (0 if the shape is invalid or not a bf16 layer with H = 16): LN output,
 * X_attn and the FFN hidden layer, 12 KB per token.  256-byte aligned. */
size_t vp_block_workspace_bytes(const vp_shape *shape);
vp_status vp_block_qkv(const vp_shape *shape, const void *X, const int32_t *pos,
                       const vp_block_weights *w, void *Q, void *K, void *V, void *ws,
                       size_t ws_bytes, void *stream);
vp_status vp_block_out(const vp_shape *shape, const void *X, const void *Y,
                       const vp_block_weights *w, void *X_out, void *ws, size_t ws_bytes,
                       void *stream);

/* ---------------------------------------------------------------------------
 * Distillation targets and losses (Section 4.4, Eq.8-11), bf16 layers.  The
 * teacher is the layer with every head running exact softmax attention,
 * A_h = softmax over keys of Q_h K_h^T / sqrt(d) (every query attends all N
 * tokens), written here A_h[k][q].
 *   vp_teacher_targets writes
 *     colmax [H, N] fp32  p^T_{h,k} = max_q A_h[k][q]            (Eq.8)
 *     smax   [H]    fp32  s^attn_h = max_{k,q} A_h[k][q] = max_k p^T_{h,k}
 *     delta  [N, H, d]    Delta^T_h = (A_h - I) V_h in y_dtype     (Eq.10)
 *   (the FULL-head kernels give delta's attention and every query's softmax
 *   normaliser, then one pass over all query-key pairs gives colmax;
 *   arithmetic in fp32, one rounding of delta).
 *   vp_router_loss: per head, Eq.9 with p_bar = colmax / sum_k colmax and
 *     r_bar = r_h, the routing vector of `state` (vp_router_score of the same
 *     K with the same `scale`, 1/sqrt(d) when 0):
 *     loss[h] = KL(p_bar || r_bar) + lambda |smax[h] - max_k r_h(k)|.
 *   vp_latent_loss: per head, Eq.11 over the head's N x d entries:
 *     loss[h] = ||D_hat - D^T||_2 + lambda (1 - cos(D_hat, D^T)); D_hat, D^T
 *     [N, H, d] in `dtype`.
 * Workspaces: vp_teacher_workspace_bytes(shape) for the targets (it includes
 * the routed layer's), vp_loss_workspace_bytes(shape) for either loss.  The
 * losses are deterministic (fixed-order sums). */
size_t vp_teacher_workspace_bytes(const vp_shape *shape);
size_t vp_loss_workspace_bytes(const vp_shape *shape);
vp_status vp_teacher_targets(const vp_shape *shape, const void *Q, const void *K, const void *V,
                             float *colmax, float *smax, void *delta, vp_dtype y_dtype,
                             void *ws, size_t ws_bytes, void *stream);
vp_status vp_router_loss(const vp_shape *shape, const void *K, const vp_router_state *state,
                         float scale, const float *colmax, const float *smax, float lambda,
                         float *loss, void *ws, size_t ws_bytes, void *stream);
vp_status vp_latent_loss(const vp_shape *shape, const void *D_hat, const void *D_t,
                         vp_dtype dtype, float lambda, float *loss, void *ws, size_t ws_bytes,
                         void *stream);

/* ---------------------------------------------------------------------------
 * Token merging before the routed attention (the paper's combination of the
 * layer with ToMe, section "VGGT-Prime & Token Merging", at merging ratios of
 * 75 % and 90 %; the paper gives no steps, these are ToMe's bipartite soft
 * matching run on the layer's inputs):
 *   metric  m_i = bf16(sum over heads of K_{i,h}), the sum in fp32 in head
 *           order;
 *   split   destinations: every token of view 0, the first `nspecial` tokens
 *           of every view, and in views 1.. the patches (the tokens after the
 *           special ones) whose index among the view's patches is a multiple
 *           of g, g the smallest stride that leaves at least M sources;
 *           sources: all other tokens;
 *   match   each source's most similar destination by cosine similarity of
 *           the metric (the first in token order on ties; 0 for a zero
 *           vector);
 *   select  the M most similar sources are merged (the lower token index
 *           first on ties);
 *   rows    the kept tokens (destinations and unmerged sources) in token
 *           order are the nrows = N - M rows of the merged sequence; a merged
 *           source joins its destination's row.
 * The routed layer then runs on the nrows rows as one sequence (S = 1,
 * P = nrows) and vp_tome_unmerge gives every token its row's output.
 *
 * vp_tome_split (host only, no device work): g and nrows for merging M of the
 *   shape's S * P tokens; VP_ERR_INVALID_ARG when M sources do not exist
 *   (M >= 0, nspecial in [0, P)).
 * vp_tome_plan (bf16 K [N, H, 64]) writes, all device int32 / fp32:
 *   row       [N]          the row of every token;
 *   row_start [nrows + 1], members [N]: the tokens of row r are
 *             members[row_start[r] .. row_start[r + 1]): its own kept token
 *             first, then the sources merged into it in token order;
 *   best      [N] (may be null): a source's most similar destination token,
 *             -1 for destinations;
 *   score     [N] (may be null): that cosine similarity (fp32), 0 for
 *             destinations.
 *   Workspace: vp_tome_workspace_bytes(shape) (~190 bytes per token).
 * vp_tome_merge: Xm[r] = mean of X[t] over the members of row r, fp32 sums
 *   in member order, one rounding; X [N, H * 64] -> Xm [nrows, H * 64] in the
 *   shape's dtype.  Member entries outside [0, N) are skipped.
 * vp_tome_merge_qkv: vp_tome_merge of Q, K and V (bf16) in one pass over the
 *   member lists (the same sums, in the same order).
 * vp_tome_unmerge: Y[t] = Ym[row[t]] ([nrows, H * 64] -> [N, H * 64], the
 *   shape's dtype); a row outside [0, nrows) gives zeros.
 * All three enqueue on `stream`, allocate nothing and are deterministic
 * (fixed-order sums, no float atomics). */
vp_status vp_tome_split(const vp_shape *shape, int64_t M, int32_t nspecial, int64_t *g,
                        int64_t *nrows);
size_t vp_tome_workspace_bytes(const vp_shape *shape);
vp_status vp_tome_plan(const vp_shape *shape, const void *K, int64_t M, int32_t nspecial,
                       int32_t *row, int32_t *row_start, int32_t *members, int32_t *best,
                       float *score, void *ws, size_t ws_bytes, void *stream);
vp_status vp_tome_merge(const vp_shape *shape, const void *X, int64_t nrows,
                        const int32_t *row_start, const int32_t *members, void *Xm,
                        void *stream);
vp_status vp_tome_merge_qkv(const vp_shape *shape, const void *Q, const void *K, const void *V,
                            int64_t nrows, const int32_t *row_start, const int32_t *members,
                            void *Qm, void *Km, void *Vm, void *stream);
vp_status vp_tome_unmerge(const vp_shape *shape, const void *Ym, int64_t nrows,
                          const int32_t *row, void *Y, void *stream);

/* Static description of a status code. */
const char *vp_status_string(vp_status s);

/* Message of the last VP_ERR_HIP on the calling thread ("" if none). */
const char *vp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* VGGT_PRIME_H */

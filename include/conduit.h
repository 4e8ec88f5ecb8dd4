/*
 * conduit.h - C ABI of the Conduit refresh step for reused visual KV caches
 * (gfx950 / MI355X).
 *
 * The paper's refresh step, per request:
 *   1. budget          k = floor(r * N_vis) over visual tokens only
 *                      (Sec. 3.1 Eq. 2; Algorithm 1 first step and k = 0 exit);
 *   2. scoring pass    per scored layer: softmax attention of the span queries
 *                      over the cached keys, head- and query-mean over the
 *                      visual columns (Sec. 3.3 Eq. 6), times the cached value
 *                      norm (Eq. 7), accumulated over layers  -> conduit_score;
 *   3. reweighting     image means g_j, coefficients c_j (Sec. 3.4 Eq. 8-9),
 *                      composite score (Sec. 3.5 Eq. 10) and one global top-k
 *                      (Eq. 11)                              -> conduit_select_topk;
 *   4. recompute       per layer: the selected rows' fresh K/V are written
 *                      into the cache, all other visual rows are reused
 *                      (Sec. 3; Sec. 4.1 cache-reuse protocol)
 *                                                            -> conduit_scatter_kv;
 *                      then each selected row attends causally over the
 *                      merged fresh/stale prefix             -> conduit_refresh_attn.
 *
 * Conventions shared by every entry point:
 *   - Tensors are caller-owned DEVICE memory unless marked HOST.  The library
 *     allocates nothing: scratch comes in through (ws, ws_bytes), sized by the
 *     matching *_workspace_bytes query.  No state is kept apart from a
 *     thread-local error string, so calls on different streams may run
 *     concurrently as long as they do not share output or workspace memory.
 *   - Every call only enqueues work on `stream` (a hipStream_t; NULL is the
 *     default stream) and never synchronises.  Device faults surface at the
 *     caller's next synchronisation.
 *   - Every argument is checked on the host before anything is enqueued.  A
 *     non-OK status means nothing was enqueued and no output was touched;
 *     conduit_last_error() then describes the problem.  With no usable GPU a
 *     valid call returns CONDUIT_ERR_HIP.
 *   - Caches are token-major: element (token t, KV head h, dim e) sits at
 *     base[row(t) * stride + h * head_dim + e], with row(t) = t for a
 *     contiguous cache and the block-table lookup of conduit_kv for a paged
 *     one.  Queries and outputs are dense
 *     [rows][n_q_heads][head_dim].  bf16 is IEEE binary32's top 16 bits.
 *     Device pointers must be 16-byte aligned and strides a multiple of
 *     16 bytes and below 32 MiB (CONDUIT_ERR_UNSUPPORTED otherwise).
 *   - Query head h reads KV head h / (n_q_heads / n_kv_heads).
 *   - Supported: head_dim 64 or 128; n_kv_heads <= 256; CONDUIT_BF16 (MFMA
 *     kernels, fp32 accumulation) or CONDUIT_F32 (fp32 throughout).  The bf16
 *     attention plans at most 4,096 blocks of (row, query head) pairs per KV
 *     head: rows * n_q_heads / n_kv_heads <= 524,288 for conduit_score and
 *     <= 1,048,576 for conduit_refresh_attn (CONDUIT_ERR_UNSUPPORTED past it);
 *     bf16 scoring also needs the span's queries below 2^31 bytes.
 *   - Results are bitwise reproducible run to run (no floating-point atomics).
 */
#ifndef CONDUIT_H
#define CONDUIT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CONDUIT_OK = 0,
  CONDUIT_ERR_INVALID_ARG = 1,   /* bad pointer, size, range or layout          */
  CONDUIT_ERR_UNSUPPORTED = 2,   /* valid but no kernel (head_dim, dtype, ...)  */
  CONDUIT_ERR_WORKSPACE = 3,     /* ws_bytes below the *_workspace_bytes query  */
  CONDUIT_ERR_HIP = 4            /* a HIP runtime call or launch failed         */
} conduit_status;

typedef enum { CONDUIT_F32 = 0, CONDUIT_BF16 = 1 } conduit_dtype;

/* Domain of the scoring softmax (Eq. 6).  CAUSAL_ROW: each span token's full
 * causal row (changed prefix, separators, every image's cached visual keys and
 * span keys up to itself), then the visual columns are kept; this is the
 * attention the model itself computes for the span.  VISUAL_ONLY: renormalised
 * over the visual keys alone. */
typedef enum { CONDUIT_NORM_CAUSAL_ROW = 0, CONDUIT_NORM_VISUAL_ONLY = 1 } conduit_norm;

/* Aggregation of the cached-key attention over span tokens and query heads. */
typedef enum {
  CONDUIT_AGG_MEAN = 0,   /* Eq. 6: mean (the deployed policy)                   */
  CONDUIT_AGG_RMS = 1     /* Eq. 4: root-mean-square, the squared-error surrogate */
} conduit_agg;

/* Selection rule of conduit_select_topk. */
typedef enum {
  CONDUIT_RANK_COMPOSITE = 0,  /* Eq. 10-11: global top-k of (s/|L|) * c_pi(t)        */
  CONDUIT_RANK_ATTENTION = 1,  /* value norm dropped: global top-k of (A/|L|) * c_pi(t) */
  CONDUIT_RANK_EXPLICIT = 2    /* quotas k_j ~ c_j n_j, then the k_j largest s of image j */
} conduit_rule;

#define CONDUIT_MAX_IMAGES 256
#define CONDUIT_MAX_LAYERS 1024  /* layers of one multi-layer call */

/* One layer's KV cache, contiguous or paged.
 *
 * Contiguous (block_table NULL, page_size = n_pages = 0): token t is row t of
 * k and v.
 *
 * Paged (the block-table KV storage of a serving engine, Sec. 4.3): k and v
 * hold n_pages physical pages of page_size rows each; logical token t lives
 * in row block_table[t / page_size] * page_size + t % page_size.  page_size
 * is a power of two from 64 to 2^20 (a 64-key attention tile then never
 * crosses a page; smaller powers of two return CONDUIT_ERR_UNSUPPORTED).
 * block_table is device int32 [ceil(n_ctx / page_size)], caller-owned and
 * read by the kernels; an entry outside [0, n_pages) is clamped into it (the
 * results are then meaningless, but no access leaves the pages).  Pages may
 * be shared between tables or unused. */
typedef struct {
  void *k;                /* device [rows][n_kv_heads][head_dim], dtype; rows =
                             n_ctx (contiguous) or n_pages * page_size (paged) */
  void *v;                /* device, same layout                                 */
  int64_t k_stride;       /* elements between consecutive rows of k,
                             >= n_kv_heads * head_dim                            */
  int64_t v_stride;       /* same for v                                          */
  int32_t n_ctx;          /* tokens in the cache (sequence positions 0..n_ctx-1) */
  int32_t n_q_heads;      /* H_q; a multiple of n_kv_heads                       */
  int32_t n_kv_heads;     /* H_kv                                                */
  int32_t head_dim;       /* 64 or 128                                           */
  int32_t dtype;          /* conduit_dtype                                       */
  int32_t page_size;      /* paged: tokens per page; contiguous: 0               */
  const int32_t *block_table; /* paged: device [ceil(n_ctx / page_size)]; else NULL */
  int32_t n_pages;        /* paged: physical pages in k and v; contiguous: 0    */
} conduit_kv;

/* The visual-token sets of Eq. 1: K images, each one contiguous run of
 * sequence positions, in ascending order and not overlapping.  Visual token t
 * (0 <= t < n_vis) is numbered image by image; image j holds tokens
 * img_off[j] .. img_off[j+1]-1 at positions img_pos[j] .. img_pos[j]+n_j-1.
 * HOST memory, read during the call only. */
typedef struct {
  int32_t n_images;       /* 1 .. CONDUIT_MAX_IMAGES                            */
  int32_t n_vis;          /* == img_off[n_images]                               */
  const int32_t *img_pos; /* HOST [n_images]                                    */
  const int32_t *img_off; /* HOST [n_images + 1], img_off[0] = 0, strictly increasing */
} conduit_images;

/* Eq. 2: k = floor(r_num * n_vis / r_den), in exact integer arithmetic.
 * Returns -1 if n_vis < 0, r_den <= 0, r_num < 0 or r_num > r_den. */
int64_t conduit_budget(int64_t n_vis, int64_t r_num, int64_t r_den);

/* ------------------------------------------------------------------------ *
 * Scoring pass for one scored layer (Sec. 3.3 Eq. 6-7; the scoring loop of
 * Algorithm 1; App. A.2 scoring forward pass).
 *
 * q        device [n_q][n_q_heads][head_dim], kv->dtype: the span queries; span
 *          token i sits at position q_pos0 + i and sees keys 0 .. q_pos0 + i.
 *          Requires q_pos0 + n_q <= kv->n_ctx and every image before q_pos0.
 * scale    logit scale (1/sqrt(head_dim) for standard attention), > 0.
 * row_lse_in   nullable device [n_q][n_q_heads] fp32: natural-log log-sum-exp of
 *          each span row over the `norm` domain, e.g. from the model's own
 *          attention of the span.  When given, the row-statistics pass is
 *          skipped.
 * row_lse_out  nullable device [n_q][n_q_heads] fp32: the row log-sum-exp.
 * agg      CONDUIT_AGG_MEAN: a_t is the mean of the attention probabilities over
 *          (span token, query head) (Eq. 6); CONDUIT_AGG_RMS: their root mean
 *          square (Eq. 4's surrogate).
 * vnorm_in nullable device [n_vis] fp32: the layer's value norms ||V_t|| as made
 *          by conduit_value_norms when the cache was built (Sec. 4.3).  When
 *          given, the cached V is not read.
 * s_acc, a_acc device [n_vis] fp32, in/out.  With accumulate = 0 they are
 *          overwritten with a_t * ||V_t|| and a_t; with accumulate = 1 these are
 *          added to the current contents.  Calling once per scored layer in
 *          layer order gives sum_l a_t^(l) ||V_t^(l)|| and sum_l a_t^(l).  Any
 *          subset of a model's layers may be scored this way (|L| is then the
 *          count passed to conduit_select_topk).
 * a_out, vnorm_out  nullable device [n_vis] fp32: this layer's a_t and ||V_t||
 *          (the norm of the n_kv_heads * head_dim concatenated cached value).
 * ws       device workspace of at least conduit_score_workspace_bytes(...).
 * ------------------------------------------------------------------------ */
size_t conduit_score_workspace_bytes(const conduit_kv *kv, int32_t n_q, const conduit_images *img);

conduit_status conduit_score(const conduit_kv *kv, const void *q, int32_t n_q, int32_t q_pos0,
                             const conduit_images *img, conduit_norm norm, conduit_agg agg,
                             float scale, const float *row_lse_in, float *row_lse_out,
                             const float *vnorm_in, float *s_acc, float *a_acc, int32_t accumulate,
                             float *a_out, float *vnorm_out,
                             void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * Allocation-free scoring pass: conduit_score with the library's own fixed
 * device scratch in place of (ws, ws_bytes).  For callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the call itself makes no hipMalloc,
 * hipFree or other allocating call; every other argument, the kernels and
 * the results are those of conduit_score, bit for bit.
 *
 * The scratch is one array of CONDUIT_SCORE_NOALLOC_MAX_BYTES per GPU the
 * library is loaded on, held until the process ends; its address is looked
 * up on the first call on each device (with that device current).  Every
 * call on a GPU shares that GPU's array and leaves its contents behind (no
 * part of it needs to start at zero: each launch writes what the next one
 * reads), so calls that overlap on one GPU (on different streams, or from
 * different threads) race and must be serialised by the caller.
 *
 * Errors: those of conduit_score, and CONDUIT_ERR_UNSUPPORTED when
 * conduit_score_workspace_bytes(kv, n_q, img) exceeds
 * CONDUIT_SCORE_NOALLOC_MAX_BYTES (nothing is enqueued; use conduit_score).
 * With kernel timing enabled, the timing events are created on first use.
 * ------------------------------------------------------------------------ */
#define CONDUIT_SCORE_NOALLOC_MAX_BYTES ((size_t)16 << 20)

conduit_status conduit_score_noalloc(const conduit_kv *kv, const void *q, int32_t n_q, int32_t q_pos0,
                                     const conduit_images *img, conduit_norm norm, conduit_agg agg,
                                     float scale, const float *row_lse_in, float *row_lse_out,
                                     const float *vnorm_in, float *s_acc, float *a_acc, int32_t accumulate,
                                     float *a_out, float *vnorm_out, hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * The scoring pass over several layers of one request (Eq. 6-7 summed over
 * the scored layers L of Algorithm 1): conduit_score of every layer in turn,
 * accumulating into s_acc and a_acc, with the layers' work in a few launches
 * (up to 16 layers in each).  The results equal those of the per-layer calls
 * up to rounding: the layers are added in order with the same arithmetic,
 * but a launch of several layers may cut each layer's row statistics into
 * fewer key splits (the grid is filled by the layers instead), which changes
 * the rounding of the row log-sum-exps (relative differences near 1e-7).
 *
 * kvs       HOST [n_layers] descriptors shaped alike (see the multi-layer
 *           merge below); q: HOST [n_layers] span queries, each as q above.
 * vnorm_in  nullable HOST [n_layers] array of nullable value-norm tables.
 * accumulate  0: the first layer overwrites s_acc / a_acc; 1: all add.
 * ws        conduit_score_layers_workspace_bytes(kvs, n_q, img, n_layers).
 * No row LSE, per-layer a_t or norm outputs (use conduit_score for those).
 * ------------------------------------------------------------------------ */
size_t conduit_score_layers_workspace_bytes(const conduit_kv *kv, int32_t n_q, const conduit_images *img,
                                           int32_t n_layers);

conduit_status conduit_score_layers(const conduit_kv *kvs, int32_t n_layers, const void *const *q, int32_t n_q,
                                    int32_t q_pos0, const conduit_images *img, conduit_norm norm,
                                    conduit_agg agg, float scale, const float *const *vnorm_in, float *s_acc,
                                    float *a_acc, int32_t accumulate, void *ws, size_t ws_bytes,
                                    hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * Value-norm table of one layer (Eq. 7's proxy; Sec. 4.3: the norms depend on
 * the cache only, so storing one scalar per visual token and layer when the
 * cache is built preserves the scores exactly and removes the V reads from
 * every later scoring pass).
 *
 * vnorm_out  device [img->n_vis] fp32: ||V_t|| over the n_kv_heads * head_dim
 *            concatenated cached value of each visual token, in visual order.
 * ------------------------------------------------------------------------ */
conduit_status conduit_value_norms(const conduit_kv *kv, const conduit_images *img, float *vnorm_out,
                                   hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * Image reweighting and global top-k (Sec. 3.4 Eq. 8-9, Sec. 3.5 Eq. 10-11,
 * the tail of Algorithm 1).
 *
 * s_acc, a_acc  device [n_vis] fp32: the layer sums produced by conduit_score.
 * n_layers      |L| >= 1, the number of layers accumulated.
 * lambda        reweighting strength in [0, 1] (1 in the paper's main setting;
 *               0 ranks by s alone, the "global top-k" of App. D).
 *               c_j = (1 - lambda) + lambda * g_j / g_bar, exactly 1 when
 *               g_j = g_bar (so always with one image) or when g_bar = 0.
 * rule          CONDUIT_RANK_COMPOSITE: the global top-k of
 *               s_hat_t = (s_acc_t / n_layers) * c_pi(t) (Eq. 10-11).
 *               CONDUIT_RANK_ATTENTION: the same with a_acc in place of s_acc
 *               (the value-norm factor dropped, Table 5's factor ablation).
 *               CONDUIT_RANK_EXPLICIT: quotas k_j proportional to c_j * n_j
 *               (largest remainder, float32 in image order, capped at n_j
 *               with the surplus re-apportioned, ties to the lower image; all
 *               weights zero falls back to n_j), then the k_j largest s_acc of
 *               each image (App. D's explicit reweighting).
 * k             budget, 0 <= k <= n_vis.  Ties in the ranked score go to the
 *               lower visual index.  k = 0 only clears mask_out.
 * idx_out       device [k] int32: selected visual indices, ascending.
 * pos_out       device [k] int32: their sequence positions, ascending.
 * mask_out      nullable device [n_vis] uint8: the refresh mask M.
 * shat_out      nullable device [n_vis] fp32: the ranked score (composite and
 *               explicit rules: (s_acc_t / n_layers) * c_pi(t); attention
 *               rule: (a_acc_t / n_layers) * c_pi(t)).
 * c_out         nullable device [n_images] fp32: the coefficients c_j.
 * quota_out     nullable device [n_images] int32: the quotas k_j
 *               (CONDUIT_RANK_EXPLICIT only; ignored otherwise).
 * ws            256-byte aligned device workspace of at least
 *               conduit_select_workspace_bytes(n_vis, n_images) bytes when
 *               k > 0 (it holds s_hat when shat_out is NULL, and for
 *               16,384 < n_vis <= 131,072 the exchange area of the
 *               multi-workgroup top-k: barrier flags, which the call clears
 *               itself, partial sums and histograms).  Its contents need no
 *               initialisation and are not meaningful afterwards.
 * ------------------------------------------------------------------------ */
size_t conduit_select_workspace_bytes(int32_t n_vis, int32_t n_images);

conduit_status conduit_select_topk(const float *s_acc, const float *a_acc, int32_t n_layers,
                                   const conduit_images *img, float lambda, conduit_rule rule,
                                   int32_t k, int32_t *idx_out, int32_t *pos_out, uint8_t *mask_out,
                                   float *shat_out, float *c_out, int32_t *quota_out,
                                   void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * Cache merge for one layer (Sec. 3: selected rows are recomputed, all other
 * cached visual entries are reused).  For each i < k, token pos[i] of kv->k and
 * kv->v is replaced by row i of k_new / v_new, in place.  The rows may mix
 * the selected visual tokens with the request's text tokens (changed prefix,
 * separators, span), which are processed normally (Sec. 3.1).
 *
 * pos           device [k] int32, distinct, each in [0, kv->n_ctx), any order
 *               (device-side precondition: a position outside the range is
 *               clamped into it, so no access leaves the cache; repeated
 *               positions race).
 * k_new, v_new  device [k][n_kv_heads][head_dim] dense, kv->dtype.
 * k_old_out, v_old_out  nullable device [k][n_kv_heads][head_dim]: receive the
 *               replaced (stale) rows, so the merge can be undone.
 * k = 0 enqueues nothing and leaves the cache untouched.
 * ------------------------------------------------------------------------ */
conduit_status conduit_scatter_kv(const conduit_kv *kv, const int32_t *pos, int32_t k,
                                  const void *k_new, const void *v_new,
                                  void *k_old_out, void *v_old_out, hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * Refresh attention for one layer: causal attention of the selected rows over
 * the merged cache (the selective recompute of Sec. 3 and Sec. 4.1).  Row i
 * sits at position pos[i] and attends to keys 0 .. pos[i] of kv (already
 * merged by conduit_scatter_kv on the same stream), itself included.  The rows
 * may include the request's text tokens, so one launch covers the whole
 * per-layer recompute attention (selected visual rows and text rows).
 *
 * q_sel   device [k][n_q_heads][head_dim], kv->dtype: fresh queries, row i for
 *         pos[i].
 * pos     device [k] int32, each in [0, kv->n_ctx), any order (device-side
 *         precondition: for a position outside the range no access leaves
 *         the cache, but that row's output is meaningless).
 *         Rows are blocked in the given order, so ascending runs (e.g. the
 *         selected rows followed by the text rows) keep blocks' key ranges
 *         tight.
 * o_out   device [k][n_q_heads][head_dim], kv->dtype (bf16 rounded to nearest
 *         even from fp32 accumulation).
 * lse_out nullable device [k][n_q_heads] fp32: natural-log log-sum-exp.
 * ws      conduit_refresh_workspace_bytes(kv, k) bytes, 256-byte aligned: the
 *         work plan and split partials (bf16), or the key splits' partials
 *         when an fp32 call has few rows (0 bytes otherwise).
 * k = 0 enqueues nothing.
 * ------------------------------------------------------------------------ */
size_t conduit_refresh_workspace_bytes(const conduit_kv *kv, int32_t k);

conduit_status conduit_refresh_attn(const conduit_kv *kv, const void *q_sel, const int32_t *pos,
                                    int32_t k, float scale, void *o_out, float *lse_out,
                                    void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * The per-layer recompute of Sec. 3 in one call: the cache merge of
 * conduit_scatter_kv (without the copy of the stale rows) followed by
 * conduit_refresh_attn over the merged cache, with the same arguments and
 * results as the two calls in that order.  For bf16 the refresh's work plan
 * and the merge run in one launch (they are independent; the attention needs
 * both), which saves a launch and the plan's time on the critical path.
 *
 * Arguments as in conduit_scatter_kv and conduit_refresh_attn; ws sized by
 * conduit_refresh_workspace_bytes(kv, k).  Errors: those of the two calls,
 * all checked before anything is enqueued.  k = 0 enqueues nothing.
 * ------------------------------------------------------------------------ */
conduit_status conduit_merge_refresh_attn(const conduit_kv *kv, const int32_t *pos, int32_t k,
                                          const void *k_new, const void *v_new, const void *q_sel,
                                          float scale, void *o_out, float *lse_out, void *ws,
                                          size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * The merge and the refresh attention of several layers of one request at
 * once (the recompute of Sec. 3 runs in every layer with the same selection
 * M, Algorithm 1).  The merged caches equal those of conduit_scatter_kv called
 * layer by layer, bit for bit; the attention computes what
 * conduit_refresh_attn computes per layer, to the same tolerance but not bit
 * for bit (with many layers in one launch the plan cuts the key ranges into
 * fewer splits).  The work of up to 16 layers goes into each launch, and the
 * refresh builds its work plan once (it depends on the rows only).
 *
 * kvs        HOST [n_layers] descriptors, 1 <= n_layers <= CONDUIT_MAX_LAYERS;
 *            every layer shaped like kvs[0] (dtype, heads, head_dim, n_ctx,
 *            strides, block table, page size and pool): only k and v differ,
 *            else CONDUIT_ERR_INVALID_ARG.
 * k_new, v_new, q_sel, o_out  HOST [n_layers] arrays of the per-layer device
 *            buffers described above (16-byte aligned).
 * lse_out    nullable HOST [n_layers] array; entries may be NULL.
 * pos, k     shared by every layer, as above.
 * ws         conduit_refresh_layers_workspace_bytes(kvs, k, n_layers) bytes
 *            (the plan and the split partials of 16 layers).
 * ------------------------------------------------------------------------ */
conduit_status conduit_scatter_kv_layers(const conduit_kv *kvs, int32_t n_layers, const int32_t *pos, int32_t k,
                                         const void *const *k_new, const void *const *v_new,
                                         hipStream_t stream);

size_t conduit_refresh_layers_workspace_bytes(const conduit_kv *kv, int32_t k, int32_t n_layers);

conduit_status conduit_refresh_attn_layers(const conduit_kv *kvs, int32_t n_layers, const void *const *q_sel,
                                           const int32_t *pos, int32_t k, float scale, void *const *o_out,
                                           float *const *lse_out, void *ws, size_t ws_bytes,
                                           hipStream_t stream);

/* ------------------------------------------------------------------------ *
 * Residual value-write error of a refresh set, a quality diagnostic of a
 * selection (the local model of Eq. 3; App. D.1 isotropic Monte Carlo
 * estimator; App. D.3 projected error).  For displacement sample m, span row i
 * (position q_pos0 + i) and query head h it computes
 *     err[m][i][h] = || sum over visual t with refreshed[t] == 0 of
 *                       alpha_{i,h,t} xi^(m)_t[h / G] ||^2
 * where alpha is the cached-key attention of the scoring pass, normalised by
 * the row log-sum-exp row_lse_in (conduit_score's row_lse_out; its norm
 * decides causal-row or visual-only normalisation), and xi_t[kv] is the
 * KV-head-kv slice of the displacement:
 *   z != NULL (isotropic):  xi^(m)_t = kappa * ||V_t|| / sqrt(n_kv_heads *
 *       head_dim) * z[m][t], so E ||xi_t||^2 = kappa^2 ||V_t||^2 when z holds
 *       standard normal draws; App. D.1 averages err over m (M = 5).
 *   z == NULL (projected):  xi_t = V_t, the residual when every stale visual
 *       value is set to zero (App. D.3); n_samples must be 1.
 * The attention output map is the identity (the library holds no weights).
 *
 * q           device [n_q][n_q_heads][head_dim], kv->dtype: span queries.
 * row_lse_in  device [n_q][n_q_heads] fp32, natural-log log-sum-exp.
 * refreshed   device [n_vis] uint8: nonzero = in the refresh set T (e.g.
 *             conduit_select_topk's mask_out).
 * z           nullable device [n_samples][n_vis][n_kv_heads][head_dim],
 *             kv->dtype, 16-byte aligned.
 * err_out     device [n_samples][n_q][n_q_heads] fp32.
 * ws          256-byte aligned, conduit_residual_workspace_bytes(kv, n_q,
 *             img, n_samples, z != NULL) bytes.
 * Errors: CONDUIT_ERR_INVALID_ARG (NULL row_lse_in / refreshed / err_out,
 * kappa not finite and > 0 with z, n_samples != 1 without z, ...),
 * CONDUIT_ERR_UNSUPPORTED if n_samples * n_kv_heads > 65535.
 * ------------------------------------------------------------------------ */
size_t conduit_residual_workspace_bytes(const conduit_kv *kv, int32_t n_q, const conduit_images *img,
                                        int32_t n_samples, int32_t iso);

conduit_status conduit_residual_error(const conduit_kv *kv, const void *q, int32_t n_q, int32_t q_pos0,
                                      const conduit_images *img, float scale, const float *row_lse_in,
                                      const uint8_t *refreshed, const void *z, int32_t n_samples,
                                      float kappa, float *err_out, void *ws, size_t ws_bytes,
                                      hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kernel timing, a tracing aid.  While enabled on the calling thread, every
 * kernel launch made by the entry points above is bracketed by two HIP
 * events recorded on the caller's stream; the first CONDUIT_PROFILE_MAX
 * launches are kept.  conduit_profile_read(i, ...) waits for launch i to
 * finish and returns its kernel's name (a static string) and duration in
 * milliseconds.  Enabling clears the record; disabling keeps it for reading.
 * The events add a small gap between launches, so leave timing off outside
 * measurement.  Errors: CONDUIT_ERR_INVALID_ARG for i out of range or NULL
 * outputs, CONDUIT_ERR_HIP if an event call fails.
 * ------------------------------------------------------------------------ */
#define CONDUIT_PROFILE_MAX 4096

conduit_status conduit_profile_enable(int32_t enabled);
int32_t conduit_profile_count(void);
conduit_status conduit_profile_read(int32_t i, const char **name, float *ms);

/* Status name, e.g. "CONDUIT_ERR_INVALID_ARG". */
const char *conduit_status_str(conduit_status status);

/* Detail for the calling thread's last non-OK return ("" if none). */
const char *conduit_last_error(void);

/* Library version string. */
const char *conduit_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CONDUIT_H */

/*
 * moddit.h -- C ABI of the MI355X (gfx950) MOD-DiT hot path.
 *
 * MOD-DiT (arXiv 2601.11641) predicts, for every attention head and every
 * query block of a video-DiT attention layer, which key/value blocks to keep,
 * from a mixture-of-distributions (MOD) linear model of the block-level
 * attention statistic (Section 4.2, Eq. 3/Eq. 4) fitted at early denoising
 * steps and extrapolated linearly across steps (Section 5.2), and then runs
 * attention over the kept blocks only (Eq. 1).  This library implements that
 * path on one GPU:
 *
 *   mod_collect_stats        dense warm-up step: pool Q/K per block, build the
 *                            pooled block-mass statistic G, fit the MOD
 *                            coefficients X = [c, d, e] (Eq. 4, min-norm)
 *   mod_predict_block_mask   sparse step: optionally re-anchor (fit again),
 *                            extrapolate c and d (Section 5.2), score blocks and
 *                            select per query block (Section 5.3)
 *   mod_block_sparse_attn_fwd  softmax attention over the kept blocks (Eq. 1)
 *   mod_update_stats         (statistic 1) after a step's attention: the
 *                            sparsity statistic of Eq. 2 on the blocks it
 *                            computed, reconstruction of Eq. 5, fit
 *
 * Conventions shared by every entry point
 *   - Q, K, V, O are bfloat16, contiguous [B, H, L, d] (d fastest), device
 *     memory owned by the caller, 16-byte aligned.  L is the token count and
 *     d the head dimension; blocks are `block` consecutive tokens, the last
 *     block may be short (n = ceil(L / block) blocks).
 *   - Tokens are frame-first; `frame_tokens` tokens make one latent frame and
 *     each frame defines one block-diagonal region (Appendix B.3).
 *   - Token-type-aware masking (Section 3): the last `text_tokens` tokens of
 *     the sequence may be text tokens that attend to, and are attended by,
 *     every token.  The MOD statistic, fit and prediction cover the
 *     Lv = L - text_tokens video tokens (nv = ceil(Lv / block) blocks); the
 *     masks cover all n blocks.  A block holding any text token is a text
 *     block (the first is Lv / block): its row keeps every block, and every
 *     row keeps it.  In a block holding both video and text tokens (Lv not a
 *     multiple of block) the video part is pooled with the video tokens.
 *   - Supported: d in {64, 128}, block in {64, 128}, 0 <= text_tokens < L,
 *     2 <= Lv / frame_tokens, Lv % frame_tokens == 0, n <= 4096.  Other
 *     shapes: MOD_ERR_UNSUPPORTED.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL is the
 *     default stream) unless stated otherwise.  Arguments are validated on
 *     the host before anything is enqueued; on error nothing is enqueued and
 *     mod_last_error() holds a message (thread-local).
 *   - No exception crosses the ABI and nothing aborts.
 *   - A mod_stats handle is used by one thread and one stream at a time.
 */
#ifndef MODDIT_H
#define MODDIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MOD_OK = 0,
    MOD_ERR_INVALID_ARG = 1,   /* null pointer, non-positive size, bad budget   */
    MOD_ERR_UNSUPPORTED = 2,   /* shape outside the supported set                */
    MOD_ERR_BAD_STATE = 3,     /* step order / predict before any collected step */
    MOD_ERR_HIP = 4,           /* HIP runtime or kernel-launch error             */
    MOD_ERR_NOMEM = 5          /* device or host allocation failed               */
} mod_status;

/* Shape of one attention layer. */
typedef struct {
    int B;             /* batch                                  */
    int H;             /* heads                                  */
    int L;             /* tokens per sequence                    */
    int d;             /* head dimension                         */
    int block;         /* tokens per block (the paper's B)       */
    int frame_tokens;  /* tokens per latent frame                */
    int text_tokens;   /* text tokens after the video (0: none)  */
} mod_shape;

/* Predictor schedule (Algorithm 1 hyper-parameters). */
typedef struct {
    int warmup_m;      /* m: dense warm-up steps (Section 5)                 */
    int delta_t;       /* re-anchor interval; <= 0 never re-anchors          */
    float tau_e;       /* block-diagonal threshold (Section 5.3)            */
    int anchor_rule;   /* 0: re-anchor at t = m + i*delta_t, i >= 1 (the
                          prediction steps of Section 5); 1: at t % delta_t == 0
                          (Algorithm 1)                                      */
    int statistic;     /* 0: the pooled block-mass statistic, fitted from Q, K
                          (mod_collect_stats, and inside mod_predict_block_mask
                          at re-anchor steps); 1: the attention sparsity
                          statistic of Eq. 2 with the reconstruction of Eq. 5,
                          fitted from the attention a step computed
                          (mod_update_stats only)                            */
    float eta;         /* statistic 1: sparsity threshold of Eq. 2, > 0     */
} mod_params;

typedef enum { MOD_BUDGET_TOPK = 0, MOD_BUDGET_MASS = 1, MOD_BUDGET_PATTERN = 2 } mod_budget_mode;

/* Sparsity budget.
 *   TOPK: keep k = clamp(ceil(density * n - 1e-6), 1, n) blocks per query
 *         block (density taken at float precision), the forced block-diagonal
 *         blocks counted first.
 *   MASS: keep the forced blocks plus the shortest score-ordered prefix of
 *         the others whose positive score mass reaches `mass` of the row's
 *         total positive mass (at least one block).
 *   PATTERN (Section 5.3, the mask as printed): per head, rank the 3n - 1
 *         predicted intensities of the parallel-diagonal and vertical
 *         patterns together (float precision, ties by pattern index:
 *         diagonals j - i = -(n-1) .. n-1 first, then columns), keep the
 *         `patterns` largest; block (i, j) is kept iff its diagonal or its
 *         column is kept, or it is forced.  The ranking uses the
 *         minimum-norm gauge of the fit.  A row that no kept pattern reaches
 *         may be empty (its attention output is zero). */
typedef struct {
    int mode;          /* mod_budget_mode              */
    float density;     /* TOPK: in (0, 1]              */
    float mass;        /* MASS: in (0, 1]              */
    int patterns;      /* PATTERN: K in [1, 3nv - 1]   */
} mod_budget;

typedef struct mod_stats mod_stats;   /* opaque, library-owned */

/* n = ceil(L / block), the blocks of the whole sequence (the masks' size);
 * 0 for a null or invalid shape. */
int mod_num_blocks(const mod_shape* shape);

/* |X| = 3nv - 1 + F coefficients per head (Eq. 4: 2nv-1 diagonals, nv
 * verticals, F = Lv / frame_tokens frame regions, over the nv video
 * blocks); 0 if invalid. */
int mod_num_coeffs(const mod_shape* shape);

/* Create the predictor state of one layer.  Builds, on the host in fp64, the
 * closed-form normal matrix of the MOD least-squares problem (Appendix B.4)
 * reduced to its Schur complement, factors and inverts it once, allocates
 * the device buffers and uploads the tables.  Synchronous.  On success *out
 * owns about (2*B*H*n*d + B*H*n*n + 8*B*H*n) * 8 bytes of device memory. */
mod_status mod_stats_create(const mod_shape* shape, const mod_params* params,
                            mod_stats** out);

/* Release the handle and its device memory (waits for the device).  NULL is
 * accepted. */
mod_status mod_stats_destroy(mod_stats* stats);

/* Dense warm-up step `step` (Algorithm 1, warm-up phase): fit the MOD
 * coefficients (Eq. 4) on the pooled block-mass statistic of q, k
 * ([B,H,L,d] bf16 device pointers) and record (step, X) as the newest of the
 * two anchors kept.  Steps must strictly increase across collect, update and
 * predict calls (else MOD_ERR_BAD_STATE).  Statistic 0 only (else
 * MOD_ERR_BAD_STATE). */
mod_status mod_collect_stats(mod_stats* stats, const void* q, const void* k, int step,
                             void* stream);

/* Statistic 1 (Section 4.1, Eq. 2 and Eq. 5; Algorithm 1): after the
 * attention of step `step` -- a dense warm-up step with full lists, or a
 * re-anchor step with that step's predicted lists -- record the anchor of
 * that step.  For every listed block (i, j) the informativeness
 *   I(i, j) = 1 - S(i, j) = fraction of the probabilities
 *             exp(scale * Q_p.K_q - lse_p), p in i, q in j, that reach eta
 * (S of Eq. 2 over the block's valid entries; decided in fp32 as
 * s >= (lse_p + log(eta)) / scale, s the fp32 product of the bf16 inputs)
 * replaces the stored value; unlisted blocks keep their previous value
 * (Eq. 5 at block level).  The MOD model is then fitted to the whole stored
 * map and (step, X) becomes the newest anchor.  The first update should
 * list every block (the stored map starts at zero).  With text tokens the
 * map covers the video blocks (i, j < nv) while the lists, the lse and the
 * probabilities cover the whole sequence.
 * q, k: [B,H,L,d] bf16 device (the step's inputs, scaled as in the
 * attention call: scale = 1/sqrt(d)); lse: [B,H,L] fp32 device, the lse the
 * attention forward returned for these lists; kv_idx, kv_cnt: the lists of
 * that call (layout of mod_predict_block_mask).  Entries outside [0, n) are
 * skipped.  `step` must follow the previous call's step, or equal it when
 * that call was the predict of this step (else MOD_ERR_BAD_STATE).
 * Statistic 1 only (else MOD_ERR_BAD_STATE). */
mod_status mod_update_stats(mod_stats* stats, const void* q, const void* k, const float* lse,
                            const int32_t* kv_idx, const int32_t* kv_cnt, int step, void* stream);

/* Sparse step `step` (Algorithm 1, main phase; Sections 5.2-5.3).
 * On the first call the block-diagonal gate of every head is fixed from the
 * anchors held (gate on iff min over anchors of mean_f e_f > tau_e).  With
 * statistic 0, if `step` is a re-anchor step, q and k are pooled and fitted
 * first (else they are not read and may be NULL); with statistic 1 anchors
 * come from mod_update_stats only and q, k are never read.  Then c and d are extrapolated to `step`
 * from the two newest anchors (zero slope with one anchor) and every query
 * block i of every head selects key blocks by the score
 *   sigma(i, j) = nv * (c~[j - i] + d~[j])
 * ranked at float precision, ties to the smaller j, the frame blocks of i
 * forced in when the gate is on (and the block holding both video and text
 * tokens, if any).  TOPK counts k over the nv video blocks.  With text
 * tokens every video row then keeps the text blocks, and the rows of the
 * text blocks keep every block.
 * Output (device, caller-owned):
 *   kv_idx [B, H, n, n] int32: row (b,h,i) starts at ((b*H+h)*n+i)*n and
 *          holds kv_cnt[(b*H+h)*n+i] ascending block indices; the rest of
 *          the row is not written.
 *   kv_cnt [B, H, n] int32, in [1, n].
 * Requires at least one recorded anchor (else MOD_ERR_BAD_STATE). */
mod_status mod_predict_block_mask(mod_stats* stats, const void* q, const void* k, int step,
                                  const mod_budget* budget, int32_t* kv_idx, int32_t* kv_cnt,
                                  void* stream);

/* Device workspace of the attention call, in bytes (0 for an invalid
 * shape): its work plan -- the (head, pair of query blocks) items ordered
 * and spread over the chip by their list lengths, rewritten by every call --
 * and room for the split-KV path (below): up to 1024 slots of partial
 * results of 8 * block * (d + 1) bytes each, fewer for short sequences
 * (none when n <= 64).  About 4 * (B*H*(n/2 + 16) + 300) bytes plus the
 * slots (47 KB + 135 MB at the 720p Hunyuan layer).  Owned by the caller;
 * two calls in flight at once need two workspaces. */
size_t mod_attn_workspace_bytes(const mod_shape* shape);

/* The smallest workspace the attention call accepts: the work plan alone
 * (the call then never splits a walk).  0 for an invalid shape. */
size_t mod_attn_plan_bytes(const mod_shape* shape);

/* Block-sparse attention forward (Eq. 1 with the block mask of the lists):
 * for every query token p of block i of head (b,h),
 *   O_p = sum over tokens q of the kept blocks of softmax_q(scale * Q_p.K_q) V_q
 *   lse_p = log sum_q exp(scale * Q_p.K_q)        (natural log)
 * with the kept blocks kv_idx[row][0 .. kv_cnt[row]) (layout of
 * mod_predict_block_mask; indices in [0, n), each at most once).  kv_idx
 * must be the whole [B, H, n, n] array: every slot of a row may be read
 * (those at or past kv_cnt are loaded with the row and ignored).  A row with
 * kv_cnt = 0 gives O = 0 and lse = -inf.  scale = 0 means 1/sqrt(d).
 * q, k, v, o: [B,H,L,d] bf16 device; lse: [B,H,L] fp32 device or NULL.
 * bf16 MFMA products, fp32 softmax and accumulation.  `frame_tokens` and
 * `text_tokens` of the shape are not used.  workspace: device memory of
 * ws_bytes bytes, 16-byte aligned, at least mod_attn_plan_bytes(shape),
 * else MOD_ERR_INVALID_ARG.
 * Split-KV: when few pairs carry long walks (few heads, dense rows), a pair
 * whose work exceeds half of a compute unit's share of the launch is split
 * into chunks of its walk, processed as separate items that write O / l and
 * LSE per row in fp32 into the workspace's slots; a merge kernel then
 * combines them (LSE = log sum_c exp(lse_c), O = sum_c exp(lse_c - LSE) O_c)
 * in chunk order, so the result is deterministic for given lists.  With
 * fewer than two slots (a workspace of mod_attn_plan_bytes) nothing is
 * split; whether a pair is split depends on the lists of all heads, so
 * outputs may differ by rounding between a split and an unsplit run. */
mod_status mod_block_sparse_attn_fwd(const mod_shape* shape, const void* q, const void* k,
                                     const void* v, const int32_t* kv_idx,
                                     const int32_t* kv_cnt, float scale, void* o, float* lse,
                                     void* workspace, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): mod_block_sparse_attn_fwd with its work plan held in a
 * library-owned device array of MOD_ATTN_NOALLOC_MAX_BYTES per device
 * instead of a caller workspace.  Same arguments, layout, numerics and
 * errors as mod_block_sparse_attn_fwd given a workspace of
 * mod_attn_plan_bytes(shape) bytes (its output is bit-identical to that
 * call's: no walk is split); shapes whose plan exceeds the array are
 * rejected with MOD_ERR_UNSUPPORTED.  The call allocates nothing:
 * the array is a static device variable whose address is resolved on the
 * first call on each device (the current device, which must be the device
 * of the pointers and the stream) and kept until the process ends.  Every
 * call on a device shares that device's array, so calls that overlap on one
 * device (concurrent streams, other threads) race on it and must be
 * serialised by the caller; calls on one stream are ordered and safe. */
#define MOD_ATTN_NOALLOC_MAX_BYTES (2u << 20)
mod_status mod_block_sparse_attn_fwd_noalloc(const mod_shape* shape, const void* q, const void* k,
                                             const void* v, const int32_t* kv_idx,
                                             const int32_t* kv_cnt, float scale, void* o, float* lse,
                                             void* stream);

/* ---- introspection (synchronous copies to host memory; for tests) ---- */

/* The sizes below count the nv video blocks (nv = n without text tokens). */

/* Anchor `slot` (0 = newest, 1 = the one before): coefficients
 * [B, H, 3nv-1+F] fp64 (order c_{-(nv-1)..nv-1}, d_{0..nv-1}, e_{0..F-1};
 * minimum-norm gauge) and its step.  MOD_ERR_BAD_STATE if absent. */
mod_status mod_stats_get_anchor(const mod_stats* stats, int slot, double* host_coeffs,
                                int* step);

/* Block means of the last fitted q, k: [B, H, nv, d] fp64 each. */
mod_status mod_stats_get_pooled(const mod_stats* stats, double* host_qbar, double* host_kbar);

/* The fitted statistic of the last fit: [B, H, nv, nv] fp64 (statistic 0: the
 * pooled block mass G; statistic 1: the stored informativeness map I). */
mod_status mod_stats_get_block_mass(const mod_stats* stats, double* host_G);

/* Last prediction (c~, d~): [B, H, 3nv-1] fp64. */
mod_status mod_stats_get_prediction(const mod_stats* stats, double* host_pred);

/* Block-diagonal gate per head, [B, H] int32 (0/1); MOD_ERR_BAD_STATE
 * before the first predict. */
mod_status mod_stats_get_gate(const mod_stats* stats, int32_t* host_gate);

const char* mod_status_string(mod_status status);
const char* mod_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MODDIT_H */

/*
 * cold.h -- C ABI of libcold.so, the MI355X (gfx950) scoring path of COLD,
 * the pre-ranking system of Wang et al., "COLD: Towards the Next Generation
 * of Pre-Ranking System" (DLP-KDD 2020).
 *
 * One call scores every candidate ad of a batch of requests with one deep
 * CTR model (Section 2, Section 3.1): per (user, ad) row it gathers the user,
 * ad and user x ad cross feature-group embeddings, sum-pools multi-valued
 * groups (Section 3.3, low precision), weights every group by its SE
 * importance (Section 3.2, Eq. 2), optionally keeps only the top-k groups
 * (Section 3.2, feature group selection), optionally applies linear_log to
 * the network input (Section 3.3, Eq. 3), and runs the fully connected
 * network D_in x ... x n_out down to a CTR (Section 4.1).
 *
 * Memory: every pointer marked "device" is device memory owned by the
 * caller; the library never allocates device memory.  Pointers marked "host"
 * are read during the call only.  Streams are hipStream_t values passed as
 * void* (NULL = the null stream).  Work is enqueued asynchronously on that
 * stream unless stated otherwise.
 *
 * Errors: every entry point returns COLD_OK (0) or a negative status; no
 * exception crosses the ABI.  Host-side checks run before anything is
 * enqueued, so a rejected call has no device side effect.
 * cold_last_error() gives the message of the model's last failure.
 *
 * Threading: a cold_model may be used by concurrent cold_score calls on
 * different streams with distinct workspaces; cold_load_weights must not
 * race with cold_score on the same model.
 */
#ifndef COLD_H
#define COLD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
#define COLD_OK 0
#define COLD_ERR_INVALID_ARG (-1)    /* null pointer, negative size, bad flag */
#define COLD_ERR_SHAPE (-2)          /* inconsistent dimensions */
#define COLD_ERR_DTYPE (-3)          /* unsupported dtype / id kind / dim */
#define COLD_ERR_NOT_LOADED (-4)     /* cold_score before cold_load_weights */
#define COLD_ERR_WORKSPACE (-5)      /* workspace or arena too small */
#define COLD_ERR_HIP (-6)            /* a HIP runtime call failed */
#define COLD_ERR_ID_RANGE (-7)       /* validate mode: an id or offset was out of range */

/* storage and compute type of embedding tables and MLP weights */
#define COLD_F32 0
#define COLD_BF16 1
#define COLD_F16 2

/* id columns: int32 row ids used as-is (must be < table rows), or raw
 * uint64 ids hashed into the table: row = mix64(raw ^ salt_g) mod rows, with
 * mix64 the SplitMix64 output function and salt_g = (g+1) * 0x9e3779b97f4a7c15
 * for feature group g.  (The paper does not describe id hashing.) */
#define COLD_IDS_DIRECT_I32 0
#define COLD_IDS_HASHED_U64 1

/* cold_score flags */
#define COLD_SCORE_VALIDATE 1        /* synchronise and report out-of-range ids */

/* Model description (host memory, copied by cold_create_model).
 * Feature groups are one per field, concatenated in the order user
 * (single-valued), user behaviour sequence (sum-pooled), ad, cross; group g
 * uses table g.  M = n_user + n_seq + n_ad + n_cross, D_in = M * emb_dim.
 * The SE block has H = max(1, M / se_reduction) hidden units.
 * widths[0] = D_in; widths[1..n_layers-1] are ReLU hidden layers;
 * widths[n_layers] is 1 (CTR = sigmoid) or 2 (softmax, CTR = class 1).
 * Supported: emb_dim * sizeof(dtype) a multiple of 16 bytes, a network
 * input row of at most 1024 such 16-byte chunks (M <= 512 at emb_dim 16 in
 * bf16/fp16), hidden widths multiples of 8 (bf16/f16), last hidden width
 * <= 8192 (fp32 head weights in 64 KB). */
typedef struct cold_model_desc {
  int32_t n_user, n_seq, n_ad, n_cross;
  int32_t emb_dim;
  int32_t id_kind;          /* COLD_IDS_* */
  int32_t dtype;            /* COLD_F32 | COLD_BF16 | COLD_F16 */
  int32_t se_reduction;     /* >= 1 */
  int32_t n_layers;         /* >= 1 */
  const int32_t *widths;    /* host [n_layers + 1] */
  const int64_t *table_rows;/* host [M], rows of each table, 1 .. 2^31-1 */
  int32_t linear_log;       /* 0/1: apply Eq. 3 to the network input */
  int32_t topk_k;           /* 0: off; else keep the k most important groups per request */
  const int32_t *cross_pairs; /* host [n_cross][2] or NULL: see below */
  int32_t se_form;          /* COLD_SE_SQUEEZE (0) or COLD_SE_LITERAL (1), see below */
} cold_model_desc;

/* Form of the SE block of Section 3.2 (Eq. 2, which prints as garbled):
 *   COLD_SE_SQUEEZE  the squeeze-and-excitation block of Hu et al. that the
 *                    section cites: z_g = mean of e_g, h = ReLU(W1 z + b1)
 *                    (H = max(1, M / se_reduction) units), s = sigmoid(W2 h + b2);
 *   COLD_SE_LITERAL  Eq. 2 as printed: s = sigmoid(W [e_1, ..., e_M] + b), one
 *                    fully connected layer from the concatenated D_in-wide
 *                    embedding to M weights: se_w1 is W [M][D_in], se_b1 is
 *                    b [M], se_w2 and se_b2 are not read (may be NULL), and
 *                    se_reduction is ignored. */
#define COLD_SE_SQUEEZE 0
#define COLD_SE_LITERAL 1

/* User x ad cross features built on the GPU (desc.cross_pairs != NULL).
 * The paper builds its cross features on the CPU next to the other feature
 * computation (Section 3.3) and does not say how a cross value is formed.
 * Here cross field f pairs user field u = cross_pairs[2f] (0 <= u < n_user)
 * with ad field a = cross_pairs[2f+1] (0 <= a < n_ad): with uid and aid the
 * two fields' raw ids (int32 ids zero-extended from their 32-bit pattern, or
 * the uint64 raw ids of a hashed model), the pair's key is
 *     key = mix64(uid) ^ aid
 * and its table row is mix64(key ^ salt_g) mod rows with the group salt of
 * the hashed id kind (group g = n_user + n_seq + n_ad + f), for either id
 * kind.  cold_batch.cross_ids is then not read and may be NULL. */

typedef struct cold_model cold_model;

/* Parameters (cold_load_weights).  Tables are used in place (not copied) and
 * must stay alive while the model scores; the rest is copied into the arena.
 *   tables[g]   device [table_rows[g]][emb_dim], dtype, 16-byte aligned
 *   se_w1       device fp32 [H][M]      se_b1 device fp32 [H]
 *   se_w2       device fp32 [M][H]      se_b2 device fp32 [M]
 *               (literal SE form: se_w1 [M][D_in], se_b1 [M], se_w2/se_b2 unused)
 *   mlp_w[l]    device [widths[l+1]][widths[l]] (out x in), dtype
 *   mlp_b[l]    device fp32 [widths[l+1]]                                  */
typedef struct cold_weights {
  const void *const *tables;    /* host array [M] of device pointers */
  const float *se_w1, *se_b1, *se_w2, *se_b2;
  const void *const *mlp_w;     /* host array [n_layers] of device pointers */
  const float *const *mlp_b;    /* host array [n_layers] of device pointers */
} cold_weights;

/* One batch of requests in the column (field-major) layout of Section 3.3.
 * Q = n_requests, R = n_rows; rows of request q are req_off[q] .. req_off[q+1]-1.
 * Id element type is int32 (COLD_IDS_DIRECT_I32) or uint64 (HASHED_U64).
 *   req_off    device int32 [Q + 1], non-decreasing, req_off[0] = 0, req_off[Q] = R
 *   user_ids   device [n_user][Q]
 *   ad_ids     device [n_ad][R]
 *   cross_ids  device [n_cross][R]
 *   seq_off    device int32 [n_seq * Q + 1]; ids of sequence field f of request q
 *              are seq_ids[seq_off[f*Q + q] .. seq_off[f*Q + q + 1] - 1]
 *   seq_ids    device [n_seq_ids]
 * Empty requests and empty sequences (pooled to zero) are allowed. */
typedef struct cold_batch {
  int64_t n_requests;
  int64_t n_rows;
  int64_t n_seq_ids;
  const int32_t *req_off;
  const void *user_ids;
  const void *ad_ids;
  const void *cross_ids;
  const int32_t *seq_off;
  const void *seq_ids;
} cold_batch;

/* Validate a model description and create the host-side model: one deep
 * CTR model that scores every candidate ad of a request (Section 2, the
 * pre-ranking problem; Section 3.1, the network over concatenated
 * group-wise embeddings; Section 4.1, its widths).  CPU only.  *out
 * receives a library-owned handle (free with cold_destroy_model).  Returns
 * COLD_ERR_INVALID_ARG / _SHAPE / _DTYPE for a description outside the
 * supported shapes above, with *out set to NULL. */
int cold_create_model(const cold_model_desc *desc, cold_model **out);

/* Free the host-side model made by cold_create_model (never device
 * memory: the arena, tables and workspaces stay the caller's).  NULL is a
 * no-op. */
void cold_destroy_model(cold_model *model);

/* Bytes of device memory the caller must provide as the weight arena: the
 * SE parameters (Section 3.2, Eq. 2) and the network's weights and biases
 * (Section 4.1), plus per-table metadata.  0 for a NULL model. */
size_t cold_weight_arena_bytes(const cold_model *model);

/* Bytes of device workspace cold_score needs for up to max_rows rows (ads)
 * and max_requests requests (the batch of Section 2: the candidate ads of a
 * request, Section 3.3: requests scored together): pooled user rows, the
 * network input and two hidden-layer buffers.  0 if the model is NULL or a
 * size is negative. */
size_t cold_workspace_bytes(const cold_model *model, int64_t max_rows, int64_t max_requests);

/* Register the tables and copy SE and MLP parameters into `arena` (device,
 * 256-byte aligned, >= cold_weight_arena_bytes).  Callable repeatedly: the
 * online model update of Section 3.4 (the model is retrained and updated
 * continuously) swaps parameters in place; ordered on `stream`, and returns
 * after the copies have completed.  The arena must stay alive while the
 * model scores.  Returns COLD_ERR_INVALID_ARG for a NULL or misaligned
 * pointer and COLD_ERR_WORKSPACE for a short arena, before any copy. */
int cold_load_weights(cold_model *model, const cold_weights *w, void *arena,
                      size_t arena_bytes, void *stream);

/* Score every row of batch b (Sections 3.1-3.3; Section 4.1 network).
 *   workspace   device, 256-byte aligned, ws_bytes >= cold_workspace_bytes(R, Q)
 *   scores      device fp32 [R]: CTR of each row
 *   importance  device fp32 [R][M] or NULL: SE weights s of each row (Eq. 2),
 *               before any top-k mask
 *   group_mask  device uint8 [Q][M] or NULL: kept groups per request (topk_k > 0)
 *   rows_out    device int32 [M][R] or NULL: table row each single-valued group
 *               of each row resolved to (-1 for sequence groups)
 *   x_out       device [R][D_in] in the model dtype, or NULL: the network input
 *               of each row, v_g = s_g e_g for every group (Section 3.2),
 *               after the top-k mask and linear_log (Section 3.3, Eq. 3) and
 *               the one rounding to the model dtype (a debug copy; the
 *               scores do not depend on it)
 *   flags       0 or COLD_SCORE_VALIDATE (then the call synchronises the stream
 *               and returns COLD_ERR_ID_RANGE if any id or offset was out of range;
 *               without it such ids read a zero embedding)
 * Asynchronous on `stream` unless validating.  Q = 0 or R = 0 is a no-op. */
int cold_score(cold_model *model, const cold_batch *b, void *workspace, size_t ws_bytes,
               float *scores, float *importance, uint8_t *group_mask, int32_t *rows_out,
               void *x_out, int32_t flags, void *stream);

/* Scoring for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * cold_score with its workspace in a device array that the library holds,
 * COLD_NOALLOC_WORKSPACE_BYTES on each GPU it runs on, until the process
 * ends; the other arguments as for cold_score.  The stream (NULL: the null
 * stream) must belong to the current device.  A batch whose
 * cold_workspace_bytes(R, Q) exceeds the array (the serving model: more
 * than eight 2,000-ad requests; the wide top-k model's 5,000-row request
 * fits) returns COLD_ERR_WORKSPACE with nothing
 * enqueued.  Every call on one GPU uses that GPU's one array, which keeps
 * the last call's contents: calls that overlap on one GPU (other streams,
 * other threads) race, so the caller serialises them.  Calls no allocating
 * routine; stage profiling does not record these calls. */
#define COLD_NOALLOC_WORKSPACE_BYTES (96ull * 1024 * 1024)
int cold_score_noalloc(cold_model *model, const cold_batch *b, float *scores, float *importance,
                       uint8_t *group_mask, int32_t *rows_out, void *x_out, int32_t flags,
                       void *stream);

/* Stage timing: measurement only, not part of scoring (the paper defines
 * no such call).  While enabled, every cold_score
 * call on this model records a HIP event on its stream before each kernel
 * stage and one after the last; cold_profile_read synchronises those events
 * and returns, per stage, its name and the summed elapsed milliseconds over
 * all calls since the previous read (stages are matched by position; every
 * profiled call of one model runs the same stage sequence).  Not for
 * concurrent cold_score calls on one model.  Enabling creates HIP events;
 * disabling destroys them.
 *   names       host char[max_stages][32] or NULL
 *   total_ms    host float[max_stages]
 *   n_stages    host: stages of the profiled calls
 *   n_calls     host: profiled calls since the previous read */
int cold_profile_enable(cold_model *model, int32_t enable);
int cold_profile_read(cold_model *model, int32_t max_stages, char (*names)[32], float *total_ms,
                      int32_t *n_stages, int32_t *n_calls);

/* Per-request top-n selection by eCPM (Section 2: the pre-ranking stage
 * passes on the N candidates of each request with the highest eCPM; its
 * footnote defines eCPM = pCTR * bid for CPC bidding).  Stateless: needs no
 * model.
 *   scores     device fp32 [n_rows]: CTR of each row (as cold_score writes it)
 *   bids       device fp32 [n_rows]: bid of each row
 *   req_off    device int32 [n_requests + 1], as in cold_batch (offsets are
 *              clamped to [0, n_rows])
 *   n_top      1 .. COLD_TOPN_MAX
 *   top_rows   device int32 [n_requests][n_top]: row indices (into the batch,
 *              not the request), best first
 *   top_ecpm   device fp32 [n_requests][n_top] or NULL: their eCPM
 * eCPM = scores[r] * bids[r], one fp32 multiplication.  Rows are ordered by
 * eCPM under the IEEE-754 totalOrder (so -0 < +0 and NaNs sort by sign
 * beyond the infinities), ties by ascending row index.  A request with
 * fewer than n_top rows fills its remaining slots with row -1 and eCPM
 * -infinity.  Asynchronous on `stream`; n_requests = 0 is a no-op.
 * Returns COLD_ERR_INVALID_ARG for a negative size, n_rows or n_requests
 * above 2^31 - 1, n_top out of range, or a NULL required pointer. */
#define COLD_TOPN_MAX 1024
int cold_select_topn(const float *scores, const float *bids, const int32_t *req_off,
                     int64_t n_requests, int64_t n_rows, int32_t n_top, int32_t *top_rows,
                     float *top_ecpm, void *stream);

/* Static text of a status code. */
const char *cold_status_string(int status);

/* Message of the last failed call on this model ("" if none; a static
 * message if model is NULL). */
const char *cold_last_error(const cold_model *model);

#ifdef __cplusplus
}
#endif
#endif /* COLD_H */

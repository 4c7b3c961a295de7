/*
 * cacheback.h -- C ABI of the MI355X receiver-conditioned KV selection path.
 *
 * The receiver's query is scored against a sender's KV cache, per layer and
 * per KV head, with attention weights; importance is summed over query rows
 * and the query heads of each GQA group; the top fraction of sender positions
 * is kept and their K/V rows are gathered into a compact cache.
 *
 * Paper: "Receiver-Conditioned Latent Communication gives 94% CacheBack",
 * Appendix C.1 (attention from the appended query tokens to the sender cache,
 * the mean-query-attention equation) and Appendix C.2 (per-sender budget
 * ceil(T/r), ties to the earlier position, source order).
 *
 * Conventions shared by every call
 *   - Device pointers are HIP device memory on the current device, 16-byte
 *     aligned (CB_ERR_ALIGN otherwise).  "stream" is a hipStream_t passed as
 *     void*; NULL means the default stream.
 *   - Every call only enqueues work on `stream` and returns; results are
 *     valid once the stream reaches that point.  No call synchronises,
 *     allocates device memory or keeps a pointer after it returns.  Calls are
 *     reentrant; calls that share a workspace must not overlap in time.
 *   - cb_score and cb_pipeline enqueue, on `stream`, a small kernel that
 *     clears the call's synchronisation words in `ws` and one persistent
 *     kernel whose resident workgroups take every work item of the call from
 *     a device queue (one more kernel adds row-group sums in cb_score when
 *     G*m > 512).  Their workgroups wait on one another through `ws`, with
 *     bounded waits; two calls sharing a workspace must not overlap.
 *   - The caller owns every buffer.  Outputs must not alias inputs.
 *   - On an argument error nothing is launched and a negative CB_ERR_* code
 *     is returned.  CB_ERR_HIP reports a launch failure.
 *   - Units: u = (s*L + l)*Hkv + g for sender s, layer l, KV head g.
 *     Query head h reads KV head h / (Hq/Hkv) (contiguous GQA groups).
 *
 * Canonical layouts (row-major, contiguous)
 *   q           [L][Hq][m][D]        receiver query projections per layer
 *   k, v        [S][L][Hkv][T][D]    sender caches (post-RoPE, as stored)
 *   importance  [S][L][Hkv][T]       fp32
 *   row_lse     [S][L][Hq][m]        fp32, natural-log softmax normaliser
 *   idx         [S][L][Hkv][keep]    int32, strictly ascending per unit
 *   k_out,v_out [L][Hkv][S*keep][D]  senders concatenated in sender order
 */
#ifndef CACHEBACK_H
#define CACHEBACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  CB_OK = 0,
  CB_ERR_NULL = -1,      /* a required pointer is NULL */
  CB_ERR_SHAPE = -2,     /* non-positive dims, Hq % Hkv != 0, D not 64/128,
                            T > 2^31 - 2^16, Hq/Hkv*m > 1024, bad scale */
  CB_ERR_DTYPE = -3,     /* dtype not CB_F32 / CB_BF16 */
  CB_ERR_RATIO = -4,     /* keep_ratio NaN or outside (0, 1] */
  CB_ERR_WORKSPACE = -5, /* workspace missing or smaller than required */
  CB_ERR_ALIGN = -6,     /* device pointer not 16-byte aligned */
  CB_ERR_HIP = -7,       /* HIP launch error */
  CB_ERR_TIMEOUT = -8    /* a dependency wait inside a kernel gave up (reported
                            by cb_score_status / cb_select_status) */
};

typedef enum { CB_F32 = 0, CB_BF16 = 1 } cb_dtype;

typedef struct cb_layout {
  int32_t layers;   /* L: scored (global-attention) layers */
  int32_t q_heads;  /* Hq */
  int32_t kv_heads; /* Hkv; Hq % Hkv == 0 */
  int32_t head_dim; /* D: 64 or 128 */
  int32_t q_len;    /* m: receiver query tokens */
  int32_t senders;  /* S: independent sender caches scored against one q */
  int64_t seq_len;  /* T: positions per sender, 1 <= T <= 2^31 - 2^16 */
  int32_t dtype;    /* cb_dtype of q, k and v */
  float scale;      /* softmax scale; 0 selects 1/sqrt(D); must be >= 0 */
} cb_layout;

/* Bytes of scratch cb_score (and cb_pipeline, whose selection uses part of
 * it) needs for `lay` (0 on an invalid layout). */
size_t cb_score_workspace_bytes(const cb_layout* lay);

/* Per-unit importance (Appendix C.1, attention from the query tokens to the
 * sender positions; mean-query-attention equation, inner sum over query rows
 * r and the heads h of one KV-head group):
 *   importance[u][t] = sum_{h in group g} sum_{r < m} softmax_t(scale * q[l][h][r] . k[s][l][g][t])
 * The softmax runs over the T sender positions only.  Each unit's importance
 * sums to G*m.  row_lse (nullable) receives log(sum_t exp(scale * q.k)) per
 * query row.  `ws` is caller-owned scratch of cb_score_workspace_bytes(lay)
 * bytes; its contents need not be initialised.  Deterministic: the same
 * inputs give bitwise-identical outputs.
 * Failure inside the kernel: workgroups of the persistent kernel wait on one
 * another with bounded waits.  A wait that gives up (it cannot in a correct
 * run; see cb_set_wait_limit) sets an error word in `ws`, every later wait
 * gives up at once, the affected importance and row_lse entries are NaN, and
 * every kernel still exits.  cb_score_status reports the word. */
int cb_score(const void* q, const void* k, const cb_layout* lay, float* importance,
             float* row_lse, void* ws, size_t ws_bytes, void* stream);

/* Budget (Appendix C.2, fan-out budget equation, with keep_ratio = 1/r):
 * ceil(keep_ratio * T) clamped to [1, T]; a product within 1e-12 (relative)
 * of an integer counts as that integer.  Host-only.  Returns CB_ERR_RATIO
 * for a ratio outside (0, 1] or NaN and CB_ERR_SHAPE for T < 1. */
int64_t cb_keep_count(int64_t T, double keep_ratio);

/* Top-k selection per unit (Appendix C.2: equal scores favour the earlier
 * position; selected positions are returned in source order).  Keeps the
 * keep = cb_keep_count(T, keep_ratio) positions of highest importance, ties
 * broken toward the lower index, and writes them strictly ascending to
 * idx[u][0..keep).  Keys compare as fp32 values with -0 == +0; NaN ranks
 * below every number.  importance: [units][T]; idx: [units][keep].
 * k_out (host pointer, nullable) receives keep.  1 <= T <= 2^31 - 2^16. */
int cb_select(const float* importance, int64_t units, int64_t T, double keep_ratio,
              int32_t* idx, int64_t* k_out, void* stream);

/* Bytes of scratch cb_select_ws uses for `units` rows of T scores: nonzero
 * when such rows are split over several workgroups (T > 16384 and at most
 * 128 units, at most 256 workgroups in all), else 0 (also for invalid
 * sizes).  Host-only. */
size_t cb_select_workspace_bytes(int64_t units, int64_t T);

/* cb_select with caller-owned scratch; the same selection, bit for bit
 * (same definition: Appendix C.2).  When cb_select_workspace_bytes(units, T)
 * is nonzero and ws holds that many bytes (16-byte aligned), each row is
 * split over several workgroups that hold their parts in registers and
 * exchange digit counts through ws: with fewer units than compute units, one
 * workgroup per row would leave most of the device idle.  Otherwise, with
 * ws = NULL, or when the device cannot hold every part at once, it runs as
 * cb_select.  ws contents need not be initialised (a small clearing kernel
 * runs first); CB_ERR_WORKSPACE if ws is given but too small.  The parts of a
 * row wait on one another with bounded waits; a wait that gives up (it
 * cannot in a correct run; see cb_set_wait_limit) leaves -1 or valid but
 * unspecified positions in that row, every kernel still exits, and
 * cb_select_status reports it.  Calls that share a ws must not overlap in
 * time (one stream per ws). */
int cb_select_ws(const float* importance, int64_t units, int64_t T, double keep_ratio,
                 int32_t* idx, int64_t* k_out, void* ws, size_t ws_bytes, void* stream);

/* Outcome of the last cb_select_ws call that used `ws` for (units, T):
 * synchronises `stream`, then returns CB_OK, or CB_ERR_TIMEOUT if a wait
 * between the parts of a row gave up.  CB_OK at once when rows of that size
 * are not split. */
int cb_select_status(int64_t units, int64_t T, const void* ws, size_t ws_bytes, void* stream);

/* Compaction: the message carries the sender state at the selected
 * positions (section 2.1, "Communication Costs": one KV entry per layer for
 * each position; Appendix C.2: selected positions in source order; fan-in
 * messages from several senders reach one receiver, section 4.2):
 *   k_out[l][g][s*keep + j][:] = k[s][l][g][idx[s][l][g][j]][:],
 * likewise v; bit-exact row copies, senders concatenated in sender order.
 * idx rows hold `keep` positions in [0, T); an entry outside that range
 * yields an all-zero output row (no out-of-bounds access). */
int cb_compact(const void* k, const void* v, const int32_t* idx, const cb_layout* lay,
               int64_t keep, void* k_out, void* v_out, void* stream);

/* The whole path in one call (section 3: the receiver query scores the
 * sender state, the sender selects positions under its budget, the selected
 * state forms the message; Appendix C.1-C.2): cb_score, then cb_select and
 * cb_compact with keep = cb_keep_count(T, keep_ratio), with the same outputs
 * as the three calls in sequence.  Enqueues, on `stream` and in this order,
 * the clearing kernel and the persistent score kernel of cb_score, one
 * select kernel (one workgroup per unit, or several per unit as in
 * cb_select_ws when cb_select_workspace_bytes(units, T) is nonzero, with
 * their scratch in ws) and one gather kernel; no host synchronisation
 * between them.  If a wait inside the score kernel gave up, the select
 * kernel writes -1 for every index (so every compacted row is zero); if a
 * wait between the parts of a split row gave up, that row holds -1 or valid
 * but unspecified positions.  cb_score_status reports either as
 * CB_ERR_TIMEOUT.
 * keep_out (host pointer, nullable) receives keep.  Buffers as for the
 * individual calls; ws as for cb_score. */
int cb_pipeline(const void* q, const void* k, const void* v, const cb_layout* lay,
                double keep_ratio, float* importance, float* row_lse, int32_t* idx,
                void* k_out, void* v_out, void* ws, size_t ws_bytes, int64_t* keep_out,
                void* stream);

/* cb_pipeline for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation and outputs, with the score workspace taken from a
 * 64 MiB array the library holds on each device it runs on (until the
 * process ends) instead of a `ws` argument.  Makes no allocation of any kind.
 * Returns CB_ERR_WORKSPACE, launching nothing, when the layout needs more
 * than 64 MiB of workspace (cb_score_workspace_bytes; the Qwen3-8B shape
 * needs 5 MB, T = 65536 x 64 units 4 MB).  Every call on a device shares that
 * device's array: calls that overlap in time on one device (other streams,
 * other host threads) race and must be serialised by the caller. */
int cb_pipeline_noalloc(const void* q, const void* k, const void* v, const cb_layout* lay,
                        double keep_ratio, float* importance, float* row_lse, int32_t* idx,
                        void* k_out, void* v_out, int64_t* keep_out, void* stream);

/* Outcome of the last cb_score / cb_pipeline call that used `ws` with layout
 * `lay`: synchronises `stream` (the one that call used), then returns CB_OK,
 * or CB_ERR_TIMEOUT if a dependency wait inside the score kernel gave up
 * (its outputs then hold NaN importance and, from cb_pipeline, -1 indices).
 * Argument errors as for cb_score. */
int cb_score_status(const cb_layout* lay, const void* ws, size_t ws_bytes, void* stream);

/* Polls after which a dependency wait inside the score kernel gives up, for
 * the calls enqueued after this one (process-wide); 0 makes every wait give
 * up at once.  Returns the previous value.  For tests of the failure path:
 * a correct run never reaches the default (about a second of polling). */
uint32_t cb_set_wait_limit(uint32_t polls);

/* ---- The paper's position-level selector and message (Appendix C) -------
 *
 * Layouts (row-major, contiguous):
 *   score, qscore, corr  [S][T]            fp32, one row per sender
 *   idx (spans)          [S][count]        int32, ascending per sender
 *   rows                 [S][T][row_bytes] continuous rows per sender
 *   rows out             [S][count][row_bytes], senders in order
 */

/* Bytes of scratch cb_position_score needs for `lay` (0 on an invalid layout
 * or one the position path does not take: G > 8, or Gp*m > 1024 with Gp the
 * group rounded up to 4 or 8). */
size_t cb_position_workspace_bytes(const cb_layout* lay);

/* Position-level score of every sender position (Appendix C.1; general score
 * of Appendix D.2):
 *   Q_t     = Pool_7( sum_l 1/(m*Hq) sum_{h, r} a[l,h,r,t] )   mean query attention
 *   C_{p,t} = ( sum_s mean_r Pool_7(b[s,r,.])^p / sum_s Pool_7(mean_r b[s,r,.])^p )^(1/(p-1))
 *   S_t     = Q_t * C_{p,t}^alpha
 * a: attention weights of cb_score (softmax over the T sender positions);
 * b[s,r,t]: the mean of a over the query heads of KV-head group s (one group
 * per layer and KV head); Pool_7: maximum over positions t-3..t+3 clipped to
 * the sequence; C = 1 where both sums vanish.  p = INFINITY gives the ratio
 * of the largest pooled per-token weight to the largest pooled mean.
 * CacheBack is p = alpha = 2; mean query attention is alpha = 0.
 * Requires 1 < p <= 8 or p = INFINITY, 0 <= alpha < inf.
 * score (required), qscore = Q_t and corr = C_{p,t} (nullable): [S][T] fp32.
 * importance (nullable): [S][L][Hkv][T], receives cb_score's importance
 * (held in `ws` when NULL).  Computed in fp32 from bf16/fp32 inputs with
 * fp32 accumulation; sums over layers and heads in fp64.  Deterministic.
 * Enqueues the clearing kernel and the persistent score kernel (second pass
 * extended with the pooled per-token sums), then two small kernels. */
int cb_position_score(const void* q, const void* k, const cb_layout* lay, double p, double alpha,
                      float* score, float* qscore, float* corr, float* importance, void* ws,
                      size_t ws_bytes, void* stream);

/* As cb_score_status, for a cb_position_score call. */
int cb_position_status(const cb_layout* lay, const void* ws, size_t ws_bytes, void* stream);

/* Budgets (Appendix C.2), host-only, integer compression ratio r >= 1:
 *   fan-out:        B = ceil(T / r)
 *   chain relative: B = T_old + ceil(T_new / r)   (relative != 0)
 *   chain fixed:    B = min(B_max, T_old + T_new)  (relative == 0)
 * CB_ERR_SHAPE for T < 1, T_old < 0, T_new < 1, r < 1 or (fixed) B_max < 1. */
int64_t cb_budget_fanout(int64_t T, int64_t r);
int64_t cb_budget_chain(int64_t T_old, int64_t T_new, int64_t r, int relative, int64_t B_max);

/* Scratch bytes of cb_select_spans (0 on invalid sizes). */
size_t cb_spans_workspace_bytes(int64_t senders, int64_t T, int32_t width);

/* Position selection per sender (Appendix C.2): the first position and the
 * last n_latent positions (the current latent steps) are kept and count
 * toward `budget`; position 0's score is replaced by the maximum score;
 * spans of `width` positions from position 0 (the last may be shorter) are
 * ranked by mean score (the fp64 sum of their fp32 scores in position order
 * over their length), equal means favouring the earlier span; spans add
 * their unselected positions in rank order while they fit, and the first
 * span that does not fit adds only its unselected positions nearest its
 * highest-scoring position (right first at equal distance, within the span)
 * until the budget is full.  idx[s][0..count) receives the selected
 * positions in source order, count = min(budget, T) (also written to
 * count_out, a nullable host pointer).  score: [S][T] fp32, finite.
 * Requires 1 <= width <= 64 and budget >= min(T, n_latent + 1)
 * (CB_ERR_SHAPE otherwise).  One workgroup per sender; integer-exact given
 * the scores. */
int cb_select_spans(const float* score, int64_t senders, int64_t T, int64_t budget,
                    int64_t n_latent, int32_t width, int32_t* idx, int64_t* count_out, void* ws,
                    size_t ws_bytes, void* stream);

/* Continuous-row message (section 3.1.2 "State Representation", Appendix
 * C.3: each selected position is sent as one row of the model's continuous
 * input representation):
 *   out[s*count + j][:] = rows[s][idx[s*count + j]][:]
 * bit-exact copies of row_bytes bytes (a multiple of 4; pointers 16-byte
 * aligned when row_bytes is a multiple of 16, else 4-byte); an index outside
 * [0, T) gives a zero row.  Also gathers per-position metadata (e.g. source
 * ids, row_bytes = 4 or 8) along a chain of messages. */
int cb_gather_rows(const void* rows, int64_t senders, int64_t T, int64_t row_bytes,
                   const int32_t* idx, int64_t count, void* out, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* cb_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* CACHEBACK_H */

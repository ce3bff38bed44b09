/*
 * timebill.h -- C ABI of the MI355X (gfx950) eviction + decode hot path of
 * TimeBill (time-budgeted LLM inference, arXiv 2512.21859).
 *
 * TimeBill picks a KV-cache eviction ratio alpha per request so that the
 * predicted worst-case time fits a budget (Sec. 5.1, Eq. alpha_with_predictor).
 * After the prefill phase a fraction alpha of the prompt's KV cache is
 * evicted once, and decoding runs over the retained cache, whose length at
 * decode step i is (1 - alpha) N_x + i - 1 (Sec. 4.2, Eq. N_kv; Sec. 5.2).
 * The paper evicts with SnapKV (Sec. 6.1).  This library provides that path:
 *
 *   tb_score_window  observation-window scores (softmax of the last w queries
 *                    against the prompt keys, summed per KV head, max-pooled);
 *                    tb_score_window_avgpool, tb_score_knorm and
 *                    tb_score_h2o are the scorer variants (mean-pooled window
 *                    scores; key norms; accumulated attention of all queries);
 *   tb_select_topk   per-KV-head top-k of the scores keeping n_keep positions;
 *   tb_compact_kv    gather of the kept K/V rows into a compact cache;
 *   tb_decode_attn   single-token grouped-query decode attention over the
 *                    compact cache, with the new token's K/V appended first
 *                    (attention definition: Sec. 4.2, FLOPs-based Modeling;
 *                    in a decoding step Q has length 1, K has length N_kv).
 *
 * Conventions
 * -----------
 * - Every pointer is a DEVICE pointer unless marked [host].  The caller owns
 *   all buffers; the library never allocates, frees or synchronises.  Work is
 *   enqueued on `stream`; TB_OK means "validated and enqueued".
 * - Every argument is validated on the host before any HIP call; on error
 *   nothing is launched and tb_last_error() describes the problem.
 *   C++ exceptions never cross this boundary.
 * - Layouts ("ragged lengths, padded strides"), all row-major:
 *     q_win      [B][Hq][w][d]     window queries of the last w prompt positions
 *     k, v       [B][Hkv][Lmax][d] prompt keys / values; sequence b valid for j < L[b]
 *     scores     [B][Hkv][Lmax]    fp32; entries j >= L[b] - w are left untouched
 *     keep_idx   [B][Hkv][Lmax]    int32; the first n_keep[b] entries are valid
 *     k_cache    [B][Hkv][cap][d]  compact K cache, row-major
 *     v_cache    [B][Hkv][cap][d]  compact V cache, row-major
 *                (the kernels walk both in 32-row tiles: cap must be a
 *                multiple of 32)
 *     kv_len     [B]               int32 current cache length per sequence (device)
 *     q, out     [B][Hq][d];  k_new, v_new [B][Hkv][d]
 *   Query head h uses KV head h / (Hq / Hkv).  The logit scale is 1/sqrt(d).
 *   Rows of k / v at j >= L[b] are never read.
 * - Supported: dtype fp32 or bf16, d in {64, 128}, B <= 64.  Scoring needs
 *   (Hq/Hkv) * w <= 1024; decoding needs Hq/Hkv <= 8.
 * - Retained length: n_keep = L - floor(alpha * L) in IEEE double, at least w.
 *   The w window positions are always kept and count toward n_keep; ties in
 *   the pooled score go to the lower position; kept positions are ascending
 *   with the window last.
 * - Re-entrant; the library keeps no device state.  Calls that share a
 *   workspace must be ordered (same stream).
 */
#ifndef TIMEBILL_H
#define TIMEBILL_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Only the functions declared here are exported; the library is built with
 * hidden visibility for everything else. */
#pragma GCC visibility push(default)

typedef enum {
  TB_OK = 0,
  TB_EINVAL = 1,        /* bad argument (null pointer, size, ratio, length) */
  TB_EUNSUPPORTED = 2,  /* valid but not supported (d, dtype, group size, B) */
  TB_EWORKSPACE = 3,    /* ws_bytes smaller than tb_workspace_bytes() */
  TB_EHIP = 4,          /* a HIP launch reported an error */
  TB_EINTERNAL = 5      /* unexpected internal failure */
} tb_status;

typedef enum { TB_F32 = 0, TB_BF16 = 1 } tb_dtype;

typedef enum {
  TB_OP_SCORE = 0,
  TB_OP_SELECT = 1,
  TB_OP_COMPACT = 2,
  TB_OP_DECODE = 3,
  TB_OP_H2O = 4
} tb_op;

/* [host] Retained positions after evicting a fraction alpha of L prompt
 * positions with a window of w (Eq. N_kv made integral): L - floor(alpha*L),
 * at least w.  Returns -1 unless 0 < w < L and 0 <= alpha < 1. */
int32_t tb_keep_count(int32_t L, double alpha, int32_t w);

/* [host] Message describing the last error on the calling thread ("" if none).
 * The pointer stays valid until the thread's next tb_* call. */
const char* tb_last_error(void);

/* [host] Workspace bytes the operation `op` needs for these sizes (0 if none).
 * `cap` is used by TB_OP_DECODE only; arguments an op does not use are
 * ignored.  Returns 0 and sets the error for invalid sizes.  For
 * TB_OP_DECODE the size covers every batch of at most B sequences with this
 * cap (the split depends on the batch size). */
size_t tb_workspace_bytes(int32_t op, int32_t B, int32_t Lmax, int32_t Hq,
                          int32_t Hkv, int32_t d, int32_t w, int32_t cap);

/* Observation-window scores (SnapKV eviction as used in Sec. 6.1; window
 * queries against all prompt keys under the causal attention of Sec. 4.2).
 * For KV head g of sequence b and prefix position j < L[b] - w:
 *   A[j] = sum over the G query heads of group g and window rows i < w of
 *          softmax_j'(q_win[h][i] . k[j'] / sqrt(d)),  j' <= L[b] - w + i,
 *   scores[j] = max of A over |j - j'| <= pool/2 within the prefix.
 * raw_scores (nullable, same layout) receives A before pooling.
 * Arithmetic: float64 dot products, exponentials and sums; fp32 output.
 * L: [host][B].  Requires w >= 1, odd pool >= 1, w < L[b] <= Lmax.
 * ws: tb_workspace_bytes(TB_OP_SCORE, B, Lmax, Hq, Hkv, d, w, 0) bytes. */
tb_status tb_score_window(const void* q_win, const void* k, int32_t B,
                          const int32_t* L, int32_t Lmax, int32_t Hq,
                          int32_t Hkv, int32_t d, int32_t w, int32_t pool,
                          tb_dtype dt, float* scores, float* raw_scores,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/* The same scores with the max-pool replaced by a mean (the average-pool
 * variant of the observation-window scorer):
 *   scores[j] = (1/pool) * sum of A[j'] over |j - j'| <= pool/2, with A taken
 *               as 0 outside the prefix [0, L[b] - w)   (divisor always pool).
 * The mean is summed in float64 from the fp32 raw scores.  Arguments,
 * requirements and workspace as tb_score_window. */
tb_status tb_score_window_avgpool(const void* q_win, const void* k, int32_t B,
                                  const int32_t* L, int32_t Lmax, int32_t Hq,
                                  int32_t Hkv, int32_t d, int32_t w, int32_t pool,
                                  tb_dtype dt, float* scores, float* raw_scores,
                                  void* ws, size_t ws_bytes, hipStream_t stream);

/* KNorm scores (the norm-based scorer cited for the fixed-ratio baselines,
 * Sec. 6.1): for KV head g of sequence b and prefix position j < L[b] - w,
 *   scores[j] = -||k[b][g][j]||_2,
 * so tb_select_topk keeps the smallest key norms (plus the window, as for
 * every scorer).  Sums of squares in float64, fp32 output; one read of K.
 * L: [host][B].  Requires w >= 1, w < L[b] <= Lmax.  No workspace. */
tb_status tb_score_knorm(const void* k, int32_t B, const int32_t* L, int32_t Lmax,
                         int32_t Hkv, int32_t d, int32_t w, tb_dtype dt,
                         float* scores, hipStream_t stream);

/* H2O scores (the accumulated-attention scorer cited for the fixed-ratio
 * baselines, Sec. 6.1): for KV head g of sequence b and every position j < L[b],
 *   scores[j] = sum over the G query heads h of group g and query positions
 *               i >= j of softmax_j'(q[h][i] . k[j'] / sqrt(d)),  j' <= i,
 * i.e. the attention mass key j receives from all prompt queries under the
 * causal softmax of Sec. 4.2.  tb_select_topk then keeps the largest prefix
 * scores plus the last w positions (the recent window).
 *   q: [B][Hq][Lmax][d], the prefill's queries at every prompt position.
 * Arithmetic: float64 dot products and sums (two passes over the causal
 * product: row statistics, then column mass), fp32 output.  Cost grows as
 * L^2: about 2 Hq L^2 d flops per call.
 * L: [host][B].  Requires 1 <= L[b] <= Lmax.
 * ws: tb_workspace_bytes(TB_OP_H2O, B, Lmax, Hq, Hkv, d, 0, 0) bytes. */
tb_status tb_score_h2o(const void* q, const void* k, int32_t B, const int32_t* L,
                       int32_t Lmax, int32_t Hq, int32_t Hkv, int32_t d, tb_dtype dt,
                       float* scores, void* ws, size_t ws_bytes, hipStream_t stream);

/* Per-KV-head top-k keeping n_keep[b] = tb_keep_count(L[b], alpha[b], w)
 * positions (Eq. N_kv: a fraction alpha of the prompt's KV is evicted once,
 * after prefill, Sec. 4.2 and Sec. 5.2).  Selects the n_keep[b] - w prefix
 * positions with the largest scores (ties -> lower position), writes them
 * ascending to keep_idx followed by the window positions L[b]-w .. L[b]-1.
 * Scores may be any finite floats (-0 equals +0); NaN is not supported.
 * L, alpha: [host][B] inputs.  n_keep: [host][B] output, filled before return.
 * ws (optional): with ws given and some prefix L[b] - w longer than 32768
 * positions, the prefix is split over several blocks per KV head (same
 * keep_idx, shorter time); ws must then hold
 * tb_workspace_bytes(TB_OP_SELECT, B, Lmax, 0, Hkv, 0, w, 0) bytes (4-byte
 * aligned; contents on entry do not matter), else TB_EWORKSPACE.  With ws
 * NULL, or every prefix at most 32768 positions, one block per KV head
 * selects and ws is not touched. */
tb_status tb_select_topk(const float* scores, int32_t B, const int32_t* L,
                         int32_t Lmax, int32_t Hkv, int32_t w,
                         const double* alpha, int32_t* keep_idx,
                         int32_t* n_keep, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/* Compaction: k_cache[b][g][i] = k[b][g][keep_idx[b][g][i]] (same for v) for
 * i < n_keep[b]; the retained caches are what decoding uses (Sec. 5.2).
 * Sets kv_len[b] = n_keep[b] on the device (stream-ordered).
 * Rows i >= n_keep[b] of the caches are not written.
 * Requires 1 <= n_keep[b] <= min(Lmax, cap), cap % 32 == 0.  Indices should lie in
 * [0, Lmax); the device clamps any other index into that range rather than
 * reading outside the prompt.  Caches must not alias k or v.
 * n_keep: [host][B].  ws: unused (may be NULL). */
tb_status tb_compact_kv(const void* k, const void* v, const int32_t* keep_idx,
                        int32_t B, const int32_t* n_keep, int32_t Lmax,
                        int32_t Hkv, int32_t d, tb_dtype dt, int32_t cap,
                        void* k_cache, void* v_cache, int32_t* kv_len,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* One decode step of grouped-query attention (Sec. 4.2: Q of length 1
 * against the N_kv cached keys).  With k_new/v_new given, row kv_len[b] of
 * the caches receives them, the query attends over kv_len[b] + 1 rows and
 * kv_len[b] is incremented on the device; with both NULL nothing is appended.
 *   out[b][h] = sum_j softmax_j(q[b][h] . K[j] / sqrt(d)) V[j]
 * over the rows of KV head h / (Hq/Hkv).  fp32 accumulation; out in `dt`.
 * Lengths live only on the device, so the call can be captured in a HIP graph.
 * bf16 uses the matrix cores (P rounded to bf16 for the PV product); fp32
 * keeps fp32 products.  Requires cap % 32 == 0.
 * The library cannot see kv_len: the caller must keep kv_len[b] + 1 <= cap
 * when appending.  A device length outside [0, cap] is clamped into it; if
 * kv_len[b] is cap when a row is to be appended, the append is dropped on the
 * device: k_new/v_new are not stored, out[b] is the attention over the cap
 * cached rows (without the new token), kv_len[b] stays cap, and the call
 * still returns TB_OK (the status is decided on the host before any launch).
 * Two kernels are enqueued (chunk partials, then their merge).
 * ws: tb_workspace_bytes(TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, cap) bytes (no
 * initialisation needed).  Calls sharing a workspace must not overlap. */
tb_status tb_decode_attn(const void* q, const void* k_new, const void* v_new,
                         void* k_cache, void* v_cache, int32_t* kv_len,
                         int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                         int32_t cap, tb_dtype dt, void* out, void* ws,
                         size_t ws_bytes, hipStream_t stream);

/* tb_decode_attn without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the chunk partials go to a scratch array
 * of TB_DECODE_SCRATCH_BYTES that the library holds in each GPU's memory from
 * load to process exit.  Same arguments, kernels, launch plan and results as
 * tb_decode_attn.  Calls whose workspace need,
 * tb_workspace_bytes(TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, cap), exceeds the
 * scratch return TB_EWORKSPACE before any launch.  Every call on a GPU uses
 * that GPU's one scratch array: calls that overlap on one GPU (different
 * streams, or graphs replayed concurrently) race and give wrong results;
 * stream-ordered calls are safe.  No memory is allocated or freed (the
 * scratch address is looked up once per device, on the first call there). */
#define TB_DECODE_SCRATCH_BYTES ((size_t)16 << 20)
tb_status tb_decode_attn_noalloc(const void* q, const void* k_new, const void* v_new,
                                 void* k_cache, void* v_cache, int32_t* kv_len,
                                 int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                                 int32_t cap, tb_dtype dt, void* out, hipStream_t stream);

/* ---- paged caches (serving) --------------------------------------------
 * The same compaction and decode over caches kept in pages of 32 rows, one
 * page holding a sequence's 32-row tile for every KV head:
 *   k_pool [n_pages][Hkv][32][d]   K rows, row-major
 *   v_pool [n_pages][Hkv][32][d]   V rows, row-major
 *   block_table [B][max_pages]     int32 (device): row t/32 of sequence b is
 *                                  in page block_table[b][t / 32]
 * A sequence holds up to max_pages * 32 rows (1 <= max_pages <= 2^25, else
 * TB_EUNSUPPORTED; 1 <= n_pages).  The pages a sequence writes
 * (compaction: tiles below n_keep[b]; decode: the tile of row kv_len[b]) must
 * be its own; entries past its length may hold any value (out-of-range
 * entries are clamped into the pool before any read, so they never fault).
 * Results equal the contiguous calls with cap = max_pages * 32. */
tb_status tb_compact_kv_paged(const void* k, const void* v, const int32_t* keep_idx,
                              int32_t B, const int32_t* n_keep, int32_t Lmax, int32_t Hkv,
                              int32_t d, tb_dtype dt, void* k_pool, void* v_pool,
                              int32_t n_pages, const int32_t* block_table, int32_t max_pages,
                              int32_t* kv_len, hipStream_t stream);
/* ws: tb_workspace_bytes(TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, max_pages * 32). */
tb_status tb_decode_attn_paged(const void* q, const void* k_new, const void* v_new,
                               void* k_pool, void* v_pool, int32_t n_pages,
                               const int32_t* block_table, int32_t max_pages,
                               int32_t* kv_len, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                               tb_dtype dt, void* out, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/* Causal grouped-query prefill attention, the step before eviction (the
 * prefill phase of Sec. 4.2, whose time the paper models as
 * a N_x^2 + b N_x + c, Eq. prefill_phase_time_raw):
 *   out[b][h][i] = sum_{j <= i} softmax_j(q[b][h][i] . k[j] / sqrt(d)) v[j]
 * over the rows of KV head h / (Hq/Hkv), for i < L[b].
 *   q, out: [B][Hq][Lmax][d];  k, v: [B][Hkv][Lmax][d]  (rows >= L[b] unread
 *   / unwritten).
 * bf16 only, on the matrix cores; softmax statistics in fp32, P rounded to
 * bf16 for the PV product.  window_stats (nullable, [B][Hq][w][2] fp32)
 * receives, for the last w rows i = L[b]-w+r, the row's logit maximum M (in
 * the units of q.k/sqrt(d)) and Z = sum_j exp(s_j - M): the observation
 * window's softmax statistics as a by-product (the eviction scorer keeps its
 * own float64 statistics; these are fp32).  Requires 1 <= L[b] <= Lmax and,
 * with window_stats, 1 <= w <= L[b].  No workspace. */
tb_status tb_prefill_attn(const void* q, const void* k, const void* v, int32_t B,
                          const int32_t* L, int32_t Lmax, int32_t Hq, int32_t Hkv,
                          int32_t d, tb_dtype dt, void* out, int32_t w,
                          float* window_stats, hipStream_t stream);

/* ---- time-budget controller (host) ------------------------------------ */

/* [host] Least-squares fit of the execution-time model from profiled pairs
 * (Sec. 4.2, profiling-based fitting): degree 1 gives coef = {p, q} of
 * t = p N + q (decode step vs KV length, Eq. decoding_step_time_raw); degree 2
 * gives coef = {a, b, c} of t = a N^2 + b N + c (prefill, Eq.
 * prefill_phase_time_raw).  Returns 0, or -1 on bad arguments / a singular
 * system (fewer than degree + 1 distinct N). */
int32_t tb_ete_fit(const double* n, const double* t, int32_t count, int32_t degree,
                   double* coef);

/* [host] Predicted worst-case execution time (Eq. wcet): prefill plus the
 * decode steps i = 1 .. n_hat_w - 1 at KV length (1 - alpha) n_x + i - 1.
 * prefill_abc = {a, b, c}, step_pq = {p, q}.  NaN on null pointers. */
double tb_wcet(const double* prefill_abc, const double* step_pq, double n_x, double alpha,
               int32_t n_hat_w);

/* [host] Smallest eviction ratio in [0, alpha_max] with
 * t_predict + WCET(alpha) <= budget (Sec. 5.1, Eq. problem_converted), in
 * closed form (Eq. alpha_with_predictor with the second term read as
 * (n_hat_w - 2) / (2 n_x); the printed version also divides it by p, which is
 * dimensionally inconsistent).  *feasible (nullable) is 1 when the budget can
 * be met at or below alpha_max, else 0 and alpha_max is returned.
 * n_hat_w <= 1 (no decode step) gives 0.
 * p = step_pq[0] = 0 (step time independent of the cache length): WCET does
 * not depend on alpha, so the result is 0 with *feasible = 1 when
 * t_predict + prefill + (n_hat_w - 1) q <= budget, else alpha_max with
 * *feasible = 0 (the closed form's limit as p -> 0 from above).
 * Returns NaN with *feasible = 0 for null pointers, n_x <= 0, alpha_max
 * outside [0, 1), p < 0 (not a decode-step model), a non-finite p, q or
 * t_predict, or a NaN budget (+inf means no limit). */
double tb_alpha_star(const double* prefill_abc, const double* step_pq, double n_x,
                     int32_t n_hat_w, double budget, double t_predict, double alpha_max,
                     int32_t* feasible);

/* [host] Response lengths the controller plans with: the predicted length
 * N_hat = min(n_max, n_hat * bucket) from the predictor's bucket index n_hat
 * and bucket size (Sec. 4.1, Eq. predictor_inference), written to *n_hat_len
 * (nullable), and the returned pessimistic length N_hat_W = min(k N_hat, n_max)
 * (Sec. 4.2, the worst-case length ahead of Eq. wcet).  -1 on bad arguments
 * (n_hat < 0, bucket < 1, k < 1, n_max < 0). */
int32_t tb_response_length(int32_t n_hat, int32_t bucket, int32_t k, int32_t n_max,
                           int32_t* n_hat_len);

/* [host] Longest predictor input that runs within the prefill phase
 * (Sec. 5.2, deployment: the response-length predictor runs beside the
 * prefill, and its input prompt is compressed so that its own execution time
 * a_p N_p^2 + b_p N_p + c_p does not exceed a N_x^2 + b N_x + c).  Returns the
 * largest integer N_p in [0, max_len] satisfying that bound, -1 when not even
 * N_p = 0 does, and -2 on bad arguments (null pointers, max_len < 0, n_x < 0,
 * or a_p or b_p negative: the model must grow with length).
 * prefill_abc = {a, b, c}, predict_abc = {a_p, b_p, c_p}. */
int64_t tb_predictor_length(const double* prefill_abc, const double* predict_abc,
                            double n_x, int64_t max_len);

#pragma GCC visibility pop

#ifdef __cplusplus
}
#endif

#endif /* TIMEBILL_H */

// C ABI of libtimebill: host-side validation, workspace carving and launch
// dispatch.  Every check happens before the first HIP call, so an invalid
// call launches nothing.  No exception crosses the boundary.

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <exception>
#include <string>

#include "../../include/timebill.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

tb_status fail(tb_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
tb_status fail(tb_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

tb_status ok() {
  g_err.clear();
  return TB_OK;
}

tb_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(TB_EHIP, "%s: %s", what, hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int32_t keep_count(int32_t L, double alpha, int32_t w) {
  if (!(w > 0 && w < L) || !(alpha >= 0.0 && alpha < 1.0)) return -1;
  const double ev = floor(alpha * static_cast<double>(L));
  const int32_t n = L - static_cast<int32_t>(ev);
  return n < w ? w : n;
}

// Workspace of the several-blocks-per-head selection (prefixes longer than
// tb::kSelMultiMinPrefix); 0 where every prefix is short enough for one block.
size_t select_ws(int32_t B, int32_t Lmax, int32_t Hkv, int32_t w) {
  if (Lmax - w <= tb::kSelMultiMinPrefix) return 0;
  return static_cast<size_t>(B) * Hkv * tb::kSelWsWords * sizeof(uint32_t);
}

bool dtype_ok(tb_dtype dt) { return dt == TB_F32 || dt == TB_BF16; }
int elem_bytes(tb_dtype dt) { return dt == TB_BF16 ? 2 : 4; }

tb_status check_common(int32_t B, int32_t Hq, int32_t Hkv, int32_t d, tb_dtype dt) {
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1 (got %d)", B);
  if (B > tb::kMaxB) return fail(TB_EUNSUPPORTED, "B must be <= %d (got %d)", tb::kMaxB, B);
  if (Hkv < 1 || Hq < 1 || Hq % Hkv != 0)
    return fail(TB_EINVAL, "need Hq %% Hkv == 0 with Hq, Hkv >= 1 (got %d, %d)", Hq, Hkv);
  if (d != 64 && d != 128) return fail(TB_EUNSUPPORTED, "d must be 64 or 128 (got %d)", d);
  if (!dtype_ok(dt)) return fail(TB_EUNSUPPORTED, "dtype must be TB_F32 or TB_BF16");
  return TB_OK;
}

size_t decode_ws(int32_t B, int32_t Hkv, int32_t G, int32_t d, int32_t cap, bool bf16) {
  const size_t n_chunks = tb::decode_plan(B, Hkv, cap, bf16).n_chunks;
  const size_t part = static_cast<size_t>(B) * Hkv * n_chunks * G * (d + tb::kPartPad) * sizeof(float);
  return align256(part) + align256(static_cast<size_t>(B) * sizeof(int32_t));
}

}  // namespace

namespace tb {

// How a decode step splits the cache (bf16).  Measured on one layer (cache
// resident in the last-level cache) and on the 28-layer shape (each layer's
// cache streamed from HBM), 410..32768 rows per KV head, graph-replayed steps:
// * One partial block per CU: a KV head gets C = floor(256 / units) blocks,
//   and its cap/32 tiles are split between them as evenly as whole tiles
//   allow (blocks of a fixed row count left up to 48 CUs idle; a second
//   round of blocks past 256 doubles the step time).
// * A block's tiles are shared by 1, 2, 4 or 8 waves: with two waves per
//   SIMD (the register budget) more waves keep more tiles in flight per CU,
//   but each wave also stages its tile's V rows through LDS, and a wave with
//   a single tile cannot hide that.  Measured with the row-major V cache at
//   28 layers (us per layer-step, 2-16 tiles per block): 2 tiles, one wave
//   9.51 against 9.62 (two); 3 tiles, two waves 10.26 against 10.64 (one);
//   4-7 tiles, four waves 11.37-13.08 against 11.59-13.42 (two); 8 tiles,
//   four waves 13.31 against 13.52 (eight); 9-16 tiles, eight waves 14.56-
//   19.13 against 14.68-19.22 (four).
// * Small caches (<= 2048 rows) keep at most 32 partials per KV head (blocks
//   of up to two tiles).  Measured with the quarter-head merge waves (us per
//   layer-step or per 28-layer token, two runs each, alternated): 2304 rows
//   6.85 against 7.10 with the cap (so the earlier 2560-row threshold was
//   lowered), 1792 rows 206.9 against 207.3-207.8 us per token without it.
// * Batches (B > 1) are usually ragged, and the plan sees only the capacity:
//   blocks past a sequence's length exit at once, so small blocks (one wave,
//   about 12 tiles) balance the real work across CUs.  On ragged batches and
//   a 64-request serving stream this was 11-28% faster than one block per CU
//   per KV head; on uniform batches it costs 2-6%.
// fp32 runs the vector-ALU kernel over blocks of `chunk` rows.
DecodePlan decode_plan(int B, int Hkv, int cap, bool bf16) {
  const long long units = static_cast<long long>(B) * Hkv;
  DecodePlan p{};
  if (!bf16) {
    p.waves = 1;
    const long long unit = decode_chunk_unit(1, false);
    long long want = (static_cast<long long>(cap) * units + 255) / 256;
    want = std::min<long long>(std::max<long long>(want, unit), 1024);
    want = std::max<long long>(want, (cap + decode_max_chunks() - 1) / decode_max_chunks());
    p.chunk = static_cast<int32_t>((want + unit - 1) / unit * unit);
    p.n_chunks = (cap + p.chunk - 1) / p.chunk;
    return p;
  }
  const long long tiles = std::max<long long>(1, cap / kVTile);
  long long C = std::max<long long>(1, 256 / units);
  if (cap <= 2048) C = std::min<long long>(C, 32);
  C = std::min(C, tiles);
  constexpr long long kBatchTiles = 12;
  const bool batch = B > 1 && tiles / C > kBatchTiles;
  if (batch) C = (tiles + kBatchTiles - 1) / kBatchTiles;
  C = std::max<long long>(1, std::min<long long>({C, tiles, decode_max_chunks()}));
  const long long per_block = tiles / C;       // every block holds per_block or per_block + 1
  int waves = 1;
  if (!batch) waves = per_block >= 9 ? 8 : per_block >= 4 ? 4 : per_block >= 3 ? 2 : 1;
  p.waves = waves;
  p.n_chunks = static_cast<int32_t>(C);
  p.chunk = static_cast<int32_t>((tiles + C - 1) / C * kVTile);   // rows of the largest block
  return p;
}

}  // namespace tb

extern "C" {

int32_t tb_keep_count(int32_t L, double alpha, int32_t w) { return keep_count(L, alpha, w); }

const char* tb_last_error(void) { return g_err.c_str(); }

size_t tb_workspace_bytes(int32_t op, int32_t B, int32_t Lmax, int32_t Hq, int32_t Hkv,
                          int32_t d, int32_t w, int32_t cap) {
  try {
    switch (op) {
      case TB_OP_SCORE: {
        if (B < 1 || Lmax < 1 || Hkv < 1 || Hq < 1 || Hq % Hkv != 0 || w < 1 ||
            static_cast<long long>(Hq / Hkv) * w > 1024) {
          fail(TB_EINVAL, "tb_workspace_bytes(SCORE): bad sizes");
          return 0;
        }
        return tb::score_ws_bytes(B, Lmax, Hkv, (Hq / Hkv) * w);
      }
      case TB_OP_SELECT: {
        if (B < 1 || Lmax < 1 || Hkv < 1 || w < 1) {
          fail(TB_EINVAL, "tb_workspace_bytes(SELECT): bad sizes");
          return 0;
        }
        return select_ws(B, Lmax, Hkv, w);
      }
      case TB_OP_COMPACT:
        return 0;
      case TB_OP_H2O: {
        if (B < 1 || Lmax < 1 || Hkv < 1 || Hq < 1 || Hq % Hkv != 0) {
          fail(TB_EINVAL, "tb_workspace_bytes(H2O): bad sizes");
          return 0;
        }
        return tb::h2o_ws_bytes(B, Lmax, Hq);
      }
      case TB_OP_DECODE: {
        if (B < 1 || Hkv < 1 || Hq < 1 || Hq % Hkv != 0 || cap < 1 || d < 1) {
          fail(TB_EINVAL, "tb_workspace_bytes(DECODE): bad sizes");
          return 0;
        }
        // sized for the larger of the two dtype decompositions, and for every
        // batch size up to B (the split depends on the batch size, so a caller
        // that sizes for its largest batch can run any smaller one)
        size_t need = 0;
        for (int32_t b = 1; b <= B; ++b)
          need = std::max({need, decode_ws(b, Hkv, Hq / Hkv, d, cap, true),
                           decode_ws(b, Hkv, Hq / Hkv, d, cap, false)});
        return need;
      }
      default:
        fail(TB_EINVAL, "tb_workspace_bytes: unknown op %d", op);
        return 0;
    }
  } catch (...) {
    fail(TB_EINTERNAL, "tb_workspace_bytes: internal error");
    return 0;
  }
}

namespace {

tb_status score_window_impl(const char* name, bool avg, const void* q_win, const void* k,
                            int32_t B, const int32_t* L, int32_t Lmax, int32_t Hq, int32_t Hkv,
                            int32_t d, int32_t w, int32_t pool, tb_dtype dt, float* scores,
                            float* raw_scores, void* ws, size_t ws_bytes, hipStream_t stream) {
  try {
    if (!q_win || !k || !L || !scores) return fail(TB_EINVAL, "%s: null pointer", name);
    tb_status st = check_common(B, Hq, Hkv, d, dt);
    if (st != TB_OK) return st;
    if (w < 1) return fail(TB_EINVAL, "w must be >= 1 (got %d)", w);
    if (pool < 1 || pool % 2 == 0) return fail(TB_EINVAL, "pool must be odd and >= 1 (got %d)", pool);
    if (pool > 129) return fail(TB_EUNSUPPORTED, "pool must be <= 129 (got %d)", pool);
    const long long R64 = static_cast<long long>(Hq / Hkv) * w;     // no int overflow for huge w
    if (R64 > 1024) return fail(TB_EUNSUPPORTED, "(Hq/Hkv)*w must be <= 1024 (got %lld)", R64);
    const int R = static_cast<int>(R64);
    for (int b = 0; b < B; ++b)
      if (!(L[b] > w && L[b] <= Lmax))
        return fail(TB_EINVAL, "need w < L[%d] <= Lmax (w=%d, L=%d, Lmax=%d)", b, w, L[b], Lmax);
    const size_t need = tb::score_ws_bytes(B, Lmax, Hkv, R);
    if (ws_bytes < need || (need > 0 && !ws))
      return fail(TB_EWORKSPACE, "%s: workspace %zu < %zu bytes", name, ws_bytes, need);

    tb::ScoreArgs a{};
    a.q_win = q_win; a.k = k; a.scores = scores; a.raw_scores = raw_scores;
    a.B = B; a.Lmax = Lmax; a.Hq = Hq; a.Hkv = Hkv; a.w = w; a.pool = pool; a.R = R;
    a.pool_avg = avg ? 1 : 0;
    a.n_tiles = (Lmax + tb::kScoreTile - 1) / tb::kScoreTile;
    a.row_chunks = (R + tb::kScoreRows - 1) / tb::kScoreRows;
    a.scale = 1.0 / sqrt(static_cast<double>(d));
    for (int b = 0; b < B; ++b) a.L[b] = L[b];
    const size_t units = static_cast<size_t>(B) * Hkv;
    char* p = static_cast<char*>(ws);
    a.e = reinterpret_cast<float*>(p);
    p += align256(units * a.n_tiles * R * tb::kScoreTile * sizeof(float));
    a.tile_m = reinterpret_cast<double*>(p);
    p += align256(units * a.n_tiles * R * sizeof(double));
    a.tile_z = reinterpret_cast<double*>(p);
    p += align256(units * a.n_tiles * R * sizeof(double));
    a.row_M = reinterpret_cast<double*>(p);
    p += align256(units * R * sizeof(double));
    a.row_Z = reinterpret_cast<double*>(p);
    p += align256(units * R * sizeof(double));
    a.raw = raw_scores ? raw_scores : reinterpret_cast<float*>(p);
    return hip_status(tb::launch_score(a, d, dt == TB_BF16, stream), name);
  } catch (const std::exception& e) {
    return fail(TB_EINTERNAL, "%s: %s", name, e.what());
  } catch (...) {
    return fail(TB_EINTERNAL, "%s: internal error", name);
  }
}

}  // namespace

tb_status tb_score_window(const void* q_win, const void* k, int32_t B, const int32_t* L,
                          int32_t Lmax, int32_t Hq, int32_t Hkv, int32_t d, int32_t w,
                          int32_t pool, tb_dtype dt, float* scores, float* raw_scores,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  return score_window_impl("tb_score_window", false, q_win, k, B, L, Lmax, Hq, Hkv, d, w, pool,
                           dt, scores, raw_scores, ws, ws_bytes, stream);
}

tb_status tb_score_window_avgpool(const void* q_win, const void* k, int32_t B, const int32_t* L,
                                  int32_t Lmax, int32_t Hq, int32_t Hkv, int32_t d, int32_t w,
                                  int32_t pool, tb_dtype dt, float* scores, float* raw_scores,
                                  void* ws, size_t ws_bytes, hipStream_t stream) {
  return score_window_impl("tb_score_window_avgpool", true, q_win, k, B, L, Lmax, Hq, Hkv, d, w,
                           pool, dt, scores, raw_scores, ws, ws_bytes, stream);
}

tb_status tb_score_h2o(const void* q, const void* k, int32_t B, const int32_t* L, int32_t Lmax,
                       int32_t Hq, int32_t Hkv, int32_t d, tb_dtype dt, float* scores, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  try {
    if (!q || !k || !L || !scores) return fail(TB_EINVAL, "tb_score_h2o: null pointer");
    tb_status st = check_common(B, Hq, Hkv, d, dt);
    if (st != TB_OK) return st;
    tb::H2oArgs a{};
    for (int b = 0; b < B; ++b) {
      if (!(L[b] >= 1 && L[b] <= Lmax))
        return fail(TB_EINVAL, "need 1 <= L[%d] <= Lmax (L=%d, Lmax=%d)", b, L[b], Lmax);
      a.L[b] = L[b];
    }
    const size_t need = tb::h2o_ws_bytes(B, Lmax, Hq);
    if (ws_bytes < need || !ws)
      return fail(TB_EWORKSPACE, "tb_score_h2o: workspace %zu < %zu bytes", ws_bytes, need);
    const size_t part = align256(static_cast<size_t>(B) * Hq * Lmax * sizeof(double));
    char* p = static_cast<char*>(ws);
    a.row_M = reinterpret_cast<double*>(p);
    a.row_Z = reinterpret_cast<double*>(p + part);
    a.col_part = reinterpret_cast<double*>(p + 2 * part);
    a.q = q; a.k = k; a.scores = scores;
    a.B = B; a.Lmax = Lmax; a.Hq = Hq; a.Hkv = Hkv;
    a.scale = 1.0 / sqrt(static_cast<double>(d));
    return hip_status(tb::launch_h2o(a, d, dt == TB_BF16, stream), "tb_score_h2o launch");
  } catch (...) {
    return fail(TB_EINTERNAL, "tb_score_h2o: internal error");
  }
}

tb_status tb_prefill_attn(const void* q, const void* k, const void* v, int32_t B,
                          const int32_t* L, int32_t Lmax, int32_t Hq, int32_t Hkv, int32_t d,
                          tb_dtype dt, void* out, int32_t w, float* window_stats,
                          hipStream_t stream) {
  try {
    if (!q || !k || !v || !L || !out) return fail(TB_EINVAL, "tb_prefill_attn: null pointer");
    tb_status st = check_common(B, Hq, Hkv, d, dt);
    if (st != TB_OK) return st;
    if (dt != TB_BF16) return fail(TB_EUNSUPPORTED, "tb_prefill_attn: bf16 only");
    if (window_stats && w < 1) return fail(TB_EINVAL, "w must be >= 1 when window_stats is given");
    tb::PrefillArgs a{};
    for (int b = 0; b < B; ++b) {
      if (!(L[b] >= 1 && L[b] <= Lmax))
        return fail(TB_EINVAL, "need 1 <= L[%d] <= Lmax (L=%d, Lmax=%d)", b, L[b], Lmax);
      if (window_stats && w > L[b])
        return fail(TB_EINVAL, "need w <= L[%d] (w=%d, L=%d)", b, w, L[b]);
      a.L[b] = L[b];
    }
    a.q = q; a.k = k; a.v = v; a.out = out; a.window_stats = window_stats;
    a.B = B; a.Lmax = Lmax; a.Hq = Hq; a.Hkv = Hkv; a.w = window_stats ? w : 0;
    a.scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(d)));
    return hip_status(tb::launch_prefill(a, d, stream), "tb_prefill_attn launch");
  } catch (...) {
    return fail(TB_EINTERNAL, "tb_prefill_attn: internal error");
  }
}

tb_status tb_score_knorm(const void* k, int32_t B, const int32_t* L, int32_t Lmax, int32_t Hkv,
                         int32_t d, int32_t w, tb_dtype dt, float* scores, hipStream_t stream) {
  try {
    if (!k || !L || !scores) return fail(TB_EINVAL, "tb_score_knorm: null pointer");
    tb_status st = check_common(B, Hkv, Hkv, d, dt);
    if (st != TB_OK) return st;
    if (w < 1) return fail(TB_EINVAL, "w must be >= 1 (got %d)", w);
    tb::KnormArgs a{};
    for (int b = 0; b < B; ++b) {
      if (!(L[b] > w && L[b] <= Lmax))
        return fail(TB_EINVAL, "need w < L[%d] <= Lmax (w=%d, L=%d, Lmax=%d)", b, w, L[b], Lmax);
      a.L[b] = L[b];
    }
    a.k = k; a.scores = scores; a.B = B; a.Lmax = Lmax; a.Hkv = Hkv; a.w = w;
    return hip_status(tb::launch_knorm(a, d, dt == TB_BF16, stream), "tb_score_knorm launch");
  } catch (...) {
    return fail(TB_EINTERNAL, "tb_score_knorm: internal error");
  }
}

tb_status tb_select_topk(const float* scores, int32_t B, const int32_t* L, int32_t Lmax,
                         int32_t Hkv, int32_t w, const double* alpha, int32_t* keep_idx,
                         int32_t* n_keep, void* ws, size_t ws_bytes, hipStream_t stream) {
  try {
    if (!scores || !L || !alpha || !keep_idx || !n_keep)
      return fail(TB_EINVAL, "tb_select_topk: null pointer");
    if (B < 1) return fail(TB_EINVAL, "B must be >= 1 (got %d)", B);
    if (B > tb::kMaxB) return fail(TB_EUNSUPPORTED, "B must be <= %d (got %d)", tb::kMaxB, B);
    if (Hkv < 1) return fail(TB_EINVAL, "Hkv must be >= 1");
    if (w < 1) return fail(TB_EINVAL, "w must be >= 1 (got %d)", w);
    tb::SelectArgs a{};
    for (int b = 0; b < B; ++b) {
      if (!(L[b] > w && L[b] <= Lmax))
        return fail(TB_EINVAL, "need w < L[%d] <= Lmax (w=%d, L=%d, Lmax=%d)", b, w, L[b], Lmax);
      if (!(alpha[b] >= 0.0 && alpha[b] < 1.0))
        return fail(TB_EINVAL, "alpha[%d] must be in [0, 1) (got %g)", b, alpha[b]);
      a.L[b] = L[b];
      a.n_keep[b] = keep_count(L[b], alpha[b], w);
    }
    a.scores = scores; a.keep_idx = keep_idx;
    a.B = B; a.Lmax = Lmax; a.Hkv = Hkv; a.w = w;
    int max_pref = 0;
    for (int b = 0; b < B; ++b) max_pref = std::max(max_pref, L[b] - w);
    const size_t need = select_ws(B, Lmax, Hkv, w);
    const bool multi = ws != nullptr && max_pref > tb::kSelMultiMinPrefix;
    if (multi && ws_bytes < need)
      return fail(TB_EWORKSPACE, "tb_select_topk: workspace %zu bytes < %zu", ws_bytes, need);
    if (multi && reinterpret_cast<uintptr_t>(ws) % 4 != 0)
      return fail(TB_EINVAL, "tb_select_topk: workspace must be 4-byte aligned");
    for (int b = 0; b < B; ++b) n_keep[b] = a.n_keep[b];
    return hip_status(multi ? tb::launch_select_multi(a, ws, stream) : tb::launch_select(a, stream),
                      "tb_select_topk launch");
  } catch (...) {
    return fail(TB_EINTERNAL, "tb_select_topk: internal error");
  }
}

namespace {

// Paged caches: table [B][max_pages] of page indices into pools of n_pages
// pages; a sequence holds up to max_pages * 32 rows.
struct Paging {
  const int32_t* table;
  int32_t max_pages, n_pages;
};

tb_status compact_impl(const char* name, const void* k, const void* v, const int32_t* keep_idx,
                       int32_t B, const int32_t* n_keep, int32_t Lmax, int32_t Hkv, int32_t d,
                       tb_dtype dt, int32_t cap, const Paging* pg, void* k_cache, void* v_cache,
                       int32_t* kv_len, hipStream_t stream) {
  try {
    if (!k || !v || !keep_idx || !n_keep || !k_cache || !v_cache || !kv_len)
      return fail(TB_EINVAL, "%s: null pointer", name);
    tb_status st = check_common(B, Hkv, Hkv, d, dt);
    if (st != TB_OK) return st;
    if (Lmax < 1 || cap < 1) return fail(TB_EINVAL, "Lmax and cap must be >= 1");
    if (cap % tb::kVTile != 0)
      return fail(TB_EINVAL, "cap must be a multiple of %d (got %d)", tb::kVTile, cap);
    tb::CompactArgs a{};
    int max_keep = 0;
    for (int b = 0; b < B; ++b) {
      if (!(n_keep[b] >= 1 && n_keep[b] <= Lmax && n_keep[b] <= cap))
        return fail(TB_EINVAL, "need 1 <= n_keep[%d] <= min(Lmax, cap) (n_keep=%d, Lmax=%d, cap=%d)",
                    b, n_keep[b], Lmax, cap);
      a.n_keep[b] = n_keep[b];
      max_keep = std::max(max_keep, n_keep[b]);
    }
    a.k = k; a.v = v; a.keep_idx = keep_idx; a.k_cache = k_cache; a.v_cache = v_cache;
    a.kv_len = kv_len; a.B = B; a.Lmax = Lmax; a.Hkv = Hkv; a.cap = cap;
    if (pg) { a.table = pg->table; a.max_pages = pg->max_pages; a.n_pages = pg->n_pages; }
    return hip_status(tb::launch_compact(a, d, elem_bytes(dt), max_keep, stream), name);
  } catch (...) {
    return fail(TB_EINTERNAL, "%s: internal error", name);
  }
}

// use_scratch: the partials go to the library-held scratch array (ws and
// ws_bytes are ignored); the need is checked against its size before any HIP
// call.
tb_status decode_impl(const char* name, const void* q, const void* k_new, const void* v_new,
                      void* k_cache, void* v_cache, int32_t* kv_len, int32_t B, int32_t Hq,
                      int32_t Hkv, int32_t d, int32_t cap, const Paging* pg, tb_dtype dt,
                      void* out, void* ws, size_t ws_bytes, hipStream_t stream,
                      bool use_scratch = false) {
  try {
    if (!q || !k_cache || !v_cache || !kv_len || !out || (!ws && !use_scratch))
      return fail(TB_EINVAL, "%s: null pointer", name);
    if ((k_new == nullptr) != (v_new == nullptr))
      return fail(TB_EINVAL, "%s: k_new and v_new must both be given or both NULL", name);
    tb_status st = check_common(B, Hq, Hkv, d, dt);
    if (st != TB_OK) return st;
    const int G = Hq / Hkv;
    if (G > 8) return fail(TB_EUNSUPPORTED, "Hq/Hkv must be <= 8 for decoding (got %d)", G);
    if (cap < 1) return fail(TB_EINVAL, "cap must be >= 1");
    if (cap % tb::kVTile != 0)
      return fail(TB_EINVAL, "cap must be a multiple of %d (got %d)", tb::kVTile, cap);
    const bool bf16 = dt == TB_BF16;
    const size_t need = decode_ws(B, Hkv, G, d, cap, bf16);
    if (use_scratch) {
      if (need > TB_DECODE_SCRATCH_BYTES)
        return fail(TB_EWORKSPACE,
                    "%s: this call needs %zu bytes of workspace; the library's scratch holds "
                    "%zu (use tb_decode_attn with a workspace)",
                    name, need, static_cast<size_t>(TB_DECODE_SCRATCH_BYTES));
      const hipError_t e = tb::decode_scratch(&ws);
      if (e != hipSuccess) return hip_status(e, "decode scratch lookup");
      ws_bytes = TB_DECODE_SCRATCH_BYTES;
    }
    if (ws_bytes < need)
      return fail(TB_EWORKSPACE, "%s: workspace %zu < %zu bytes", name, ws_bytes, need);
    tb::DecodeArgs a{};
    a.q = q; a.k_new = k_new; a.v_new = v_new; a.k_cache = k_cache; a.v_cache = v_cache;
    a.kv_len = kv_len; a.out = out;
    a.B = B; a.Hkv = Hkv; a.cap = cap;
    if (pg) { a.table = pg->table; a.max_pages = pg->max_pages; a.n_pages = pg->n_pages; }
    const tb::DecodePlan plan = tb::decode_plan(B, Hkv, cap, bf16);
    a.chunk = plan.chunk;
    a.n_chunks = plan.n_chunks;
    a.waves = plan.waves;
    a.tiles_q = (cap / tb::kVTile) / plan.n_chunks;
    a.tiles_r = (cap / tb::kVTile) % plan.n_chunks;
    a.append = k_new != nullptr;
    a.scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(d)));
    char* p = static_cast<char*>(ws);
    a.part = reinterpret_cast<float*>(p);
    p += align256(static_cast<size_t>(B) * Hkv * a.n_chunks * G * (d + tb::kPartPad) * sizeof(float));
    a.seq_len = reinterpret_cast<int32_t*>(p);
    return hip_status(tb::launch_decode(a, G, d, bf16, stream), name);
  } catch (...) {
    return fail(TB_EINTERNAL, "%s: internal error", name);
  }
}

tb_status check_paging(const char* name, const int32_t* table, int32_t max_pages,
                       int32_t n_pages) {
  if (!table) return fail(TB_EINVAL, "%s: null block table", name);
  if (max_pages < 1 || n_pages < 1)
    return fail(TB_EINVAL, "%s: max_pages and n_pages must be >= 1 (got %d, %d)", name,
                max_pages, n_pages);
  // the capacity max_pages * 32 rows must stay a positive int32
  if (max_pages > (1 << 25))
    return fail(TB_EUNSUPPORTED, "%s: max_pages must be <= 2^25 (got %d)", name, max_pages);
  return TB_OK;
}

}  // namespace

tb_status tb_compact_kv(const void* k, const void* v, const int32_t* keep_idx, int32_t B,
                        const int32_t* n_keep, int32_t Lmax, int32_t Hkv, int32_t d,
                        tb_dtype dt, int32_t cap, void* k_cache, void* v_cache,
                        int32_t* kv_len, void* ws, size_t ws_bytes, hipStream_t stream) {
  (void)ws; (void)ws_bytes;
  return compact_impl("tb_compact_kv", k, v, keep_idx, B, n_keep, Lmax, Hkv, d, dt, cap, nullptr,
                      k_cache, v_cache, kv_len, stream);
}

tb_status tb_compact_kv_paged(const void* k, const void* v, const int32_t* keep_idx, int32_t B,
                              const int32_t* n_keep, int32_t Lmax, int32_t Hkv, int32_t d,
                              tb_dtype dt, void* k_pool, void* v_pool, int32_t n_pages,
                              const int32_t* block_table, int32_t max_pages, int32_t* kv_len,
                              hipStream_t stream) {
  tb_status st = check_paging("tb_compact_kv_paged", block_table, max_pages, n_pages);
  if (st != TB_OK) return st;
  const Paging pg{block_table, max_pages, n_pages};
  return compact_impl("tb_compact_kv_paged", k, v, keep_idx, B, n_keep, Lmax, Hkv, d, dt,
                      max_pages * tb::kVTile, &pg, k_pool, v_pool, kv_len, stream);
}

tb_status tb_decode_attn(const void* q, const void* k_new, const void* v_new, void* k_cache,
                         void* v_cache, int32_t* kv_len, int32_t B, int32_t Hq, int32_t Hkv,
                         int32_t d, int32_t cap, tb_dtype dt, void* out, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  return decode_impl("tb_decode_attn", q, k_new, v_new, k_cache, v_cache, kv_len, B, Hq, Hkv, d,
                     cap, nullptr, dt, out, ws, ws_bytes, stream);
}

tb_status tb_decode_attn_noalloc(const void* q, const void* k_new, const void* v_new,
                                 void* k_cache, void* v_cache, int32_t* kv_len, int32_t B,
                                 int32_t Hq, int32_t Hkv, int32_t d, int32_t cap, tb_dtype dt,
                                 void* out, hipStream_t stream) {
  return decode_impl("tb_decode_attn_noalloc", q, k_new, v_new, k_cache, v_cache, kv_len, B, Hq,
                     Hkv, d, cap, nullptr, dt, out, nullptr, 0, stream, /*use_scratch=*/true);
}

tb_status tb_decode_attn_paged(const void* q, const void* k_new, const void* v_new,
                               void* k_pool, void* v_pool, int32_t n_pages,
                               const int32_t* block_table, int32_t max_pages, int32_t* kv_len,
                               int32_t B, int32_t Hq, int32_t Hkv, int32_t d, tb_dtype dt,
                               void* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  tb_status st = check_paging("tb_decode_attn_paged", block_table, max_pages, n_pages);
  if (st != TB_OK) return st;
  const Paging pg{block_table, max_pages, n_pages};
  return decode_impl("tb_decode_attn_paged", q, k_new, v_new, k_pool, v_pool, kv_len, B, Hq, Hkv,
                     d, max_pages * tb::kVTile, &pg, dt, out, ws, ws_bytes, stream);
}


}  // extern "C"

// Launch-argument structs and launchers of the gfx950 kernels.  The C ABI in
// api.hip validates every argument before calling these.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tb {

constexpr int kMaxB = 64;        // per-sequence values travel in kernel arguments
constexpr int kScoreTile = 64;   // keys per scoring tile
constexpr int kScoreRows = 256;  // window rows per scoring block
constexpr int kVTile = 32;       // rows per tile of the compact caches (and per page)
// Floats after the d outputs of a decode partial record (m, l, padding): with
// d + kPartPad floats per record every 32-value slice a merge wave reads is
// one 128-byte line (with d + 4: two lines for most slices; measured 13.53
// against 13.61 us per decode call on the 28-layer L = 32768 benchmark).
constexpr int kPartPad = 32;

// ---------------------------------------------------------------- scoring
struct ScoreArgs {
  const void* q_win;      // [B][Hq][w][d]
  const void* k;          // [B][Hkv][Lmax][d]
  float* scores;          // [B][Hkv][Lmax]
  float* raw_scores;      // nullable, same layout
  float* e;               // ws: [B][Hkv][n_tiles][R][64] exp(s - tile max), fp32
  double* tile_m;         // ws: [B][Hkv][R][n_tiles]
  double* tile_z;         // ws: [B][Hkv][R][n_tiles]
  double* row_M;          // ws: [B][Hkv][R]
  double* row_Z;          // ws: [B][Hkv][R]
  float* raw;             // raw scores: raw_scores if given, else ws [B][Hkv][Lmax]
  int32_t B, Lmax, Hq, Hkv, w, pool, R, n_tiles, row_chunks;
  int32_t pool_avg;       // 0: max-pool, 1: mean over the window (zeros outside the prefix)
  int32_t stream_e;       // set by launch_score: e written with streaming stores
  int32_t pack_pairs;     // set by launch_score: row pairs P of packed K1 blocks, 0 if unpacked
  double scale;           // 1/sqrt(d)
  int32_t L[kMaxB];
};
size_t score_ws_bytes(int B, int Lmax, int Hkv, int R);
hipError_t launch_score(const ScoreArgs& a, int d, bool bf16, hipStream_t st);

// ---------------------------------------------------------------- KNorm
struct KnormArgs {
  const void* k;          // [B][Hkv][Lmax][d]
  float* scores;          // [B][Hkv][Lmax]: -||k_j|| for j < L[b] - w
  int32_t B, Lmax, Hkv, w;
  int32_t L[kMaxB];
};
hipError_t launch_knorm(const KnormArgs& a, int d, bool bf16, hipStream_t st);

// ---------------------------------------------------------------- H2O
struct H2oArgs {
  const void* q;          // [B][Hq][Lmax][d]  all prompt queries
  const void* k;          // [B][Hkv][Lmax][d]
  float* scores;          // [B][Hkv][Lmax]: accumulated attention for j < L[b]
  double* row_M;          // ws: [B][Hq][Lmax] row max (logit units)
  double* row_Z;          // ws: [B][Hq][Lmax] row normaliser
  double* col_part;       // ws: [B][Hq][Lmax] per-head column mass
  int32_t B, Lmax, Hq, Hkv;
  double scale;           // 1/sqrt(d)
  int32_t L[kMaxB];
};
size_t h2o_ws_bytes(int B, int Lmax, int Hq);
hipError_t launch_h2o(const H2oArgs& a, int d, bool bf16, hipStream_t st);

// ---------------------------------------------------------------- prefill
struct PrefillArgs {
  const void* q;          // [B][Hq][Lmax][d] bf16
  const void* k;          // [B][Hkv][Lmax][d]
  const void* v;          // [B][Hkv][Lmax][d]
  void* out;              // [B][Hq][Lmax][d]
  float* window_stats;    // nullable [B][Hq][w][2]: (row max, normaliser) of the last w rows
  int32_t B, Lmax, Hq, Hkv, w;
  float scale_log2;       // log2(e)/sqrt(d)
  int32_t L[kMaxB];
};
hipError_t launch_prefill(const PrefillArgs& a, int d, hipStream_t st);

// ---------------------------------------------------------------- selection
struct SelectArgs {
  const float* scores;    // [B][Hkv][Lmax]
  int32_t* keep_idx;      // [B][Hkv][Lmax]
  int32_t B, Lmax, Hkv, w;
  int32_t L[kMaxB];
  int32_t n_keep[kMaxB];
};
hipError_t launch_select(const SelectArgs& a, hipStream_t st);
// Several blocks per (sequence, KV head); ws holds kSelWsWords 32-bit words per
// unit, B * Hkv units.
constexpr int kSelMaxChunks = 32;
constexpr int kSelWsWords = 4 * kSelMaxChunks + 8 + 3 * 2048;
constexpr int kSelMultiMinPrefix = 32768;   // longer prefixes go to several blocks
int select_chunks(int max_pref);
hipError_t launch_select_multi(const SelectArgs& a, void* ws, hipStream_t st);

// ---------------------------------------------------------------- compaction
struct CompactArgs {
  const void* k;          // [B][Hkv][Lmax][d]
  const void* v;
  const int32_t* keep_idx;  // [B][Hkv][Lmax]
  void* k_cache;          // [B][Hkv][cap][d]
  void* v_cache;          // [B][Hkv][cap][d]
  int32_t* kv_len;        // [B]
  int32_t B, Lmax, Hkv, cap;
  // paged caches (table != nullptr): tile t of sequence b lives in page
  // table[b * max_pages + t] of pools [n_pages][Hkv][32][d] (K and V)
  const int32_t* table;
  int32_t max_pages, n_pages;
  int32_t n_keep[kMaxB];
};
hipError_t launch_compact(const CompactArgs& a, int d, int elem_bytes, int max_keep,
                          hipStream_t st);

// ---------------------------------------------------------------- decode
// Element offset of the 32-row tile t of (sequence b, KV head g) in the K
// cache and in the V cache (the same offset for both).  Contiguous caches:
// [B][Hkv][cap][d]; paged: pools [n_pages][Hkv][32][d], page from the block
// table, clamped into the pool.
template <bool PAGED, typename Args>
__device__ __forceinline__ size_t cache_tile_off(const Args& a, int b, int g, int t, int d) {
  if constexpr (PAGED) {
    int page = a.table[static_cast<size_t>(b) * a.max_pages + t];
    page = page < 0 ? 0 : (page >= a.n_pages ? a.n_pages - 1 : page);
    return (static_cast<size_t>(page) * a.Hkv + g) * kVTile * d;
  } else {
    return ((static_cast<size_t>(b) * a.Hkv + g) * a.cap + static_cast<size_t>(t) * kVTile) * d;
  }
}

struct DecodeArgs {
  const void* q;          // [B][Hq][d]
  const void* k_new;      // [B][Hkv][d] (unused when append == 0)
  const void* v_new;
  void* k_cache;          // [B][Hkv][cap][d]
  void* v_cache;          // [B][Hkv][cap][d]
  int32_t* kv_len;        // [B]
  void* out;              // [B][Hq][d]
  float* part;            // ws: [B][Hkv][n_chunks][G][d+kPartPad] chunk partials (o, m, l)
  int32_t* seq_len;       // ws: [B] attended length of this step
  int32_t B, Hkv, cap, chunk, n_chunks, append;
  int32_t waves;          // waves per partial block (bf16: 1 or 4)
  int32_t tiles_q, tiles_r;  // bf16: (cap / 32) / n_chunks and (cap / 32) % n_chunks
  const int32_t* table;   // paged caches (nullptr: contiguous); see CompactArgs
  int32_t max_pages, n_pages;
  float scale_log2;       // log2(e)/sqrt(d)
};
// How a decode launch splits the cache: rows per block, blocks per KV head and
// waves per block (every wave takes chunk / waves rows).
struct DecodePlan {
  int32_t chunk, n_chunks, waves;
};
DecodePlan decode_plan(int B, int Hkv, int cap, bool bf16);
int decode_chunk_unit(int waves, bool bf16);
int decode_max_chunks();
hipError_t launch_decode(const DecodeArgs& a, int G, int d, bool bf16, hipStream_t st);
// The current device's address of the library-held decode scratch array
// (TB_DECODE_SCRATCH_BYTES); looked up once per device.
hipError_t decode_scratch(void** ptr);

}  // namespace tb

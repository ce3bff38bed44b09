// Single-token grouped-query decode attention over the compact KV cache,
// with the new token's K/V appended in the same step.
//
// Cache layout: K and V rows are row-major, [B][Hkv][cap][d].  The kernels
// walk the cache in tiles of 32 rows; paged caches (a block table per
// sequence) keep those tiles as pages of pools [pages][Hkv][32][d], and a
// wave's 32-row step starts with one table lookup.  The matrix-core PV
// product wants "8 consecutive keys of one V column" per lane: each wave
// copies a tile's V rows into its own LDS buffer (16-byte chunks swizzled by
// row) and reads the operand back with the gfx950 transpose read.  Measured
// against a cache stored as transposed 32-row tiles (one 16-byte global load
// per operand, no LDS): bit-identical, 0-3.5% faster for caches of 8k-33k
// rows, 4-7% slower below 4k rows (one wave per block, where the LDS round
// trip is not hidden).
//
// Two launches per decode step and layer (both capturable in a HIP graph):
//   partial kernel, grid = (n_chunks, Hkv, B): block (c, g, b) covers a
//     share of the 32-row tiles of KV head g of sequence b for all
//     G = Hq/Hkv query heads of the group, so every K/V byte is read from HBM
//     once per step, and writes one partial (m, l, o[G][d]).  bf16: the cap/32
//     tiles are split as evenly as whole tiles allow (T tiles, C blocks: the
//     first T mod C blocks take one tile more), so one block per CU covers
//     the cache with no CU left idle; fp32: blocks of `chunk` rows.  A block
//     has one wave (the wave stores its partial from registers) or 2, 4 or 8
//     (bf16: wave w takes every WAVES-th tile of the block from its w-th on;
//     the block combines the waves through LDS).
//   merge kernel, grid = (Hq * d / 32, B): one wave per 32 output values of a
//     query head combines that head's chunk partials by log-sum-exp in a
//     fixed order and writes them; the first wave advances kv_len[b].
// bf16 runs on the matrix cores (v_mfma_f32_16x16x32_bf16), one wave per
// 32-key block at a time:
//   S^T[32 keys x 16 heads] = K[32 x d] . Q^T[d x 16]   (heads padded to 16)
//   O^T[d x 16 heads]      += V^T[d x 32] . P^T[32 x 16]
// The K tile rows are permuted so that lane group q of the S^T result holds
// keys 8q..8q+7 of the block, exactly the k-slots the P^T operand needs: the
// softmax and the bf16 packing of P stay in the lane, and the per-head
// rescale of O^T is lane-local too (head = lane % 16 in both layouts).
// fp32 inputs keep fp32 arithmetic on the vector ALUs (16 lanes per key row,
// DPP row reductions).
// The appended row is read from k_new/v_new by the block that owns it (and
// stored into the caches there), so no block reads a row written in the same
// launch.  Lengths are read on the device only.  No atomics; every reduction
// has a fixed order, so results are bit-reproducible.

#include <mutex>

#include "../../include/timebill.h"
#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kVT = kVTile;           // rows per cache tile (32)
constexpr float kLazy = 8.f;          // slack of the bf16 kernel's exponent reference (log2 units)

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

// transpose read of 4 bf16: within each 16-lane group, lane i receives
// element i % 4 of the 8-byte chunks read by lanes 4j + i / 4, j = 0..3
__device__ __forceinline__ u32x2 lds_read_tr16(const void* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s*)p));
}

// Chunk c of V row R of a wave's buffer sits at c ^ vswz(R): a half-wave's
// transpose reads (rows 8 g + 0..3 and 8 (g + 1) + 0..3, 32 bytes each)
// then cover all banks.  Rows R and R + 4 (and R + 32 k) share the swizzle.
template <int D>
__device__ __forceinline__ int vswz(int R) {
  if constexpr (D == 128) return 2 * ((R & 3) | (((R >> 3) & 1) << 2));   // 16 chunks per row
  else return 2 * (((R >> 1) & 1) | (((R >> 3) & 1) << 1));               // 8 chunks per row
}

// --------------------------------------------------------------------------
// bf16: matrix-core partial kernel.
// --------------------------------------------------------------------------
// At least two waves per SIMD (<= 256 VGPRs), whatever the block size.
template <int D, int G, int WAVES, bool PAGED>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(2)))
void decode_mfma_kernel(DecodeArgs a) {
  static_assert(G >= 1 && G <= 16, "query heads per KV head must fit 16 columns");
  constexpr int KC = D / 32;            // k-chunks of the QK^T product
  constexpr int NC = D / 16;            // d-blocks of the PV product
  const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);    // wave-uniform
  const int q4 = lane >> 4, r16 = lane & 15;
  const int Hkv = a.Hkv, Hq = Hkv * G;

  // Each wave's V rows of its current tile (32 rows x CH chunks of 16 bytes,
  // chunk c of row R at c ^ vswz(R)); after the tile loop the same bytes hold
  // the wave's (o) for the block's combine: [G][D / 4 + 1] float4 per wave,
  // +1 spreading the heads over banks (3.7 KB of the 8 KB at G = 7, d = 128).
  constexpr int CH = D / 8;                       // 16-byte chunks per row
  static_assert(G * (D / 4 + 1) * 16 <= kVT * CH * 16, "combine buffer fits the V buffer");
  __shared__ u32x4 s_v[WAVES][kVT * CH];
  __shared__ float s_ml[WAVES][16][2];

  const size_t bg = static_cast<size_t>(b) * Hkv + g;
  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* vc = static_cast<const uint16_t*>(a.v_cache);
  const uint16_t* kn = static_cast<const uint16_t*>(a.k_new) + bg * D;
  const uint16_t* vn = static_cast<const uint16_t*>(a.v_new) + bg * D;
  const int cap = a.cap;
  // block c: tiles [c q + min(c, r), + q + (c < r)), q = n_tiles / n_chunks and
  // r = n_tiles % n_chunks from the host (no device division before the first
  // load)
  const int t_lo = c * a.tiles_q + min(c, a.tiles_r);
  const int t_hi = t_lo + a.tiles_q + (c < a.tiles_r ? 1 : 0);
  const int t_first = t_lo + wave;               // this wave: t_first, t_first + WAVES, ...
  // K tile row permutation: MFMA row r of tile t <-> key 8*(r/4) + 4*t + r%4.
  const int krow0 = 8 * (r16 >> 2) + (r16 & 3);

  // Everything below up to the length check is issued without waiting for
  // kv_len: the first block's K/V loads only need rows < cap, so the length
  // load and the data loads are in flight together.
  // V rows: the tile's 32 x CH chunks, chunk p = 64 u + lane (row p / CH)
  constexpr int VPL = kVT * CH / 64;              // V chunks per lane (8 at d = 128)
  u32x4 kr[2][KC], vr[VPL];
  auto load_block = [&](int base) {            // base: a multiple of 32 below cap
    const size_t off = cache_tile_off<PAGED>(a, b, g, base / kVT, D);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const uint16_t* src = kc + off + static_cast<size_t>(krow0 + 4 * t) * D;
#pragma unroll
      for (int k = 0; k < KC; ++k) kr[t][k] = ld16(src + 32 * k + 8 * q4);
    }
    const uint16_t* vtile = vc + off;
#pragma unroll
    for (int u = 0; u < VPL; ++u) vr[u] = ld16(vtile + static_cast<size_t>(64 * u + lane) * 8);
  };
  u32x4* sv = s_v[wave];
  int n0 = a.kv_len[b];
  if (t_first < t_hi) load_block(kVT * t_first);

  // Q^T operand: lane holds head r16, d = 32*kc + 8*q4 .. +8 (zero past G).
  bf16x8 qB[KC];
  {
    const uint16_t* qh = static_cast<const uint16_t*>(a.q) + (static_cast<size_t>(b) * Hq + g * G) * D;
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      // unconditional load of a valid head, zeroed past G
      u32x4 v = ld16(qh + min(r16, G - 1) * D + 32 * k + 8 * q4);
      if (r16 >= G) v = u32x4{0u, 0u, 0u, 0u};
      qB[k] = as_bf16x8(v);
    }
  }
  // the appended row, as the lanes use it: K slices and the V^T column values
  u32x4 knew[KC];
  uint16_t vnew[NC];
  if (a.append) {
#pragma unroll
    for (int k = 0; k < KC; ++k) knew[k] = ld16(kn + 32 * k + 8 * q4);
#pragma unroll
    for (int n = 0; n < NC; ++n) vnew[n] = vn[16 * n + r16];
  }

  n0 = n0 < 0 ? 0 : (n0 > cap ? cap : n0);
  const int app = (a.append && n0 < cap) ? 1 : 0;
  const int N = n0 + app;
  const int t_end = min(t_hi, (N + kVT - 1) / kVT);   // tiles holding a row below N

  // The block owning row n0 stores the appended row (K row, V^T column) from
  // the registers that already hold it: no reload, nothing waits on it.
  if (app && n0 / kVT >= t_lo && n0 / kVT < t_hi && wave == 0) {
    const size_t off = cache_tile_off<PAGED>(a, b, g, n0 / kVT, D);
    if (r16 == 0) {
      uint16_t* kd = static_cast<uint16_t*>(a.k_cache) + off + static_cast<size_t>(n0 % kVT) * D;
#pragma unroll
      for (int k = 0; k < KC; ++k) *reinterpret_cast<u32x4*>(kd + 32 * k + 8 * q4) = knew[k];
    }
    if (q4 == 0) {
      uint16_t* vd = static_cast<uint16_t*>(a.v_cache) + off + static_cast<size_t>(n0 % kVT) * D;
#pragma unroll
      for (int n = 0; n < NC; ++n) vd[16 * n + r16] = vnew[n];
    }
  }

  f32x4 accO[NC];
#pragma unroll
  for (int n = 0; n < NC; ++n) accO[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Exponent reference of head r16 (same in the 4 lane groups), kept on the
  // raw dot products (the scale is positive and enters each exponent through
  // one FMA): it moves only when a tile's maximum passes it by more than
  // kLazy scaled log2 units, so p <= 2^kLazy and most tiles need no rescale
  // of O^T.
  float m_run = -INFINITY;
  float m_thr = -INFINITY;   // m_run + kLazy / scale
  float m_sc = -INFINITY;    // m_run * scale, the partial's reference (log2 units)
  float l_part = 0.f;        // this lane's share of the running sum of head r16

  for (int t = t_first; t < t_end; t += WAVES) {
    const int base = kVT * t;
    u32x4 ck[2][KC], cv[NC];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int k = 0; k < KC; ++k) ck[t][k] = kr[t][k];
    // this tile's V rows into the wave's buffer (the wave's earlier reads of
    // it are done: LDS accesses of one wave complete in order)
#pragma unroll
    for (int u = 0; u < VPL; ++u) {
      const int cidx = 64 * u + lane, R = cidx / CH;
      sv[R * CH + ((cidx % CH) ^ vswz<D>(R))] = vr[u];
    }
    if (t + WAVES < t_end) load_block(kVT * (t + WAVES));   // prefetch the next tile

    // wave-uniform: does this tile hold the appended row, or run past the end?
    const bool has_new = app && n0 >= base && n0 < base + kVT;
    const bool tail = base + kVT > N;
    // ---- the appended row's K slices replace the (stale) cache rows
    if (has_new) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bool hit = base + krow0 + 4 * t == n0;
#pragma unroll
        for (int k = 0; k < KC; ++k) ck[t][k] = hit ? knew[k] : ck[t][k];
      }
    }
    // ---- S^T = K Q^T: lane holds keys base + 8*q4 + 4*t + i, head r16
    f32x4 S[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < KC; ++k)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ck[t][k]), qB[k], acc, 0, 0, 0);
      S[t] = acc;
    }
    float s[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) s[j] = S[j >> 2][j & 3];
    if (tail) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (base + 8 * q4 + j >= N) s[j] = -INFINITY;
    }
    float xm = s[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) xm = fmaxf(xm, s[j]);
    // rare (always on a head's first tile): some lane's keys pass the
    // threshold; the head's maximum over the 4 lane groups becomes the
    // reference and O^T and the sum are rescaled by 2^(old - new)
    if (__builtin_amdgcn_ballot_w64(xm > m_thr)) {
      float mt = fmaxf(xm, __shfl_xor(xm, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      // finite: every tile visited has at least one valid key (base < N)
      const float m_new = mt > m_thr ? mt : m_run;
      const float sc_new = m_new * a.scale_log2;
      const float corr = __builtin_amdgcn_exp2f(m_sc - sc_new);
      l_part *= corr;
#pragma unroll
      for (int n = 0; n < NC; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) accO[n][i] *= corr;
      m_run = m_new;
      m_sc = sc_new;
      m_thr = m_new + kLazy / a.scale_log2;
    }
    // hardware exp2 (results below 2^-126 of the reference flush to zero)
    float p[8];
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) { p[j] = __builtin_amdgcn_exp2f(fmaf(s[j], a.scale_log2, -m_sc)); psum += p[j]; }
    l_part += psum;
    bf16x8 pB;
#pragma unroll
    for (int j = 0; j < 8; ++j) pB[j] = static_cast<__bf16>(p[j]);

    // ---- V^T operand by transpose reads: lane (q4, r16) reads 8 bytes (d =
    // 16 n + 4 (r16 & 3) .. +3) of rows 8 q4 + r16 / 4 and + 4, and receives
    // d = 16 n + r16 of keys 8 q4 .. 8 q4 + 7; rows +4 share the swizzle
#pragma unroll
    for (int n = 0; n < NC; ++n) {
      const int R1 = 8 * q4 + (r16 >> 2);
      const int ch = 2 * n + ((r16 & 3) >> 1);
      const uint16_t* p1 = reinterpret_cast<const uint16_t*>(sv + R1 * CH + (ch ^ vswz<D>(R1))) + (r16 & 1) * 4;
      const u32x2 lo = lds_read_tr16(p1), hi = lds_read_tr16(p1 + 4 * D);
      cv[n] = u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
    // zero keys past the end, patch the appended row (branch-free word masks
    // over this lane's 8 keys)
    if (tail || has_new) {
      const int kq = base + 8 * q4;               // first key of this lane's 8
      const int cnt = min(max(N - kq, 0), 8);     // valid keys among the 8
      const int pos = n0 - kq;                    // slot of the appended row
      const bool inr = app && pos >= 0 && pos < cnt;
      const int pw = pos >> 1;
      const uint32_t sh = (pos & 1) * 16u;
#pragma unroll
      for (int n = 0; n < NC; ++n) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t keep = cnt >= 2 * w + 2 ? 0xffffffffu : (cnt == 2 * w + 1 ? 0xffffu : 0u);
          uint32_t x = cv[n][w] & keep;
          const uint32_t patched = (x & ~(0xffffu << sh)) | (static_cast<uint32_t>(vnew[n]) << sh);
          cv[n][w] = (inr && w == pw) ? patched : x;
        }
      }
    }
#pragma unroll
    for (int n = 0; n < NC; ++n)
      accO[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cv[n]), pB, accO[n], 0, 0, 0);
  }

  // ---- merge the lane groups' sums, then the waves, into this block's partial
  float l_tot = l_part + __shfl_xor(l_part, 16);
  l_tot += __shfl_xor(l_tot, 32);
  float* part = a.part + (bg * a.n_chunks + c) * G * (D + kPartPad);
  if constexpr (WAVES == 1) {
    // one wave: its (o, m, l) is the block's partial, stored from registers
    // (lane (q4, r16) holds d = 16 n + 4 q4 .. +3 of head r16)
    if (r16 < G) {
#pragma unroll
      for (int n = 0; n < NC; ++n)
        *reinterpret_cast<float4*>(part + r16 * (D + kPartPad) + 16 * n + 4 * q4) =
            make_float4(accO[n][0], accO[n][1], accO[n][2], accO[n][3]);
      if (q4 == 0) *reinterpret_cast<float2*>(part + r16 * (D + kPartPad) + D) = make_float2(m_sc, l_tot);
    }
    if (c == 0 && g == 0 && tid == 0) a.seq_len[b] = N;
    return;
  }
  // the wave's (o) goes into its own V buffer (its last reads of it are done);
  // the waves are combined with the hardware base-2 exponential (2489 ->
  // 2498 tokens/s on the 28-layer benchmark against the library exp2f,
  // though 3-7 us per token slower at alpha = 0)
  auto s_o = [&](int wv, int h, int e4) -> float4& {
    return reinterpret_cast<float4*>(s_v[wv])[h * (D / 4 + 1) + e4];
  };
  if (r16 < G) {
#pragma unroll
    for (int n = 0; n < NC; ++n)
      s_o(wave, r16, 4 * n + q4) = make_float4(accO[n][0], accO[n][1], accO[n][2], accO[n][3]);
  }
  if (q4 == 0) { s_ml[wave][r16][0] = m_sc; s_ml[wave][r16][1] = l_tot; }
  __syncthreads();

  for (int idx = tid; idx < G * (D / 4); idx += 64 * WAVES) {
    const int h = idx / (D / 4), e4 = idx % (D / 4);
    float M = -INFINITY;
#pragma unroll
    for (int wv = 0; wv < WAVES; ++wv) M = fmaxf(M, s_ml[wv][h][0]);
    float L = 0.f;
    float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
    if (M != -INFINITY) {
#pragma unroll
      for (int wv = 0; wv < WAVES; ++wv) {
        const float sc = __builtin_amdgcn_exp2f(s_ml[wv][h][0] - M);
        const float4 x = s_o(wv, h, e4);
        L += s_ml[wv][h][1] * sc;
        O.x += x.x * sc; O.y += x.y * sc; O.z += x.z * sc; O.w += x.w * sc;
      }
    }
    *reinterpret_cast<float4*>(part + h * (D + kPartPad) + 4 * e4) = O;
    if (e4 == 0) *reinterpret_cast<float2*>(part + h * (D + kPartPad) + D) = make_float2(M, L);
  }
  if (c == 0 && g == 0 && tid == 0) a.seq_len[b] = N;
}

// --------------------------------------------------------------------------
// fp32: vector-ALU partial kernel (keeps fp32 products; no narrowing).
// --------------------------------------------------------------------------
constexpr int kValuThreads = 256;
constexpr int kValuWaves = kValuThreads / 64;
constexpr int kUnroll = 4;                  // rows per 16-lane row group per iteration
constexpr int kRowsPerIter = 4 * kUnroll;   // rows per wave per iteration

template <int D, int G, bool PAGED>
__global__ __launch_bounds__(kValuThreads) void decode_valu_kernel(DecodeArgs a) {
  constexpr int DPL = D / 16;                     // elements per lane
  const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int grp = lane >> 4, sub = lane & 15;
  const int Hkv = a.Hkv, Hq = Hkv * G;

  __shared__ float s_o[kValuWaves][G][D];
  __shared__ float s_ml[kValuWaves][G][2];

  int n0 = a.kv_len[b];
  n0 = n0 < 0 ? 0 : (n0 > a.cap ? a.cap : n0);
  const int app = (a.append && n0 < a.cap) ? 1 : 0;
  const int N = n0 + app;
  const int lo = c * a.chunk;
  const int hi = min(lo + a.chunk, N);

  const size_t bg = static_cast<size_t>(b) * Hkv + g;
  const float* kc = static_cast<const float*>(a.k_cache);
  const float* vc = static_cast<const float*>(a.v_cache);
  const float* kn = static_cast<const float*>(a.k_new) + bg * D;
  const float* vn = static_cast<const float*>(a.v_new) + bg * D;

  if (app && n0 >= lo && n0 < hi && wave == 0) {
    const size_t off = cache_tile_off<PAGED>(a, b, g, n0 / kVT, D);
    float* kd = static_cast<float*>(a.k_cache) + off + static_cast<size_t>(n0 % kVT) * D;
    float* vd = static_cast<float*>(a.v_cache) + off + static_cast<size_t>(n0 % kVT) * D;
    constexpr int PER = (D + 63) / 64;
    float kx[PER], vx[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane + 64 * i;
      kx[i] = e < D ? kn[e] : 0.f;
      vx[i] = e < D ? vn[e] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane + 64 * i;
      if (e < D) { kd[e] = kx[i]; vd[e] = vx[i]; }
    }
  }

  float qf[G][DPL];
  {
    const float* qb = static_cast<const float*>(a.q) + (static_cast<size_t>(b) * Hq + g * G) * D;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < DPL; ++e) qf[h][e] = qb[h * D + sub * DPL + e] * a.scale_log2;
  }
  float m[G], l[G], o[G][DPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY; l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[h][e] = 0.f;
  }

  const int per_wave = a.chunk / kValuWaves;
  const int wlo = lo + wave * per_wave;
  const int whi = min(wlo + per_wave, hi);
  for (int base = wlo; base < whi; base += kRowsPerIter) {
    float kf[kUnroll][DPL], vf[kUnroll][DPL];
    bool valid[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int row = base + u * 4 + grp;
      valid[u] = row < whi;
      const bool is_new = app && row == n0;
      const int rr = valid[u] ? row : wlo;                      // a row inside the cache
      const size_t off = cache_tile_off<PAGED>(a, b, g, rr / kVT, D);
      const float* krow = kc + off + static_cast<size_t>(rr % kVT) * D;
      const float* vrow = vc + off + static_cast<size_t>(rr % kVT) * D;
#pragma unroll
      for (int e = 0; e < DPL; ++e) {
        const int d = sub * DPL + e;
        kf[u][e] = valid[u] ? (is_new ? kn[d] : krow[d]) : 0.f;
        vf[u][e] = valid[u] ? (is_new ? vn[d] : vrow[d]) : 0.f;
      }
    }
    float s[kUnroll][G];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc = fmaf(qf[h][e], kf[u][e], acc);
        acc = row16_sum(acc);
        s[u][h] = valid[u] ? acc : -INFINITY;
      }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mx = m[h];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) mx = fmaxf(mx, s[u][h]);
      if (mx == -INFINITY) continue;
      const float corr = exp2f(m[h] - mx);
      float p[kUnroll];
      float psum = 0.f;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) { p[u] = exp2f(s[u][h] - mx); psum += p[u]; }
      l[h] = l[h] * corr + psum;
#pragma unroll
      for (int e = 0; e < DPL; ++e) {
        float acc = o[h][e] * corr;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc = fmaf(p[u], vf[u][e], acc);
        o[h][e] = acc;
      }
      m[h] = mx;
    }
  }

#pragma unroll
  for (int h = 0; h < G; ++h) {
    float M = fmaxf(m[h], __shfl_xor(m[h], 16));
    M = fmaxf(M, __shfl_xor(M, 32));
    const float sc = (M == -INFINITY) ? 0.f : exp2f(m[h] - M);
    float lh = l[h] * sc;
    lh += __shfl_xor(lh, 16);
    lh += __shfl_xor(lh, 32);
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      float x = o[h][e] * sc;
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      o[h][e] = x;
    }
    m[h] = M;
    l[h] = lh;
  }
  if (grp == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int e = 0; e < DPL; ++e) s_o[wave][h][sub * DPL + e] = o[h][e];
      if (sub == 0) { s_ml[wave][h][0] = m[h]; s_ml[wave][h][1] = l[h]; }
    }
  }
  __syncthreads();

  float* part = a.part + (bg * a.n_chunks + c) * G * (D + kPartPad);
  for (int idx = tid; idx < G * D; idx += kValuThreads) {
    const int h = idx / D, e = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int wv = 0; wv < kValuWaves; ++wv) M = fmaxf(M, s_ml[wv][h][0]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int wv = 0; wv < kValuWaves; ++wv) {
        const float sc = exp2f(s_ml[wv][h][0] - M);
        L += s_ml[wv][h][1] * sc;
        O += s_o[wv][h][e] * sc;
      }
    }
    part[h * (D + kPartPad) + e] = O;
    if (e == 0) { part[h * (D + kPartPad) + D] = M; part[h * (D + kPartPad) + D + 1] = L; }
  }
  if (c == 0 && g == 0 && tid == 0) a.seq_len[b] = N;
}

// --------------------------------------------------------------------------
// Merge of the chunk partials of one query head, by one wave per E4 float4
// slices of its output (grid = (Hq * NQ, B), NQ = d / (4 E4) waves per head):
// lane = (chunk split sp of 64 / E4, slice e4); each lane issues one round of
// KPT partials' loads (the m, l of a partial are read by all NQ waves of its
// head), then the splits are combined by cross-lane swaps in a fixed order
// (lower split first).  One round covers (64 / E4) * KPT chunks with no LDS
// and no barrier; more chunks take more rounds.  Weights use the hardware
// base-2 exponential (arguments <= 0; results below 2^-126 flush to zero,
// as in the partial kernel): 13.37 against 13.52 us per decode call with the
// library exp2f on the 28-layer L = 32768 benchmark.  Every chunk writes a partial
// (empty chunks carry m = -inf, l = 0), so the merge runs over all of them and
// never waits for the length; the length is only needed for the kv_len store.
// --------------------------------------------------------------------------
template <typename T, int D, int G, int E4, int KPT>
__global__ __launch_bounds__(64) void decode_merge_split_kernel(DecodeArgs a) {
  constexpr int NQ = D / 4 / E4;             // waves per query head
  constexpr int SPL = 64 / E4;               // chunk splits per wave
  const int h = blockIdx.x / NQ, qd = blockIdx.x % NQ, b = blockIdx.y;
  const int Hkv = a.Hkv, Hq = Hkv * G;
  const int g = h / G, hh = h % G;
  const int lane = threadIdx.x, e4 = qd * E4 + lane % E4, sp = lane / E4;
  const int N = a.seq_len[b];
  const int n_used = a.n_chunks;
  const size_t bg = static_cast<size_t>(b) * Hkv + g;
  const float* base = a.part + (bg * a.n_chunks * G + hh) * (D + kPartPad);
  constexpr size_t CSTRIDE = static_cast<size_t>(G) * (D + kPartPad);

  float M = -INFINITY, L = 0.f;
  float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int c0 = sp; c0 < n_used; c0 += SPL * KPT) {
    float mm[KPT], ll[KPT];
    float4 oo[KPT];
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int cc = c0 + k * SPL;
      const float* pc = base + min(cc, n_used - 1) * CSTRIDE;
      const float2 ml = *reinterpret_cast<const float2*>(pc + D);
      oo[k] = *reinterpret_cast<const float4*>(pc + 4 * e4);
      mm[k] = cc < n_used ? ml.x : -INFINITY;
      ll[k] = cc < n_used ? ml.y : 0.f;
    }
    // keep every load above this point: they must all be in flight together
    __builtin_amdgcn_sched_barrier(0);
    float mx = M;
#pragma unroll
    for (int k = 0; k < KPT; ++k) mx = fmaxf(mx, mm[k]);
    if (mx == -INFINITY) continue;
    const float corr = __builtin_amdgcn_exp2f(M - mx);
    L *= corr; O.x *= corr; O.y *= corr; O.z *= corr; O.w *= corr;
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const float wgt = __builtin_amdgcn_exp2f(mm[k] - mx);
      L += wgt * ll[k];
      O.x += wgt * oo[k].x; O.y += wgt * oo[k].y; O.z += wgt * oo[k].z; O.w += wgt * oo[k].w;
    }
    M = mx;
  }
  // splits s and s ^ (off / E4) meet at lanes l and l ^ off; both lanes combine
  // (lower split, upper split) in that order, so they hold identical results
#pragma unroll
  for (int off = 32; off >= E4; off >>= 1) {
    const float Mo = __shfl_xor(M, off), Lo = __shfl_xor(L, off);
    const float4 Oo = make_float4(__shfl_xor(O.x, off), __shfl_xor(O.y, off),
                                  __shfl_xor(O.z, off), __shfl_xor(O.w, off));
    const bool upper = (lane & off) != 0;
    const float Ma = upper ? Mo : M, La = upper ? Lo : L;
    const float Mb = upper ? M : Mo, Lb = upper ? L : Lo;
    const float4 Oa = upper ? Oo : O, Ob = upper ? O : Oo;
    const float Mn = fmaxf(Ma, Mb);
    if (Mn != -INFINITY) {
      const float w1 = __builtin_amdgcn_exp2f(Ma - Mn), w2 = __builtin_amdgcn_exp2f(Mb - Mn);
      L = La * w1 + Lb * w2;
      O = make_float4(Oa.x * w1 + Ob.x * w2, Oa.y * w1 + Ob.y * w2,
                      Oa.z * w1 + Ob.z * w2, Oa.w * w1 + Ob.w * w2);
    }
    M = Mn;
  }
  if (sp == 0) {
    const float inv = L > 0.f ? 1.f / L : 0.f;
    T* out = static_cast<T*>(a.out) + (static_cast<size_t>(b) * Hq + h) * D + 4 * e4;
    if constexpr (sizeof(T) == 2) {
      typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
      *reinterpret_cast<bf16x4*>(out) =
          bf16x4{static_cast<__bf16>(O.x * inv), static_cast<__bf16>(O.y * inv),
                 static_cast<__bf16>(O.z * inv), static_cast<__bf16>(O.w * inv)};
    } else {
      *reinterpret_cast<float4*>(out) = make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv);
    }
  }
  if (blockIdx.x == 0 && lane == 0) a.kv_len[b] = N;
}

template <typename T, int D, int G, bool PAGED>
hipError_t launch_both(const DecodeArgs& a, hipStream_t st) {
  const dim3 grid(a.n_chunks, a.Hkv, a.B);
  if constexpr (sizeof(T) == 2) {
    switch (a.waves) {
      case 1: decode_mfma_kernel<D, G, 1, PAGED><<<grid, 64, 0, st>>>(a); break;
      case 2: decode_mfma_kernel<D, G, 2, PAGED><<<grid, 128, 0, st>>>(a); break;
      case 4: decode_mfma_kernel<D, G, 4, PAGED><<<grid, 256, 0, st>>>(a); break;
      case 8: decode_mfma_kernel<D, G, 8, PAGED><<<grid, 512, 0, st>>>(a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    decode_valu_kernel<D, G, PAGED><<<grid, kValuThreads, 0, st>>>(a);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // 8 float4 slices per wave (a quarter of a head's output at d = 128, half
  // at d = 64), one round of loads for up to 128 chunks.  Measured on the
  // 28-layer L = 32768 benchmark (tokens/s, two runs each, alternated):
  // 2423-2425 against 2368-2369 with one wave per whole head (<= 32 chunks)
  // and a 256-thread block per head with an LDS tree (33-64); 16 slices per
  // wave 2414, 4 slices 2359-2360.  Against those at other shapes (us per
  // decode call): 128-256 chunks (1-2 KV heads, d = 128, 8192-32768 rows)
  // 7.2-9.6 against 8.0-10.8; d = 64, 32-64 chunks 5.7-14.7 against 6.0-15.0.
  if (a.n_chunks <= 32)
    decode_merge_split_kernel<T, D, G, 8, 4><<<dim3(a.Hkv * G * (D / 32), a.B), 64, 0, st>>>(a);
  else if (a.n_chunks <= 64)
    decode_merge_split_kernel<T, D, G, 8, 8><<<dim3(a.Hkv * G * (D / 32), a.B), 64, 0, st>>>(a);
  else
    decode_merge_split_kernel<T, D, G, 8, 16><<<dim3(a.Hkv * G * (D / 32), a.B), 64, 0, st>>>(a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_g(const DecodeArgs& a, int G, hipStream_t st) {
  switch (G) {
#define TB_CASE(GG) case GG: return a.table ? launch_both<T, D, GG, true>(a, st) \
                                             : launch_both<T, D, GG, false>(a, st);
    TB_CASE(1) TB_CASE(2) TB_CASE(3) TB_CASE(4) TB_CASE(5) TB_CASE(6) TB_CASE(7) TB_CASE(8)
#undef TB_CASE
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int decode_chunk_unit(int waves, bool bf16) { return bf16 ? waves * kVT : kValuWaves * kRowsPerIter; }
int decode_max_chunks() { return 4096; }

// Workspace of tb_decode_attn_noalloc: one array per GPU, held from load to
// process exit.  Host code never passes the array's name to a kernel (on the
// host it is a stand-in, not a device address): decode_scratch() looks up the
// current device's address once and hands that out.
namespace {
static __device__ __align__(256) unsigned char scratch[TB_DECODE_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];
}  // namespace

hipError_t decode_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_addr[dev] = p;
  }
  *ptr = g_scratch_addr[dev];
  return hipSuccess;
}

hipError_t launch_decode(const DecodeArgs& a, int G, int d, bool bf16, hipStream_t st) {
  if (bf16) return d == 128 ? launch_g<bf16_t, 128>(a, G, st) : launch_g<bf16_t, 64>(a, G, st);
  return d == 128 ? launch_g<float, 128>(a, G, st) : launch_g<float, 64>(a, G, st);
}

}  // namespace tb

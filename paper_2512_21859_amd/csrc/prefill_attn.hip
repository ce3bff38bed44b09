// Causal grouped-query prefill attention (bf16, matrix cores), with the
// softmax statistics of the last w query rows (the observation window) as a
// by-product.
//
// This is the step before the eviction path: eviction follows the prefill
// phase (Sec. 4.2, Sec. 5.2), whose execution time the paper models as
// a N_x^2 + b N_x + c (Eq. prefill_phase_time_raw); the quadratic term is this
// attention.  out[b][h][i] = sum_{j <= i} softmax_j(q[b][h][i] . k[b][g][j] /
// sqrt(d)) v[b][g][j], g = h / (Hq / Hkv).
//
// Block = the query rows of one query head (4 or 8 waves of 32 rows; 16 per
// wave for short prompts: the launch below), blocks issued heaviest first
// (latest rows) and grouped by KV head on the XCDs, so the query heads that
// read the same K/V rows do so through one L2 (measured: 962-969 -> 1144-1145
// TFLOP/s at N = 32768, 530-543 -> 867-877 at 4096).  K and V stream through
// LDS 64 or 128 keys at a time,
// double-buffered: each stage goes global -> LDS by direct loads (no
// registers), issued one stage ahead, one barrier per stage.  Both stay
// row-major in LDS (16-byte chunks XOR-swizzled by row against bank
// conflicts); the V^T operand ("8 consecutive keys of one d") comes from
// transpose reads of row-major V.  Per 32-key step a wave computes
//   S^T[32 keys x 16 queries] = K Q^T   and   O^T[d x 16 queries] += V^T P^T
// for its two 16-query column tiles with v_mfma_f32_16x16x32_bf16.  As in the
// decode kernel, the K rows of an MFMA tile are permuted (row r of tile t <->
// key 8(r/4) + 4t + r%4) so that lane group q of the S^T result holds keys
// 8q .. 8q+7 of the step, exactly the P^T operand: the online softmax, the
// bf16 packing of P and the rescale of O^T stay in the lane.  Softmax runs in
// the base-2 domain with fp32 statistics (an exponent reference on the raw
// dot products, the scale folded into each exponent's FMA); P is rounded to
// bf16 for the PV product.  The reference moves only when a row's maximum
// exceeds it by more than 2^8, so O^T is rescaled (and a correction
// exponential computed) only in the few steps where that happens.  Each step runs its two column tiles phase by phase (both QK
// products, one mask branch, both softmaxes, one statistics branch, one
// rescale test, both PV products), so one tile's products overlap the
// other's exponentials: +4% at N = 16384-32768 over one tile at a time,
// bit-identical output.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr float kLazy = 8.f;                  // reference slack, scaled log2 units

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// max over the four 16-lane groups (lanes l, l^16, l^32, l^48) with the
// row-swap permutes: a self-swap leaves each lane's value in one result and
// its partner's in the other
// (NaN-propagating maximum: one three-input instruction, no quieting of
// the matrix-core results first)
__device__ __forceinline__ float fmax2(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float group_max(float x) {
  const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmax2(__uint_as_float(h[0]), __uint_as_float(h[1]));
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmax2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// K rows sit in LDS unpadded, their 16-byte chunks permuted by row: chunk c
// of row R is stored at c ^ kswz(R).  A K-operand read has 16 lanes take one
// chunk index from the rows {0-3, 8-11, 16-19, 24-27} (+4 t) of the permuted
// tile; the swizzle sends those 16 rows to 16 different bank groups (with a
// padded stride rows R and R+16 shared banks: a 2-way conflict on every read).
template <int D>
__device__ __forceinline__ int kswz(int R) {
  if constexpr (D == 128) return (R & 3) | ((R >> 1) & 12);          // 16 chunks per row
  else return ((R >> 1) & 1) | ((R >> 2) & 6);                       // 8 chunks; rows pair up in 256 B
}

// V rows sit row-major in LDS, chunk c of row R at c ^ vswz(R).  A transpose
// read has 16 lanes take 32 bytes (chunks 2n, 2n + 1) of 4 consecutive rows;
// a half-wave covers rows 8g + 0..3 and 8(g + 1) + 0..3, and the swizzle
// spreads those 256 bytes over all banks.
template <int D>
__device__ __forceinline__ int vswz(int R) {
  if constexpr (D == 128) return 2 * ((R & 3) | (((R >> 3) & 1) << 2));       // 16 chunks per row
  else return 2 * (((R >> 1) & 1) | (((R >> 3) & 1) << 1));                  // 8 chunks per row
}

typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

// 16 bytes global -> LDS without a register: a wave's 64 lanes fill 1 KB
// starting at the wave-uniform LDS address `lds`, lane l at lds + 16 l
__device__ __forceinline__ void lds_load16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// transpose read of 4 bf16: within each 16-lane group, lane i receives
// element i % 4 of the 8-byte chunks read by lanes 4j + i / 4, j = 0..3
__device__ __forceinline__ u32x2 lds_read_tr16(const void* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s*)p));
}

// broadcast lane r16's value (lane group 0) to the lanes r16 + 16 q4
__device__ __forceinline__ float from_group0(float x, int lane) {
  return __shfl(x, lane & 15);
}

// WAVES waves of CQ column tiles each per block; K and V stages of STAGE keys
template <int D, int CQ, int WAVES, int STAGE>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(CQ == 2 ? 2 : 1)))
void prefill_attn_kernel(PrefillArgs a) {
  constexpr int kWaves = WAVES;
  constexpr int kStage = STAGE;               // keys per LDS stage
  constexpr int kRowsPerWave = 16 * CQ;       // CQ 16-query column tiles per wave
  constexpr int kBlockRows = kWaves * kRowsPerWave;
  constexpr int KC = D / 32;                  // k-chunks of the QK^T product
  constexpr int NC = D / 16;                  // d-blocks of the PV product
  // Block order (one-dimensional grid): workgroup i runs on XCD i % 8, and
  // XCD x takes the units x, x + 8, x + 16, ... of (query tile rank, batch,
  // KV head), heaviest tiles first; the G query heads of a unit sit in G
  // consecutive slots of that XCD.  So the blocks that stream the same K/V
  // rows share one XCD's L2, and with Hkv dividing 8 each XCD only ever
  // reads one KV head.
  const int G = a.Hq / a.Hkv;
  const int wg = static_cast<int>(blockIdx.x);
  const int slot = wg >> 3, unit = (slot / G) * 8 + (wg & 7);
  const int g = unit % a.Hkv, rb = unit / a.Hkv, b = rb % a.B, rank = rb / a.B;
  int lmax = 0;
  for (int bb = 0; bb < a.B; ++bb) lmax = max(lmax, a.L[bb]);
  if (rank >= (lmax + kBlockRows - 1) / kBlockRows) return;  // padding of the last XCD round
  const int h = g * G + slot % G;
  const int L = a.L[b];
  const int n_qt = (L + kBlockRows - 1) / kBlockRows;
  const int qt = n_qt - 1 - rank;                               // heaviest tiles first
  if (qt < 0) return;                                           // shorter sequence of the batch
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q4 = lane >> 4, r16 = lane & 15;

  // Stage buffers, double-buffered: [buffer][K, V][row * CH + chunk] in
  // 16-byte chunks; K row R keeps chunk c at c ^ kswz(R), V row R at c ^ vswz(R).
  constexpr int CH = D / 8;                   // 16-byte chunks per row
  constexpr int SCH = kStage * CH;            // chunks per stage and matrix
  constexpr int PER_THREAD = SCH / (64 * kWaves);
  // two distinct arrays (not one indexed by a runtime buffer number), so the
  // compiler can tell the loads in flight into one from the reads of the other
  __shared__ u32x4 s_kv0[2][SCH];
  __shared__ u32x4 s_kv1[2][SCH];

  const uint16_t* qh = static_cast<const uint16_t*>(a.q) + (static_cast<size_t>(b) * a.Hq + h) * a.Lmax * D;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const uint16_t* kg = static_cast<const uint16_t*>(a.k) + bg * a.Lmax * D;
  const uint16_t* vg = static_cast<const uint16_t*>(a.v) + bg * a.Lmax * D;

  const int row0 = qt * kBlockRows + wave * kRowsPerWave;     // this wave's first query
  // Q^T operands: column tile cq, lane holds query row0 + 16 cq + r16, d = 32 kc + 8 q4 .. +8
  u32x4 qB[CQ][KC];
#pragma unroll
  for (int cq = 0; cq < CQ; ++cq) {
    const int qi = min(row0 + 16 * cq + r16, L - 1);            // rows past L: any valid row
    const uint16_t* src = qh + static_cast<size_t>(qi) * D;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) qB[cq][kc] = *reinterpret_cast<const u32x4*>(src + 32 * kc + 8 * q4);
  }

  f32x4 accO[CQ][NC];
  // row sums of P on the matrix cores: a V^T tile whose row 0 is all ones, so
  // the sum (of the same bf16-rounded P the numerator uses) lands in row 0 of
  // accL: item 0 of the lanes of group 0
  f32x4 accL[CQ];
  // The exponent reference of each row, on the raw dot products (the scale
  // is positive): it moves only when a step's maximum exceeds it by more
  // than kLazy in scaled log2 units, so P <= 2^kLazy (bf16 and the fp32
  // accumulators keep the same relative precision at that size) and most
  // steps need no correction exponential and no rescale of O^T.
  float m_ref[CQ];
  float m_thr[CQ];                            // m_ref + kLazy / scale: a step past it moves m_ref
  float m_sc[CQ];                             // m_ref * scale (the exponents' offset)
  // the window rows' statistics are reported exact to fp32 (unrounded P,
  // true maximum), so the waves holding window rows also keep a vector-ALU
  // sum and the true running maximum
  float l_part[CQ], m_max[CQ];
#pragma unroll
  for (int cq = 0; cq < CQ; ++cq) {
#pragma unroll
    for (int n = 0; n < NC; ++n) accO[cq][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    accL[cq] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_ref[cq] = -INFINITY;
    m_thr[cq] = -INFINITY;
    m_sc[cq] = -INFINITY;
    l_part[cq] = 0.f;
    m_max[cq] = -INFINITY;
  }
  const uint32_t one2 = r16 == 0 ? 0x3F803F80u : 0u;          // two bf16 ones
  const u32x4 onesA = {one2, one2, one2, one2};
  const int krow0 = 8 * (r16 >> 2) + (r16 & 3);                // permuted K row of MFMA row r16

  const int key_end = min(L, (qt + 1) * kBlockRows);            // causal limit of the block
  const int wave_key_end = min(L, row0 + kRowsPerWave);         // causal limit of this wave
  const bool stats_wave = a.window_stats != nullptr && row0 + kRowsPerWave > L - a.w;

  // One stage of STAGE keys goes global -> LDS by direct loads, one stage
  // ahead: load u of thread tid fills chunk position p = 64 WAVES u + tid of K and of V
  // (a wave's 64 lanes write 1 KB contiguous), taking from global memory the
  // chunk the swizzled layout keeps there.  Keys past L read row L - 1 (any
  // valid row: they are masked).
  auto load_stage = [&](int s0, u32x4 (&dst)[2][SCH]) {
#pragma unroll
    for (int u = 0; u < PER_THREAD; ++u) {
      const int p = u * 64 * kWaves + tid;
      const int R = p / CH, cp = p % CH;
      const size_t row = static_cast<size_t>(min(s0 + R, L - 1)) * D;
      const int wbase = u * 64 * kWaves + 64 * wave;          // wave-uniform LDS chunk base
      lds_load16(kg + row + 8 * (cp ^ kswz<D>(R)), &dst[0][wbase]);
      lds_load16(vg + row + 8 * (cp ^ vswz<D>(R)), &dst[1][wbase]);
    }
  };

  auto compute_stage = [&](int s0, const u32x4 (&src)[2][SCH]) {
    const u32x4* sk = src[0];
    const u32x4* sv = src[1];
#pragma unroll
    for (int sub = 0; sub < kStage / 32; ++sub) {
      const int base = s0 + 32 * sub;                           // first key of the 32-key step
      if (base >= wave_key_end) continue;                       // wave-uniform: all keys masked
      // K operands of the step (shared by both column tiles)
      u32x4 kA[2][KC];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
          const int R = 32 * sub + krow0 + 4 * t;
          kA[t][kc] = sk[R * CH + ((4 * kc + q4) ^ kswz<D>(R))];
        }
      // V^T operands by transpose reads: lane (q4, r16) fetches d = 16 n +
      // 4 (r16 & 3) .. +3 of keys 8 q4 + r16 / 4 (and + 4) and receives
      // d = 16 n + r16 of keys 8 q4 .. 8 q4 + 7
      u32x4 vA[NC];
#pragma unroll
      for (int n = 0; n < NC; ++n) {
        const int R1 = 32 * sub + 8 * q4 + (r16 >> 2), R2 = R1 + 4;
        const int cv = 2 * n + ((r16 & 3) >> 1);                // chunk of d = 16 n + 4 (r16 & 3)
        const int half = (r16 & 1) * 4;                         // bf16 offset of that half chunk
        const uint16_t* p1 = reinterpret_cast<const uint16_t*>(sv + R1 * CH + (cv ^ vswz<D>(R1))) + half;
        const uint16_t* p2 = reinterpret_cast<const uint16_t*>(sv + R2 * CH + (cv ^ vswz<D>(R2))) + half;
        const u32x2 lo = lds_read_tr16(p1), hi = lds_read_tr16(p2);
        vA[n] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      }
      const bool need_mask = base + 32 > row0;                  // step reaches this wave's diagonal
      // The step runs in phases over the column tiles: every tile's QK
      // products, the mask, every tile's softmax, the window statistics, one
      // rescale test, every tile's PV products.  Kept apart (each wave-uniform
      // branch taken once per step, not once per tile), the products of one
      // tile can issue beside the other tile's exponentials.
      f32x4 S[CQ][2];
#pragma unroll
      for (int cq = 0; cq < CQ; ++cq)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kc = 0; kc < KC; ++kc)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kA[t][kc]), as_bf16x8(qB[cq][kc]), acc, 0, 0, 0);
          S[cq][t] = acc;
        }
      // lane holds keys base + 8 q4 + j (j = 4t + i) of query row0 + 16 cq + r16
      if (need_mask) {
#pragma unroll
        for (int cq = 0; cq < CQ; ++cq) {
          const int qi = row0 + 16 * cq + r16;
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (base + 8 * q4 + j > qi) S[cq][j >> 2][j & 3] = -INFINITY;
        }
      }
      // Each lane first compares the maximum of its own 8 keys with the
      // reference; only when some lane exceeds it by more than kLazy (always
      // on a row's first step: m_ref = -inf there, and every wave's first
      // step holds key 0, which no query masks) does the wave take the row
      // maxima over the 4 lane groups and move those rows' references.
      float xm[CQ];
      bool grow = false;
#pragma unroll
      for (int cq = 0; cq < CQ; ++cq) {
        const f32x4 s0 = S[cq][0], s1 = S[cq][1];
        xm[cq] = fmax2(fmax2(fmax2(s0[0], s0[1]), fmax2(s0[2], s0[3])),
                       fmax2(fmax2(s1[0], s1[1]), fmax2(s1[2], s1[3])));
        grow = grow || xm[cq] > m_thr[cq];
      }
      if (__builtin_amdgcn_ballot_w64(grow)) {                 // rare
#pragma unroll
        for (int cq = 0; cq < CQ; ++cq) {
          const float mt = group_max(xm[cq]);
          const float m_new = (mt - m_ref[cq]) * a.scale_log2 > kLazy ? mt : m_ref[cq];
          // 2^((old - new) scale): exactly 1 where the reference stays, 0 on
          // the first step
          const float corr = __builtin_amdgcn_exp2f((m_ref[cq] - m_new) * a.scale_log2);
#pragma unroll
          for (int n = 0; n < NC; ++n)
#pragma unroll
            for (int i = 0; i < 4; ++i) accO[cq][n][i] *= corr;
          accL[cq][0] *= corr;
          l_part[cq] *= corr;
          m_ref[cq] = m_new;
          m_sc[cq] = m_new * a.scale_log2;
          m_thr[cq] = m_new + kLazy / a.scale_log2;
        }
      }
      float p[CQ][8];
#pragma unroll
      for (int cq = 0; cq < CQ; ++cq) {
        const float mc = m_sc[cq];
        // hardware exp2: results below 2^-126 flush to zero, far below a
        // softmax term that can matter next to the reference's term
#pragma unroll
        for (int j = 0; j < 8; ++j) p[cq][j] = __builtin_amdgcn_exp2f(fmaf(S[cq][j >> 2][j & 3], a.scale_log2, -mc));
      }
      if (stats_wave) {                                       // wave-uniform
#pragma unroll
        for (int cq = 0; cq < CQ; ++cq) {
          float psum = 0.f;
#pragma unroll
          for (int j = 0; j < 8; ++j) psum += p[cq][j];
          l_part[cq] += psum;
          m_max[cq] = fmax2(m_max[cq], group_max(xm[cq]));
        }
      }
      bf16x8 pB[CQ];
#pragma unroll
      for (int cq = 0; cq < CQ; ++cq)
#pragma unroll
        for (int j = 0; j < 8; ++j) pB[cq][j] = static_cast<__bf16>(p[cq][j]);
#pragma unroll
      for (int cq = 0; cq < CQ; ++cq) {
        accL[cq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(onesA), pB[cq], accL[cq], 0, 0, 0);
#pragma unroll
        for (int n = 0; n < NC; ++n)
          accO[cq][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vA[n]), pB[cq], accO[cq][n], 0, 0, 0);
      }
    }
  };

  // stage pipeline, unrolled by two over the two buffers: wait for this
  // stage's loads (and for every wave to be done with the other buffer),
  // start the next stage's loads into the other buffer, compute.  (The
  // compiler cannot tell the transpose reads from the loads landing in the
  // other buffer and makes them wait for those loads, so the overlap is the
  // first step's K reads and QK products; still 9% faster than staging
  // through registers, and bit-identical to it.)
  load_stage(0, s_kv0);
  for (int s0 = 0; s0 < key_end; s0 += 2 * kStage) {
    __builtin_amdgcn_s_waitcnt(0x0F70);                         // vmcnt(0)
    __syncthreads();
    if (s0 + kStage < key_end) load_stage(s0 + kStage, s_kv1);
    compute_stage(s0, s_kv0);
    if (s0 + kStage >= key_end) break;
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
    if (s0 + 2 * kStage < key_end) load_stage(s0 + 2 * kStage, s_kv0);
    compute_stage(s0 + kStage, s_kv1);
  }

  // finalize: lane holds d = 16 n + 4 q4 .. +3 of query row0 + 16 cq + r16
  uint16_t* outh = static_cast<uint16_t*>(a.out) + (static_cast<size_t>(b) * a.Hq + h) * a.Lmax * D;
#pragma unroll
  for (int cq = 0; cq < CQ; ++cq) {
    const float l_tot = from_group0(accL[cq][0], lane);      // sum of the P the numerator used
    float z = 0.f;                                            // unrounded sum (window waves)
    if (stats_wave) {
      z = l_part[cq] + __shfl_xor(l_part[cq], 16);
      z += __shfl_xor(z, 32);
      z *= __builtin_amdgcn_exp2f((m_ref[cq] - m_max[cq]) * a.scale_log2);   // to the true maximum
    }
    const int qi = row0 + 16 * cq + r16;
    if (qi < L) {
      const float inv = 1.f / l_tot;
      typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
      uint16_t* dst = outh + static_cast<size_t>(qi) * D;
#pragma unroll
      for (int n = 0; n < NC; ++n)
        *reinterpret_cast<bf16x4*>(dst + 16 * n + 4 * q4) =
            bf16x4{static_cast<__bf16>(accO[cq][n][0] * inv), static_cast<__bf16>(accO[cq][n][1] * inv),
                   static_cast<__bf16>(accO[cq][n][2] * inv), static_cast<__bf16>(accO[cq][n][3] * inv)};
      // window rows: row max (natural-log units) and normaliser of the softmax
      if (stats_wave && q4 == 0 && qi >= L - a.w) {
        float* ws = a.window_stats + ((static_cast<size_t>(b) * a.Hq + h) * a.w + (qi - (L - a.w))) * 2;
        ws[0] = m_max[cq] * a.scale_log2 * 0.69314718055994531f;   // raw max -> natural units
        ws[1] = z;
      }
    }
  }
}

}  // namespace

template <int CQ, int WAVES, int STAGE>
hipError_t launch_prefill_cq(const PrefillArgs& a, int d, int lmax, hipStream_t st) {
  constexpr int rows = WAVES * 16 * CQ;
  // units of (query tile rank, batch, KV head), padded to whole rounds of
  // the 8 XCDs, times the G query heads of each
  const int units = ((lmax + rows - 1) / rows) * a.B * a.Hkv;
  const dim3 grid(((units + 7) / 8) * 8 * (a.Hq / a.Hkv));
  if (d == 128) prefill_attn_kernel<128, CQ, WAVES, STAGE><<<grid, 64 * WAVES, 0, st>>>(a);
  else          prefill_attn_kernel<64, CQ, WAVES, STAGE><<<grid, 64 * WAVES, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs& a, int d, hipStream_t st) {
  // Block shapes by prompt length (28 q / 4 kv heads, d = 128, measured on
  // one box, alternated; TFLOP/s):
  // * two column tiles per wave (225 VGPRs, two waves per SIMD); three or
  //   four tiles cut the LDS operand reads per product but need one wave
  //   per SIMD, and measured slower (530 and 462 against 900 at 32768);
  // * N >= 8192: 8 waves (256 rows) and 128-key stages, 128 KB of LDS, one
  //   block per CU: the stage's global -> LDS traffic and barriers are
  //   shared by twice the rows: 1147 -> 1191-1194 at 32768, 1137 -> 1166 at
  //   16384, 1078 -> 1099 at 8192, but 1020 -> 971-983 at 6144;
  // * below that 4 waves (128 rows) and 64-key stages, two blocks per CU;
  // * up to 1024 tokens one column tile per wave (64-row blocks): the
  //   128-row launch has 224 blocks for 256 CUs at N = 1024 and the heaviest
  //   query tile's serial steps set the time; twice the blocks with half
  //   the work per step: 49 -> 58 at N = 256, 124 -> 144 at 512, 284 -> 301
  //   at 1024 (at 2048 it lost 7%, at 4096 27%).
  int lmax = 0;
  for (int b = 0; b < a.B; ++b) lmax = max(lmax, a.L[b]);
  if (lmax <= 1024) return launch_prefill_cq<1, 4, 64>(a, d, lmax, st);
  if (lmax < 8192) return launch_prefill_cq<2, 4, 64>(a, d, lmax, st);
  return launch_prefill_cq<2, 8, 128>(a, d, lmax, st);
}

}  // namespace tb

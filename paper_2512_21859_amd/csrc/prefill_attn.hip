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
// Block = 128 query rows of one query head (4 waves x 32 rows), blocks issued
// heaviest first (latest rows).  K and V stream through LDS 64 keys at a time,
// the next stage's global loads in flight during the current stage's products;
// V is written into LDS transposed so that "8 consecutive keys of one V
// column" is one 16-byte read.  Per 32-key step a wave computes
//   S^T[32 keys x 16 queries] = K Q^T   and   O^T[d x 16 queries] += V^T P^T
// for its two 16-query column tiles with v_mfma_f32_16x16x32_bf16.  As in the
// decode kernel, the K rows of an MFMA tile are permuted (row r of tile t <->
// key 8(r/4) + 4t + r%4) so that lane group q of the S^T result holds keys
// 8q .. 8q+7 of the step, exactly the P^T operand: the online softmax, the
// bf16 packing of P and the rescale of O^T stay in the lane.  Softmax runs in
// the base-2 domain with fp32 statistics (the running max on the raw dot
// products, the scale folded into each exponent's FMA); P is rounded to bf16
// for the PV product.  O^T is rescaled only in steps where some row's max
// moved.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kWaves = 4;
constexpr int kStage = 64;                    // keys per LDS stage
constexpr int kVPad = 8;                      // bf16 padding of a V^T row in LDS

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

// broadcast lane r16's value (lane group 0) to the lanes r16 + 16 q4
__device__ __forceinline__ float from_group0(float x, int lane) {
  return __shfl(x, lane & 15);
}

template <int D, int CQ>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(CQ == 2 ? 2 : 1)))
void prefill_attn_kernel(PrefillArgs a) {
  constexpr int kRowsPerWave = 16 * CQ;       // CQ 16-query column tiles per wave
  constexpr int kBlockRows = kWaves * kRowsPerWave;
  constexpr int KC = D / 32;                  // k-chunks of the QK^T product
  constexpr int NC = D / 16;                  // d-blocks of the PV product
  const int h = blockIdx.y, b = blockIdx.z;
  const int L = a.L[b];
  const int n_qt = (L + kBlockRows - 1) / kBlockRows;
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.x);     // heaviest tiles first
  if (qt < 0) return;
  const int G = a.Hq / a.Hkv, g = h / G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q4 = lane >> 4, r16 = lane & 15;

  __shared__ uint16_t s_k[kStage][D];
  __shared__ uint16_t s_vt[D][kStage + kVPad];

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
  float m_run[CQ];                            // running max of the raw dot products
  // the window rows' normaliser is reported exact to fp32 (unrounded P), so
  // the waves holding window rows also keep a vector-ALU sum
  float l_part[CQ];
#pragma unroll
  for (int cq = 0; cq < CQ; ++cq) {
#pragma unroll
    for (int n = 0; n < NC; ++n) accO[cq][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    accL[cq] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[cq] = -INFINITY;
    l_part[cq] = 0.f;
  }
  const uint32_t one2 = r16 == 0 ? 0x3F803F80u : 0u;          // two bf16 ones
  const u32x4 onesA = {one2, one2, one2, one2};
  const int krow0 = 8 * (r16 >> 2) + (r16 & 3);                // permuted K row of MFMA row r16

  const int key_end = min(L, (qt + 1) * kBlockRows);            // causal limit of the block
  const int wave_key_end = min(L, row0 + kRowsPerWave);         // causal limit of this wave
  const bool stats_wave = a.window_stats != nullptr && row0 + kRowsPerWave > L - a.w;

  // Staging of 64 keys, fetched into registers one stage ahead.  K: thread =
  // (key tid/4, quarter tid%4 of d), rows copied as they are.  V: thread
  // t < (64/4)(D/8) takes 4-key group t%16 and d-octet t/16 (the 16 groups
  // of a d-octet fill 128 contiguous bytes of a V^T row, so a wave's writes
  // do not collide in LDS banks), reads 4 keys x 8 d and transposes them in
  // registers (byte permutes) into 8 rows of V^T x 4 keys, stored as 8-byte
  // writes.
  constexpr int KQ = D / 4;                   // K elements per thread
  constexpr int VD8 = D / 8;                  // d-octets
  constexpr int VTASKS = (kStage / 4) * VD8;  // (4-key group, d-octet) tasks
  const int kr = tid >> 2, kpart = tid & 3;
  u32x4 kreg[KQ / 8], vreg[4];
  auto fetch = [&](int s0) {
    const int key = min(s0 + kr, L - 1);
    const uint16_t* ks = kg + static_cast<size_t>(key) * D + kpart * KQ;
#pragma unroll
    for (int e = 0; e < KQ / 8; ++e) kreg[e] = *reinterpret_cast<const u32x4*>(ks + 8 * e);
    if (tid < VTASKS) {
      const int k4 = tid % (kStage / 4), d8 = tid / (kStage / 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kv = min(s0 + 4 * k4 + j, L - 1);
        vreg[j] = *reinterpret_cast<const u32x4*>(vg + static_cast<size_t>(kv) * D + 8 * d8);
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int e = 0; e < KQ / 8; ++e)
      *reinterpret_cast<u32x4*>(&s_k[kr][8 * ((kpart * (KQ / 8) + e) ^ kswz<D>(kr))]) = kreg[e];
    if (tid < VTASKS) {
      const int k4 = tid % (kStage / 4), d8 = tid / (kStage / 4);
      // vreg[j] holds d = 8 d8 .. +7 of key 4 k4 + j (two bf16 per dword);
      // V^T row 8 d8 + 2c + h takes half h of dword c from keys j = 0..3
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        // byte selectors: low halves of (x, y) -> 0x05040100, high halves -> 0x07060302
        const uint32_t lo01 = __builtin_amdgcn_perm(vreg[1][c], vreg[0][c], 0x05040100u);
        const uint32_t lo23 = __builtin_amdgcn_perm(vreg[3][c], vreg[2][c], 0x05040100u);
        const uint32_t hi01 = __builtin_amdgcn_perm(vreg[1][c], vreg[0][c], 0x07060302u);
        const uint32_t hi23 = __builtin_amdgcn_perm(vreg[3][c], vreg[2][c], 0x07060302u);
        typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;
        *reinterpret_cast<u32x2*>(&s_vt[8 * d8 + 2 * c][4 * k4]) = u32x2{lo01, lo23};
        *reinterpret_cast<u32x2*>(&s_vt[8 * d8 + 2 * c + 1][4 * k4]) = u32x2{hi01, hi23};
      }
    }
  };

  fetch(0);
  for (int s0 = 0; s0 < key_end; s0 += kStage) {
    __syncthreads();                          // the previous stage's reads are done
    stage();
    __syncthreads();
    if (s0 + kStage < key_end) fetch(s0 + kStage);   // in flight during the products
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
          kA[t][kc] = *reinterpret_cast<const u32x4*>(&s_k[R][8 * ((4 * kc + q4) ^ kswz<D>(R))]);
        }
      // V^T operands: d = 16 n + r16, keys 8 q4 .. +8 of the step
      u32x4 vA[NC];
#pragma unroll
      for (int n = 0; n < NC; ++n)
        vA[n] = *reinterpret_cast<const u32x4*>(&s_vt[16 * n + r16][32 * sub + 8 * q4]);
      const bool need_mask = base + 32 > row0;                  // step reaches this wave's diagonal
#pragma unroll
      for (int cq = 0; cq < CQ; ++cq) {
        f32x4 S[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kc = 0; kc < KC; ++kc)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kA[t][kc]), as_bf16x8(qB[cq][kc]), acc, 0, 0, 0);
          S[t] = acc;
        }
        // lane holds keys base + 8 q4 + j (j = 4t + i) of query row0 + 16 cq + r16;
        // the running max is kept on the raw dot products (the scale is
        // positive) and the scale enters each exponent through one FMA
        const int qi = row0 + 16 * cq + r16;
        float s[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] = S[j >> 2][j & 3];
        if (need_mask) {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (base + 8 * q4 + j > qi) s[j] = -INFINITY;
        }
        float mt = fmax2(fmax2(fmax2(s[0], s[1]), fmax2(s[2], s[3])),
                         fmax2(fmax2(s[4], s[5]), fmax2(s[6], s[7])));
        mt = group_max(mt);
        // finite: every wave's first step holds key 0, which no query masks
        const float m_new = fmax2(m_run[cq], mt);
        const float mc = m_new * a.scale_log2;
        // 1 when the max did not move; 0 on the first step (m_run = -inf)
        const float corr = __builtin_amdgcn_exp2f((m_run[cq] - m_new) * a.scale_log2);
        m_run[cq] = m_new;
        bf16x8 pB;
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          // hardware exp2: results below 2^-126 flush to zero, far below a
          // softmax term that can matter next to the row max's term of 1
          p[j] = __builtin_amdgcn_exp2f(fmaf(s[j], a.scale_log2, -mc));
          pB[j] = static_cast<__bf16>(p[j]);
        }
        if (stats_wave) {                                     // wave-uniform
          float psum = 0.f;
#pragma unroll
          for (int j = 0; j < 8; ++j) psum += p[j];
          l_part[cq] = l_part[cq] * corr + psum;
        }
        // rescaling by exactly 1 changes nothing: skip it unless some lane's max moved
        if (__builtin_amdgcn_ballot_w64(corr != 1.f)) {
#pragma unroll
          for (int n = 0; n < NC; ++n)
#pragma unroll
            for (int i = 0; i < 4; ++i) accO[cq][n][i] *= corr;
          accL[cq][0] *= corr;
        }
        accL[cq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(onesA), pB, accL[cq], 0, 0, 0);
#pragma unroll
        for (int n = 0; n < NC; ++n)
          accO[cq][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vA[n]), pB, accO[cq][n], 0, 0, 0);
      }
    }
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
        ws[0] = m_run[cq] * a.scale_log2 * 0.69314718055994531f;   // raw max -> natural units
        ws[1] = z;
      }
    }
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs& a, int d, hipStream_t st) {
  // two column tiles per wave (244 VGPRs, two waves per SIMD); four tiles
  // halve the LDS operand reads per product but need one wave per SIMD, and
  // measured slower (310 vs 584 TFLOP/s at N = 32768)
  constexpr int CQ = 2;
  constexpr int rows = kWaves * 16 * CQ;
  int lmax = 0;
  for (int b = 0; b < a.B; ++b) lmax = max(lmax, a.L[b]);
  const dim3 grid((lmax + rows - 1) / rows, a.Hq, a.B);
  if (d == 128) prefill_attn_kernel<128, CQ><<<grid, 64 * kWaves, 0, st>>>(a);
  else          prefill_attn_kernel<64, CQ><<<grid, 64 * kWaves, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tb

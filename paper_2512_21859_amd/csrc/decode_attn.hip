// Single-token grouped-query decode attention over the compact KV cache,
// with the new token's K/V appended in the same launch.
//
// Work decomposition (one launch per decode step and layer):
//   grid  = (n_chunks, Hkv, B), block = 256 threads (4 waves).
//   Block (c, g, b) handles key rows [c*chunk, (c+1)*chunk) of KV head g of
//   sequence b for all G = Hq/Hkv query heads of that group, so every K/V
//   byte is read from HBM exactly once per step.
//   Inside a wave, a 16-lane row group owns one key row at a time; each lane
//   holds d/16 consecutive elements (16 bytes for bf16 d=128 and fp32 d=64),
//   so a wave instruction reads 4 whole rows.  Dot products are reduced over
//   the 16 lanes with DPP (fixed order); the softmax is online (running max
//   and sum per head) in the exp2 domain, with q pre-scaled by log2(e)/sqrt(d).
//   The four row groups and then the four waves are merged in a fixed order,
//   giving one partial (m, l, o[G][d]) per block.
//   The block that takes the last ticket of (b, g) merges the chunk partials
//   in chunk order (log-sum-exp), writes out[b][g*G .. g*G+G-1] and re-arms
//   its counter; the last head merger of sequence b then advances kv_len[b].
// Lengths are read on the device only, so the launch is graph-capturable.
// No floating-point atomics are used: results are bit-reproducible.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

template <int WORDS>
struct Raw {
  uint32_t w[WORDS];
};

template <int WORDS>
__device__ __forceinline__ Raw<WORDS> ld_raw(const void* p) {
  Raw<WORDS> r;
  if constexpr (WORDS == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    r.w[0] = v.x; r.w[1] = v.y;
  } else {
#pragma unroll
    for (int i = 0; i < WORDS / 4; ++i) {
      const uint4 v = reinterpret_cast<const uint4*>(p)[i];
      r.w[4 * i] = v.x; r.w[4 * i + 1] = v.y; r.w[4 * i + 2] = v.z; r.w[4 * i + 3] = v.w;
    }
  }
  return r;
}

template <int WORDS>
__device__ __forceinline__ void st_raw(void* p, const Raw<WORDS>& r) {
  if constexpr (WORDS == 2) {
    *reinterpret_cast<uint2*>(p) = make_uint2(r.w[0], r.w[1]);
  } else {
#pragma unroll
    for (int i = 0; i < WORDS / 4; ++i)
      reinterpret_cast<uint4*>(p)[i] =
          make_uint4(r.w[4 * i], r.w[4 * i + 1], r.w[4 * i + 2], r.w[4 * i + 3]);
  }
}

template <typename T, int WORDS>
__device__ __forceinline__ void widen(const Raw<WORDS>& r, float* out) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < WORDS; ++i) {
      out[2 * i] = __uint_as_float(r.w[i] << 16);
      out[2 * i + 1] = __uint_as_float(r.w[i] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < WORDS; ++i) out[i] = __uint_as_float(r.w[i]);
  }
}

__device__ __forceinline__ float exp2_guarded(float x) {
  // exp2(-inf) = 0 is what we want; the only guard needed is against
  // (-inf) - (-inf), which callers avoid by checking the running max.
  return exp2f(x);
}

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 4;                  // rows per row group per iteration
constexpr int kRowsPerIter = 4 * kUnroll;   // rows per wave per iteration

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a) {
  constexpr int DPL = D / 16;                     // elements per lane
  constexpr int WORDS = DPL * sizeof(T) / 4;      // 32-bit words per lane
  const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int grp = lane >> 4, sub = lane & 15;
  const int Hkv = a.Hkv, Hq = Hkv * G;

  __shared__ float s_o[kWaves][G][D];
  __shared__ float s_ml[kWaves][G][2];
  __shared__ int s_last;

  int n0 = a.kv_len[b];
  n0 = n0 < 0 ? 0 : (n0 > a.cap ? a.cap : n0);
  const int app = (a.append && n0 < a.cap) ? 1 : 0;
  const int N = n0 + app;
  const int lo = c * a.chunk;
  const int hi = min(lo + a.chunk, N);

  const size_t head_off = (static_cast<size_t>(b) * Hkv + g) * a.cap;
  const T* kc = static_cast<const T*>(a.k_cache) + head_off * D;
  const T* vc = static_cast<const T*>(a.v_cache) + head_off * D;
  const T* kn = static_cast<const T*>(a.k_new) + (static_cast<size_t>(b) * Hkv + g) * D;
  const T* vn = static_cast<const T*>(a.v_new) + (static_cast<size_t>(b) * Hkv + g) * D;

  // The block whose chunk holds row n0 stores the appended row.  No other
  // block of this launch reads that row from the cache.
  if (app && n0 >= lo && n0 < hi && wave == 0 && grp == 0) {
    st_raw<WORDS>(static_cast<T*>(a.k_cache) + (head_off + n0) * D + sub * DPL,
                  ld_raw<WORDS>(kn + sub * DPL));
    st_raw<WORDS>(static_cast<T*>(a.v_cache) + (head_off + n0) * D + sub * DPL,
                  ld_raw<WORDS>(vn + sub * DPL));
  }

  // q slice of every head of the group, pre-scaled into the exp2 domain.
  float qf[G][DPL];
  {
    const T* qb = static_cast<const T*>(a.q) + (static_cast<size_t>(b) * Hq + g * G) * D;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      widen<T, WORDS>(ld_raw<WORDS>(qb + h * D + sub * DPL), qf[h]);
#pragma unroll
      for (int e = 0; e < DPL; ++e) qf[h][e] *= a.scale_log2;
    }
  }

  float m[G], l[G], o[G][DPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY; l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[h][e] = 0.f;
  }

  const int per_wave = a.chunk / kWaves;
  const int wlo = lo + wave * per_wave;
  const int whi = min(wlo + per_wave, hi);
  for (int base = wlo; base < whi; base += kRowsPerIter) {
    Raw<WORDS> kr[kUnroll], vr[kUnroll];
    bool valid[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int row = base + u * 4 + grp;
      valid[u] = row < whi;
      if (valid[u]) {
        const bool is_new = app && row == n0;
        kr[u] = ld_raw<WORDS>((is_new ? kn : kc + static_cast<size_t>(row) * D) + sub * DPL);
        vr[u] = ld_raw<WORDS>((is_new ? vn : vc + static_cast<size_t>(row) * D) + sub * DPL);
      } else {
#pragma unroll
        for (int i = 0; i < WORDS; ++i) { kr[u].w[i] = 0u; vr[u].w[i] = 0u; }
      }
    }
    float s[kUnroll][G];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      float kf[DPL];
      widen<T, WORDS>(kr[u], kf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc = fmaf(qf[h][e], kf[e], acc);
        acc = row16_sum(acc);
        s[u][h] = valid[u] ? acc : -INFINITY;
      }
    }
    float vf[kUnroll][DPL];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) widen<T, WORDS>(vr[u], vf[u]);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mx = m[h];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) mx = fmaxf(mx, s[u][h]);
      if (mx == -INFINITY) continue;               // nothing valid yet
      const float corr = exp2_guarded(m[h] - mx);  // m = -inf gives 0
      float p[kUnroll];
      float psum = 0.f;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) { p[u] = exp2_guarded(s[u][h] - mx); psum += p[u]; }
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

  // Merge the four row groups of the wave (lanes sub, sub+16, sub+32, sub+48).
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float M = fmaxf(m[h], __shfl_xor(m[h], 16));
    M = fmaxf(M, __shfl_xor(M, 32));
    const float sc = (M == -INFINITY) ? 0.f : exp2_guarded(m[h] - M);
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

  // Merge the waves in a fixed order and write this block's partial.
  const size_t bg = static_cast<size_t>(b) * Hkv + g;
  float* part = a.part + (bg * a.n_chunks + c) * (G * (D + 2));
  for (int idx = tid; idx < G * D; idx += kThreads) {
    const int h = idx / D, e = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) M = fmaxf(M, s_ml[wv][h][0]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int wv = 0; wv < kWaves; ++wv) {
        const float sc = exp2_guarded(s_ml[wv][h][0] - M);
        L += s_ml[wv][h][1] * sc;
        O += s_o[wv][h][e] * sc;
      }
    }
    part[h * D + e] = O;
    if (e == 0) { part[G * D + 2 * h] = M; part[G * D + 2 * h + 1] = L; }
  }

  // Ticket: the last block of (b, g) merges the chunk partials.
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const int t = atomicAdd(a.head_ctr + bg, 1);
    s_last = (t == a.n_chunks - 1);
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  const int n_used = (N + a.chunk - 1) / a.chunk;
  const float* parts = a.part + bg * a.n_chunks * (G * (D + 2));
  T* out = static_cast<T*>(a.out) + (static_cast<size_t>(b) * Hq + g * G) * D;
  for (int idx = tid; idx < G * D; idx += kThreads) {
    const int h = idx / D, e = idx % D;
    float M = -INFINITY;
    for (int cc = 0; cc < n_used; ++cc)
      M = fmaxf(M, parts[cc * (G * (D + 2)) + G * D + 2 * h]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
      for (int cc = 0; cc < n_used; ++cc) {
        const float* pc = parts + cc * (G * (D + 2));
        const float mc = pc[G * D + 2 * h];
        const float sc = exp2_guarded(mc - M);
        L += pc[G * D + 2 * h + 1] * sc;
        O += pc[h * D + e] * sc;
      }
    }
    Elem<T>::store1(out + h * D + e, L > 0.f ? O / L : 0.f);
  }
  __syncthreads();
  if (tid == 0) {
    a.head_ctr[bg] = 0;                 // re-arm for the next launch
    __threadfence();
    const int t = atomicAdd(a.seq_ctr + b, 1);
    if (t == Hkv - 1) {                 // every head of b has read kv_len[b]
      a.kv_len[b] = N;
      a.seq_ctr[b] = 0;
    }
  }
}

template <typename T, int D>
hipError_t launch_g(const DecodeArgs& a, int G, hipStream_t st) {
  const dim3 grid(a.n_chunks, a.Hkv, a.B);
  switch (G) {
#define TB_CASE(GG) case GG: decode_kernel<T, D, GG><<<grid, kThreads, 0, st>>>(a); break;
    TB_CASE(1) TB_CASE(2) TB_CASE(3) TB_CASE(4) TB_CASE(5) TB_CASE(6) TB_CASE(7) TB_CASE(8)
#undef TB_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int decode_rows_per_chunk_unit() { return kWaves * kRowsPerIter; }

hipError_t launch_decode(const DecodeArgs& a, int G, int d, bool bf16, hipStream_t st) {
  if (bf16) return d == 128 ? launch_g<bf16_t, 128>(a, G, st) : launch_g<bf16_t, 64>(a, G, st);
  return d == 128 ? launch_g<float, 128>(a, G, st) : launch_g<float, 64>(a, G, st);
}

}  // namespace tb

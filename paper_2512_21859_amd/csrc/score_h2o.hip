// H2O scoring: the attention mass each prompt key receives from every prompt
// query under the causal softmax (the accumulated-attention scorer cited for
// the paper's fixed-ratio baselines, Sec. 6.1), summed over the query heads of
// its KV head.
//
//   A[g][j] = sum_{h in group g} sum_{i >= j} exp(s_hij - M_hi) / Z_hi,
//   s_hij = q[h][i] . k[g][j] / sqrt(d),  M_hi, Z_hi = max and sum of row i.
//
// Two passes over the causal (row tile, key tile) pairs, both on the float64
// matrix cores (v_mfma_f64_16x16x4_f64), since the selection compares scores
// within 1e-6 relative:
//   rows: block = a pair of 64-row query tiles (p, T-1-p) of one query head, so
//     every block covers T+1 causal tile pairs; key tiles stream through LDS;
//     each row keeps a running (max, sum) merged tile by tile in float64;
//   cols: block = a pair of 64-key tiles of one query head; query-row tiles
//     stream through LDS; p = exp(s - M)/Z summed over the tile's rows (lanes
//     then waves, fixed order) into per-head column masses;
//   merge: sums the G heads' column masses of a KV head in order, fp32 out.
// Per-logit exponentials reduce their argument exactly in float64 and
// evaluate 2^f (|f| <= 1/2) in fp32, as in the window scorer: on this part
// fp64 vector work competes with the fp64 matrix work for throughput.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

typedef __attribute__((ext_vector_type(4))) double f64x4;

constexpr int kTile = 64;          // query rows / keys per tile
constexpr int kThreads = 256;      // 4 waves of 16 rows

template <typename T>
__device__ __forceinline__ void load8(const T* p, float* out);
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, float* out) {
  Elem<bf16_t>::widen(ldg16(p), out);
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float* out) {
  Elem<float>::widen(ldg16(p), out);
  Elem<float>::widen(ldg16(p + 4), out + 4);
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(u & 0xffffffffu), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(u >> 32), CTRL, 0xF, 0xF, false);
  return __longlong_as_double((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) |
                              static_cast<uint32_t>(lo));
}
__device__ __forceinline__ double row16_sum_f64(double x) {
  x += dpp_f64<kDppQuadXor1>(x);
  x += dpp_f64<kDppQuadXor2>(x);
  x += dpp_f64<kDppRowHalfMirror>(x);
  x += dpp_f64<kDppRowMirror>(x);
  return x;
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_max_f32(float x) {
  x = fmaxf(x, dpp_f32<kDppQuadXor1>(x));
  x = fmaxf(x, dpp_f32<kDppQuadXor2>(x));
  x = fmaxf(x, dpp_f32<kDppRowHalfMirror>(x));
  x = fmaxf(x, dpp_f32<kDppRowMirror>(x));
  return x;
}
// 2^t as fp32 for a float64 t: t = n + f, n = round(t) exact, |f| <= 1/2
// rounded to fp32, hardware 2^f, exact scaling (tiny results flush to 0).
__device__ __forceinline__ float exp2_split(double t) {
  const double n = rint(fmax(t, -300.0));
  return ldexpf(__builtin_amdgcn_exp2f(static_cast<float>(t - n)), static_cast<int>(n));
}

// Stage 64 rows (row0.., valid below n_rows) of a [rows][D] matrix into LDS as
// fp32; thread t takes row t/4, elements (t%4)*D/4 ..; invalid rows are zero.
template <typename T, int D>
__device__ __forceinline__ void stage_tile(float (*dst)[D + 1], const T* src, int row0, int n_rows) {
  constexpr int PER = D / 4;
  const int r = threadIdx.x >> 2, c0 = (threadIdx.x & 3) * PER;
  float v[PER];
  if (row0 + r < n_rows) {
    const T* p = src + static_cast<size_t>(row0 + r) * D + c0;
#pragma unroll
    for (int e = 0; e < PER; e += 8) load8<T>(p + e, v + e);
  } else {
#pragma unroll
    for (int e = 0; e < PER; ++e) v[e] = 0.f;
  }
#pragma unroll
  for (int e = 0; e < PER; ++e) dst[r][c0 + e] = v[e];
}

// acc[kt] = Q[16 wave + rows] . K[16 kt + cols] over d (item v of lane l: row
// l/16 + 4v, column l%16 of the 16 x 16 tile).
template <int D>
__device__ __forceinline__ void tile_products(const float (*qs)[D + 1], const float (*ks)[D + 1],
                                              int wave, int q4, int r16, f64x4 acc[4]) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) acc[kt] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int k4 = 0; k4 < D / 4; ++k4) {
    const int dd = 4 * k4 + q4;
    const double av = static_cast<double>(qs[16 * wave + r16][dd]);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const double bv = static_cast<double>(ks[16 * kt + r16][dd]);
      acc[kt] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[kt], 0, 0, 0);
    }
  }
}

// Block order (one-dimensional grid): workgroup i runs on XCD i % 8, and
// XCD x takes the units x, x + 8, ... of (tile pair, batch, KV head), the G
// query heads of a unit in G consecutive slots of it, so the blocks that
// stream one KV head's keys share that XCD's L2 (L = 8192, 28 q / 4 kv
// heads: 9689-9709 -> 9621-9626 us per call; the passes are bound by the
// float64 products).  False for the padding of the last round.
__device__ __forceinline__ bool h2o_block(const H2oArgs& a, int& p, int& h, int& b) {
  const int G = a.Hq / a.Hkv;
  const int wg = static_cast<int>(blockIdx.x);
  const int slot = wg >> 3, unit = (slot / G) * 8 + (wg & 7);
  const int g = unit % a.Hkv, rb = unit / a.Hkv;
  b = rb % a.B;
  p = rb / a.B;
  h = g * G + slot % G;
  int nt_max = 0;
  for (int bb = 0; bb < a.B; ++bb) nt_max = max(nt_max, (a.L[bb] + kTile - 1) / kTile);
  return p < (nt_max + 1) / 2;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_rows_kernel(H2oArgs a) {
  int p, h, b;
  if (!h2o_block(a, p, h, b)) return;
  const int L = a.L[b], nt = (L + kTile - 1) / kTile;
  const int G = a.Hq / a.Hkv, g = h / G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q4 = lane >> 4, r16 = lane & 15;
  __shared__ float qs[kTile][D + 1];
  __shared__ float ks[kTile][D + 1];
  const T* qh = static_cast<const T*>(a.q) + (static_cast<size_t>(b) * a.Hq + h) * a.Lmax * D;
  const T* kg = static_cast<const T*>(a.k) + (static_cast<size_t>(b) * a.Hkv + g) * a.Lmax * D;
  const double c = a.scale * 1.4426950408889634;
  const size_t rowbase = (static_cast<size_t>(b) * a.Hq + h) * a.Lmax;

  for (int side = 0; side < 2; ++side) {
    const int rt = side == 0 ? p : nt - 1 - p;
    if (rt < 0 || rt >= nt || (side == 1 && rt <= p)) continue;   // block-uniform
    __syncthreads();
    stage_tile<T, D>(qs, qh, rt * kTile, L);
    double m_run[4], z_run[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) { m_run[v] = -INFINITY; z_run[v] = 0.0; }
    for (int kt = 0; kt <= rt; ++kt) {
      stage_tile<T, D>(ks, kg, kt * kTile, L);
      __syncthreads();
      f64x4 acc[4];
      tile_products<D>(qs, ks, wave, q4, r16, acc);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = rt * kTile + 16 * wave + q4 + 4 * v;
        bool ok[4];
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int key = kt * kTile + 16 * j + r16;
          ok[j] = key <= row && key < L;
          mx = fmaxf(mx, ok[j] ? static_cast<float>(acc[j][v]) : -INFINITY);
        }
        const double md = row16_max_f32(mx);      // reference dot product of the row
        float zs = 0.f;
        if (md != -INFINITY) {
#pragma unroll
          for (int j = 0; j < 4; ++j) zs += ok[j] ? exp2_split((acc[j][v] - md) * c) : 0.f;
        }
        const double z = row16_sum_f64(static_cast<double>(zs));
        if (md != -INFINITY) {                    // merge (md * scale, z) into the row's state
          const double ml = md * a.scale;
          if (ml > m_run[v]) {
            z_run[v] = (m_run[v] == -INFINITY ? 0.0 : z_run[v] * exp(m_run[v] - ml)) + z;
            m_run[v] = ml;
          } else {
            z_run[v] += z * exp(ml - m_run[v]);
          }
        }
      }
      __syncthreads();
    }
    if (r16 == 0) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = rt * kTile + 16 * wave + q4 + 4 * v;
        if (row < L) {
          a.row_M[rowbase + row] = m_run[v];
          a.row_Z[rowbase + row] = z_run[v];
        }
      }
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_cols_kernel(H2oArgs a) {
  int p, h, b;
  if (!h2o_block(a, p, h, b)) return;
  const int L = a.L[b], nt = (L + kTile - 1) / kTile;
  const int G = a.Hq / a.Hkv, g = h / G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q4 = lane >> 4, r16 = lane & 15;
  __shared__ float qs[kTile][D + 1];
  __shared__ float ks[kTile][D + 1];
  __shared__ double s_col[kThreads / 64][kTile];
  const T* qh = static_cast<const T*>(a.q) + (static_cast<size_t>(b) * a.Hq + h) * a.Lmax * D;
  const T* kg = static_cast<const T*>(a.k) + (static_cast<size_t>(b) * a.Hkv + g) * a.Lmax * D;
  const double c = a.scale * 1.4426950408889634;
  const size_t rowbase = (static_cast<size_t>(b) * a.Hq + h) * a.Lmax;

  for (int side = 0; side < 2; ++side) {
    const int kt = side == 0 ? p : nt - 1 - p;
    if (kt < 0 || kt >= nt || (side == 1 && kt <= p)) continue;   // block-uniform
    __syncthreads();
    stage_tile<T, D>(ks, kg, kt * kTile, L);
    double col[4] = {0.0, 0.0, 0.0, 0.0};         // column 16 j + r16 of this key tile
    for (int rt = kt; rt < nt; ++rt) {
      stage_tile<T, D>(qs, qh, rt * kTile, L);
      __syncthreads();
      f64x4 acc[4];
      tile_products<D>(qs, ks, wave, q4, r16, acc);
      double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = rt * kTile + 16 * wave + q4 + 4 * v;
        if (row < L) {
          const double Mr = a.row_M[rowbase + row];
          const double invZ = 1.0 / a.row_Z[rowbase + row];
          const double off = Mr * 1.4426950408889634;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = kt * kTile + 16 * j + r16;
            if (key <= row && key < L)
              part[j] += static_cast<double>(exp2_split(fma(acc[j][v], c, -off))) * invZ;
          }
        }
      }
      // sum over the 4 row groups of the wave (lanes r16, r16+16, +32, +48), fixed order
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        double x = part[j];
        x += __shfl_xor(x, 16);
        x += __shfl_xor(x, 32);
        col[j] += x;
      }
      __syncthreads();
    }
    if (q4 == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) s_col[wave][16 * j + r16] = col[j];
    }
    __syncthreads();
    if (tid < kTile) {
      const int key = kt * kTile + tid;
      if (key < L)
        a.col_part[rowbase + key] = ((s_col[0][tid] + s_col[1][tid]) + s_col[2][tid]) + s_col[3][tid];
    }
  }
}

// A[b][g][j] = sum over the G query heads of group g, in head order.
__global__ __launch_bounds__(kThreads) void h2o_merge_kernel(H2oArgs a) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= a.L[b]) return;
  const int G = a.Hq / a.Hkv;
  double s = 0.0;
  for (int hh = 0; hh < G; ++hh)
    s += a.col_part[(static_cast<size_t>(b) * a.Hq + g * G + hh) * a.Lmax + j];
  a.scores[(static_cast<size_t>(b) * a.Hkv + g) * a.Lmax + j] = static_cast<float>(s);
}

template <typename T, int D>
hipError_t launch_typed(const H2oArgs& a, hipStream_t st) {
  int nt_max = 0;
  for (int b = 0; b < a.B; ++b) nt_max = max(nt_max, (a.L[b] + kTile - 1) / kTile);
  const int units = (nt_max + 1) / 2 * a.B * a.Hkv;          // (tile pair, batch, KV head)
  const dim3 grid(((units + 7) / 8) * 8 * (a.Hq / a.Hkv));
  h2o_rows_kernel<T, D><<<grid, kThreads, 0, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  h2o_cols_kernel<T, D><<<grid, kThreads, 0, st>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 g3((a.Lmax + kThreads - 1) / kThreads, a.Hkv, a.B);
  h2o_merge_kernel<<<g3, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace

size_t h2o_ws_bytes(int B, int Lmax, int Hq) {
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  return 3 * up(static_cast<size_t>(B) * Hq * Lmax * sizeof(double));
}

hipError_t launch_h2o(const H2oArgs& a, int d, bool bf16, hipStream_t st) {
  if (bf16) return d == 128 ? launch_typed<bf16_t, 128>(a, st) : launch_typed<bf16_t, 64>(a, st);
  return d == 128 ? launch_typed<float, 128>(a, st) : launch_typed<float, 64>(a, st);
}

}  // namespace tb

// Observation-window scoring: softmax of the last w queries against all
// prompt keys, summed per KV head over the G*w window rows, then max-pooled.
//
// Precision.  The selection that follows is compared position by position, so
// scores are kept to ~1e-7 relative: dot products of the (exact) bf16/fp32
// inputs are accumulated in float64, exponentials are float64, and sums are
// float64.  Only the per-tile exponentials are stored as fp32 (relative
// rounding 6e-8) and the final scores are rounded to fp32 once.
//
// Three kernels, all with fixed-order reductions (no atomics):
//   K1 score_tiles: block = (64-key tile, <=256 window rows) of one KV head.
//      Stages the window queries (transposed, fp32) and the key tile (fp64)
//      in LDS in 32-wide d chunks; each thread computes a 4-row x 16-key
//      micro-tile of float64 dot products (the 16 keys are a wave-uniform LDS
//      broadcast).  Applies the causal mask, takes the tile max m per row,
//      stores e = exp(s - m) as fp32 and z = sum(e) per row.
//   K2 row_stats: one wave per window row merges the tiles' (m, z) into the
//      row's global max M and normaliser Z.
//   K3 score_accum: block = 64 prefix columns (+ pool halo).  For each column
//      j, A[j] = sum_r e[r][j] * exp(m[r][tile(j)] - M[r]) / Z[r] in float64,
//      then the max-pool over |j - j'| <= pool/2 within the prefix.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

constexpr int kThreads = 256;
constexpr int kT = kScoreTile;     // keys per tile (64)
constexpr int kRows = kScoreRows;  // rows per block (256)
constexpr int kDC = 32;            // d chunk staged in LDS

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

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void score_tiles_kernel(ScoreArgs a) {
  const int tile = blockIdx.x / a.row_chunks, rc = blockIdx.x % a.row_chunks;
  const int g = blockIdx.y, b = blockIdx.z;
  const int L = a.L[b];
  const int kbase_tile = tile * kT;
  if (kbase_tile >= L) return;
  const int G = a.Hq / a.Hkv, R = a.R, w = a.w;
  const int row0 = rc * kRows;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  __shared__ float qT[kDC][kRows];                 // 32 KB
  __shared__ double kT_[kDC][kT];                  // 16 KB
  __shared__ double red[4][kRows];                 // 8 KB

  double acc[4][16];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 16; ++c) acc[r][c] = 0.0;

  const T* kh = static_cast<const T*>(a.k) + (static_cast<size_t>(b) * a.Hkv + g) * a.Lmax * D;
  for (int dc = 0; dc < D; dc += kDC) {
    // Stage the window queries of this d chunk, transposed: qT[dd][row].
    {
      const int r = row0 + tid;
      float qv[kDC];
      if (r < R) {
        const int h = g * G + r / w, i = r % w;
        const T* src = static_cast<const T*>(a.q_win) +
                       ((static_cast<size_t>(b) * a.Hq + h) * w + i) * D + dc;
#pragma unroll
        for (int e = 0; e < kDC; e += 8) load8<T>(src + e, qv + e);
      } else {
#pragma unroll
        for (int e = 0; e < kDC; ++e) qv[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < kDC; ++e) qT[e][tid] = qv[e];
    }
    // Stage the key tile of this d chunk in float64: kT_[dd][key].
    {
      const int kk = tid >> 2, dp = (tid & 3) * 8;
      const int j = kbase_tile + kk;
      float kv[8];
      if (j < L) {
        load8<T>(kh + static_cast<size_t>(j) * D + dc + dp, kv);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kv[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) kT_[dp + e][kk] = static_cast<double>(kv[e]);
    }
    __syncthreads();
#pragma unroll 4
    for (int dd = 0; dd < kDC; ++dd) {
      const float4 q4 = *reinterpret_cast<const float4*>(&qT[dd][4 * lane]);
      const double q[4] = {q4.x, q4.y, q4.z, q4.w};
      double kv[16];
#pragma unroll
      for (int c = 0; c < 16; c += 2) {
        const double2 k2 = *reinterpret_cast<const double2*>(&kT_[dd][16 * wave + c]);
        kv[c] = k2.x; kv[c + 1] = k2.y;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 16; ++c) acc[r][c] = fma(q[r], kv[c], acc[r][c]);
    }
    __syncthreads();
  }

  // Masked logits; tile max per row.
  const int kbase = kbase_tile + 16 * wave;
  double rmax[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int rg = row0 + 4 * lane + r;
    const int lim = (rg < R) ? min(L - 1, L - w + rg % w) : -1;   // last visible key
    double mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const double s = (kbase + c <= lim) ? acc[r][c] * a.scale : -INFINITY;
      acc[r][c] = s;
      mx = fmax(mx, s);
    }
    rmax[r] = mx;
    red[wave][4 * lane + r] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int rr = 4 * lane + r;
    rmax[r] = fmax(fmax(red[0][rr], red[1][rr]), fmax(red[2][rr], red[3][rr]));
  }
  __syncthreads();

  // e = exp(s - m) (fp32 store) and per-row partial sums.
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  float* ebase = a.e + (bg * a.n_tiles + tile) * static_cast<size_t>(R) * kT;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int rg = row0 + 4 * lane + r;
    double zsum = 0.0;
    float ef[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const double ev = (rmax[r] == -INFINITY) ? 0.0 : exp(acc[r][c] - rmax[r]);
      zsum += ev;
      ef[c] = static_cast<float>(ev);
    }
    red[wave][4 * lane + r] = zsum;
    if (rg < R) {
      float4* dst = reinterpret_cast<float4*>(ebase + static_cast<size_t>(rg) * kT + 16 * wave);
#pragma unroll
      for (int c = 0; c < 4; ++c)
        dst[c] = make_float4(ef[4 * c], ef[4 * c + 1], ef[4 * c + 2], ef[4 * c + 3]);
    }
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rr = 4 * lane + r, rg = row0 + rr;
      if (rg < R) {
        const size_t o = (bg * a.n_tiles + tile) * R + rg;
        a.tile_m[o] = rmax[r];
        a.tile_z[o] = ((red[0][rr] + red[1][rr]) + red[2][rr]) + red[3][rr];
      }
    }
  }
}

// One wave per (b, g, row): global max and normaliser over the row's tiles.
__global__ __launch_bounds__(kThreads) void row_stats_kernel(ScoreArgs a) {
  const int wid = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int total = a.B * a.Hkv * a.R;
  if (wid >= total) return;
  const int r = wid % a.R;
  const int bg = wid / a.R;
  const int b = bg / a.Hkv;
  const int nt = (a.L[b] + kT - 1) / kT;
  double M = -INFINITY, Z = 0.0;
  for (int t = lane; t < nt; t += 64) {
    const size_t o = (static_cast<size_t>(bg) * a.n_tiles + t) * a.R + r;
    const double m = a.tile_m[o], z = a.tile_z[o];
    if (m == -INFINITY) continue;
    if (m > M) { Z = Z * exp(M - m) + z; M = m; }
    else       { Z += z * exp(m - M); }
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    // Both partners evaluate the same expression with the same operand order
    // (lower lane first), so every lane ends with bit-identical (M, Z).
    const double Mo = __shfl_xor(M, off), Zo = __shfl_xor(Z, off);
    const bool upper = (lane & off) != 0;
    const double Ma = upper ? Mo : M, Za = upper ? Zo : Z;
    const double Mb = upper ? M : Mo, Zb = upper ? Z : Zo;
    const double Mn = fmax(Ma, Mb);
    Z = (Mn == -INFINITY) ? 0.0 : Za * exp(Ma - Mn) + Zb * exp(Mb - Mn);
    M = Mn;
  }
  if (lane == 0) {
    a.row_M[static_cast<size_t>(bg) * a.R + r] = M;
    a.row_Z[static_cast<size_t>(bg) * a.R + r] = Z;
  }
}

constexpr int kMaxHalo = 64;

__global__ __launch_bounds__(kThreads) void score_accum_kernel(ScoreArgs a) {
  const int ct = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int L = a.L[b], pref = L - a.w;
  const int j0 = ct * kT;
  if (j0 >= pref) return;
  const int R = a.R, hp = a.pool / 2;
  const int ncols = kT + 2 * hp;
  const int nt = (L + kT - 1) / kT;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const int tid = threadIdx.x;

  __shared__ double coef[3][1024];                 // tiles ct-1, ct, ct+1
  __shared__ double part[4][kT + 2 * kMaxHalo];
  __shared__ double raw[kT + 2 * kMaxHalo];

  for (int idx = tid; idx < 3 * R; idx += kThreads) {
    const int tt = ct - 1 + idx / R, r = idx % R;
    double cv = 0.0;
    if (tt >= 0 && tt < nt) {
      const double m = a.tile_m[(bg * a.n_tiles + tt) * R + r];
      const double M = a.row_M[bg * R + r], Z = a.row_Z[bg * R + r];
      if (m != -INFINITY && Z > 0.0) cv = exp(m - M) / Z;
    }
    coef[idx / R][r] = cv;
  }
  __syncthreads();

  const float* ebg = a.e + bg * a.n_tiles * static_cast<size_t>(R) * kT;
  for (int item = tid; item < 4 * ncols; item += kThreads) {
    const int col = item % ncols, rg = item / ncols;
    const int j = j0 - hp + col;
    double s = 0.0;
    if (j >= 0 && j < pref) {
      const int tt = j / kT, jj = j % kT;
      const float* et = ebg + static_cast<size_t>(tt) * R * kT + jj;
      const double* cf = coef[tt - ct + 1];
      for (int r = rg; r < R; r += 4) s = fma(static_cast<double>(et[static_cast<size_t>(r) * kT]), cf[r], s);
    }
    part[rg][col] = s;
  }
  __syncthreads();
  for (int col = tid; col < ncols; col += kThreads)
    raw[col] = ((part[0][col] + part[1][col]) + part[2][col]) + part[3][col];
  __syncthreads();

  if (tid < kT) {
    const int j = j0 + tid;
    if (j < pref) {
      const int col = tid + hp;
      double mx = raw[col];
      for (int dj = -hp; dj <= hp; ++dj) {
        const int jn = j + dj;
        if (jn >= 0 && jn < pref) mx = fmax(mx, raw[col + dj]);
      }
      const size_t o = bg * a.Lmax + j;
      a.scores[o] = static_cast<float>(mx);
      if (a.raw_scores) a.raw_scores[o] = static_cast<float>(raw[col]);
    }
  }
}

}  // namespace

size_t score_ws_bytes(int B, int Lmax, int Hkv, int R) {
  const size_t n_tiles = (static_cast<size_t>(Lmax) + kT - 1) / kT;
  const size_t units = static_cast<size_t>(B) * Hkv;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  size_t bytes = up(units * n_tiles * R * kT * sizeof(float));       // e
  bytes += 2 * up(units * n_tiles * R * sizeof(double));             // tile m, z
  bytes += 2 * up(units * R * sizeof(double));                       // row M, Z
  return bytes;
}

hipError_t launch_score(const ScoreArgs& a, int d, bool bf16, hipStream_t st) {
  const dim3 g1(a.n_tiles * a.row_chunks, a.Hkv, a.B);
  if (bf16) {
    if (d == 128) score_tiles_kernel<bf16_t, 128><<<g1, kThreads, 0, st>>>(a);
    else          score_tiles_kernel<bf16_t, 64><<<g1, kThreads, 0, st>>>(a);
  } else {
    if (d == 128) score_tiles_kernel<float, 128><<<g1, kThreads, 0, st>>>(a);
    else          score_tiles_kernel<float, 64><<<g1, kThreads, 0, st>>>(a);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int waves = a.B * a.Hkv * a.R;
  row_stats_kernel<<<(waves + 3) / 4, kThreads, 0, st>>>(a);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const dim3 g3((a.Lmax + kT - 1) / kT, a.Hkv, a.B);
  score_accum_kernel<<<g3, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tb

// Observation-window scoring: softmax of the last w queries against all
// prompt keys, summed per KV head over the G*w window rows, then max-pooled.
//
// Precision.  The selection that follows is compared position by position, so
// scores are kept to ~1e-7 relative: dot products of the (exact) bf16/fp32
// inputs are accumulated in float64, exponent arguments are reduced in float64,
// and sums are float64.  The per-logit exponentials (fp32, within ~1.5e-7
// relative) and the raw scores (fp32 rounding, 6e-8) are the only
// single-precision values; pooling is a max, so it is exact.
//
// Four kernels, all with fixed-order reductions (no atomics):
//   K1 score_tiles: block = (64-key tile, <=256 window rows) of one KV head,
//      512 threads; wave w owns 32 rows x the 64 keys (waves whose rows are all
//      padding skip the products).  With 4, 6 or 7 row pairs and enough
//      blocks, a block instead takes 8 consecutive units (32 rows x one tile,
//      numbered tile-major) over at most two tiles, so no wave idles.
//      Window queries (as fp32) and keys (as
//      float64, converted once since every wave reads them) are staged in LDS
//      in 32-wide d chunks, the next chunk's global loads in flight while the
//      current one is multiplied; the float64 dot products run on the matrix
//      cores (v_mfma_f64_16x16x4_f64, 2 x 4 tiles of 16 x 16 per wave).  Each
//      row's 64 logits sit in one 16-lane DPP row, so the causal mask, a tile
//      reference m (the row's largest dot product rounded to fp32) and
//      z = sum exp(s - m) need no LDS.  Stores e = exp(s - m) (fp32, one float4
//      per lane and row: keys r, r+16, r+32, r+48) and (m, z) per (row, tile).
//   K2 row_stats: one wave per window row merges its tiles' (m, z) into the
//      row's global max M and normaliser Z.
//   K3 score_accum: block = 64 prefix columns; A[j] = sum_r e[r][j] *
//      exp(m[r][tile] - M[r]) / Z[r] in float64 (four row groups, four
//      independent accumulators each, combined in a fixed order); raw A as fp32.
//   K4 pool: max of the raw scores over |j - j'| <= pool/2 within the prefix
//      (or their mean with zeros outside the prefix and divisor pool, summed in
//      float64, for the average-pool variant).
//
// The per-logit exponential is the one place fp64 arithmetic is avoided: on
// this part the fp64 vector instructions compete with the fp64 matrix
// instructions for the same throughput, so K1's epilogue reduces the argument
// in fp64 (exactly) and evaluates 2^f for |f| <= 1/2 in fp32.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

typedef __attribute__((ext_vector_type(4))) double f64x4;
typedef __attribute__((ext_vector_type(4))) float f32x4n;

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

// 2^t as fp32 for a float64 t >= -300: t = n + f with n = round(t) exact and
// |f| <= 1/2, so only f is rounded to fp32 (relative effect on 2^f below
// 3e-8); 2^f comes from the hardware base-2 exponential (about 1 ulp) and the
// scaling by 2^n is exact (results under the smallest fp32 subnormal are 0).
__device__ __forceinline__ float exp2_split(double t) {
  const double n = rint(t);
  return ldexpf(__builtin_amdgcn_exp2f(static_cast<float>(t - n)), static_cast<int>(n));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(u & 0xffffffffu), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(u >> 32), CTRL, 0xF, 0xF, false);
  return __longlong_as_double((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) |
                              static_cast<uint32_t>(lo));
}
// Sum over the 16 lanes of a DPP row; every lane gets the result, in a fixed
// order (deterministic).
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

constexpr int kTilesThreads = 512;
constexpr int kWaveRows = 32;      // window rows per wave in score_tiles

// Work unit of a wave: 32 window rows x one 64-key tile.  NS = 1: block =
// (tile, 256-row chunk), wave w takes rows 32 w .. 32 w + 31 (waves past R
// idle).  NS = 2 (R <= 256 with P = ceil(R / 32) row pairs, P in {4, 6, 7}):
// the units are numbered tile-major, u = P t + p, and block j takes units
// 8 j .. 8 j + 7, so every wave has one and the block's units span at most two
// tiles, whose keys it stages together.  With one idle wave per block (R =
// 224) the busiest SIMD of a CU carries as many waves as at R = 256 and the
// block barriers pace every block by it; packing gives each block 8 busy waves.
template <typename T, int D, int NS>
__global__ __launch_bounds__(kTilesThreads, 2) void score_tiles_kernel(ScoreArgs a) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int L = a.L[b];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int t0, tile, pair, row0;                       // block's first tile; this wave's unit
  if constexpr (NS == 1) {
    t0 = tile = blockIdx.x / a.row_chunks;
    row0 = (blockIdx.x % a.row_chunks) * kRows;
    pair = wave;
  } else {
    const int P = a.pack_pairs;
    const int u = static_cast<int>(blockIdx.x) * 8 + wave;
    t0 = static_cast<int>(blockIdx.x) * 8 / P;
    tile = u / P;
    pair = u % P;
    row0 = 0;
  }
  if (t0 * kT >= L) return;                       // block-uniform
  const int kbase = tile * kT;
  const int G = a.Hq / a.Hkv, R = a.R, w = a.w;
  const int q4 = lane >> 4, r16 = lane & 15;
  // wave-uniform: the unit has real rows and real keys
  const bool active = row0 + kWaveRows * pair < R && kbase < L;

  __shared__ float qs[kRows][kDC + 1];             // +1: conflict-free column reads
  __shared__ double ks[NS * kT][kDC + 1];        // keys staged as float64: every wave reads them
  __shared__ int s_lim[kRows];                     // last key a row sees (-1: padding)
  if (tid < kRows) {
    const int r = row0 + tid;
    s_lim[tid] = r < R ? min(L - 1, L - w + r % w) : -1;
  }

  // Staging: two threads per window row (16 elements each) and four threads
  // per key (8 elements each; the first 256 threads when NS = 1).
  const int qrow = tid >> 1, qoff = (tid & 1) * 16;
  const bool qvalid = row0 + qrow < R;
  const T* qsrc = nullptr;
  if (qvalid) {
    const int r = row0 + qrow, h = g * G + r / w, i = r % w;
    qsrc = static_cast<const T*>(a.q_win) + ((static_cast<size_t>(b) * a.Hq + h) * w + i) * D + qoff;
  }
  const int kk = (tid & (NS * 256 - 1)) >> 2, kdp = (tid & 3) * 8;
  const bool kvalid = tid < NS * 256 && t0 * kT + kk < L;
  const T* ksrc = static_cast<const T*>(a.k) +
                  ((static_cast<size_t>(b) * a.Hkv + g) * a.Lmax + t0 * kT + kk) * D + kdp;
  float qv[16], kv[8];
  auto fetch = [&](int dc) {
    if (qvalid) {
      load8<T>(qsrc + dc, qv);
      load8<T>(qsrc + dc + 8, qv + 8);
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) qv[e] = 0.f;
    }
    if (kvalid) {
      load8<T>(ksrc + dc, kv);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) kv[e] = 0.f;
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int e = 0; e < 16; ++e) qs[qrow][qoff + e] = qv[e];
    if (tid < NS * 256) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ks[kk][kdp + e] = static_cast<double>(kv[e]);
    }
  };

  f64x4 acc[2][4];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) acc[rt][kt] = f64x4{0.0, 0.0, 0.0, 0.0};

  fetch(0);
  stage();
  __syncthreads();
#pragma unroll 1
  for (int dc = 0; dc < D; dc += kDC) {
    const bool more = dc + kDC < D;
    if (more) fetch(dc + kDC);                     // in flight during the products
    if (active) {
#pragma unroll
      for (int k4 = 0; k4 < kDC / 4; ++k4) {
        const int dd = 4 * k4 + q4;                // this lane's k index
        double av[2], bv[4];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          av[rt] = static_cast<double>(qs[kWaveRows * pair + 16 * rt + r16][dd]);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) bv[kt] = ks[(tile - t0) * kT + 16 * kt + r16][dd];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
            acc[rt][kt] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[rt], bv[kt], acc[rt][kt], 0, 0, 0);
      }
    }
    __syncthreads();
    if (more) {
      stage();
      __syncthreads();
    }
  }
  if (!active) return;

  // acc[rt][kt][v] = q(row 16 rt + q4 + 4 v) . k(key 16 kt + r16) of this wave
  // (the float64 16x16x4 product returns rows interleaved: item v of lane l is
  // row l/16 + 4v, column l%16).
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  float* ebase = a.e + (bg * a.n_tiles + tile) * static_cast<size_t>(R) * kT;
  const double c = a.scale * 1.4426950408889634;  // exp(x) = 2^(x log2 e)
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int rl = kWaveRows * pair + 16 * rt + q4 + 4 * v;
      const int lim = s_lim[rl];
      bool ok[4];
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        ok[kt] = kbase + 16 * kt + r16 <= lim;
        mx = fmaxf(mx, ok[kt] ? static_cast<float>(acc[rt][kt][v]) : -INFINITY);
      }
      // reference: the row's largest dot product rounded to fp32 (exact as a
      // double); e and m below use the same value, so any nearby one is as good
      const double md = row16_max_f32(mx);
      const double mdc = md * c;
      float ev[4], zs = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        ev[kt] = ok[kt] ? exp2_split(fma(acc[rt][kt][v], c, -mdc)) : 0.f;
        zs += ev[kt];
      }
      const double z = row16_sum_f64(static_cast<double>(zs));
      const int rg = row0 + rl;
      if (rg < R) {
        float* dst = ebase + static_cast<size_t>(rg) * kT + 4 * r16;
        if (a.stream_e) __builtin_nontemporal_store(f32x4n{ev[0], ev[1], ev[2], ev[3]},
                                                    reinterpret_cast<f32x4n*>(dst));
        else            *reinterpret_cast<float4*>(dst) = make_float4(ev[0], ev[1], ev[2], ev[3]);
        if (r16 == 0) {
          const size_t o = (bg * R + rg) * a.n_tiles + tile;
          a.tile_m[o] = md * a.scale;       // -inf when the whole row-tile is masked
          a.tile_z[o] = z;
        }
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
  const size_t rowo = (static_cast<size_t>(bg) * a.R + r) * a.n_tiles;
  double M = -INFINITY, Z = 0.0;
  // the lane's tiles t = lane, lane + 64, ... in that order, their loads
  // issued 8 at a time ahead of the merge (one memory round trip per 8)
  constexpr int kAhead = 8;
  for (int t0 = lane; t0 < nt; t0 += 64 * kAhead) {
    double mv[kAhead], zv[kAhead];
#pragma unroll
    for (int k = 0; k < kAhead; ++k) {
      const int t = min(t0 + 64 * k, nt - 1);
      mv[k] = a.tile_m[rowo + t];
      zv[k] = a.tile_z[rowo + t];
    }
#pragma unroll
    for (int k = 0; k < kAhead; ++k) {
      const double m = mv[k], z = zv[k];
      if (t0 + 64 * k >= nt || m == -INFINITY) continue;
      if (m > M) { Z = Z * exp(M - m) + z; M = m; }
      else       { Z += z * exp(m - M); }
    }
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

// Column sums of one 64-column tile: thread (rg, col), rows r = rg + 4k.
__global__ __launch_bounds__(kThreads) void score_accum_kernel(ScoreArgs a) {
  const int ct = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int L = a.L[b], pref = L - a.w;
  const int j0 = ct * kT;
  if (j0 >= pref) return;
  const int R = a.R;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const int tid = threadIdx.x;

  __shared__ double coef[1024];
  __shared__ double part[16][kT];

  for (int r = tid; r < R; r += kThreads) {
    const double m = a.tile_m[(bg * R + r) * a.n_tiles + ct];
    const double M = a.row_M[bg * R + r], Z = a.row_Z[bg * R + r];
    coef[r] = (m != -INFINITY && Z > 0.0) ? exp(m - M) / Z : 0.0;
  }
  __syncthreads();
  // Key col of a tile row is stored at 4 (col % 16) + col / 16, so the 16-byte
  // vector at 4 q holds cols q, q + 16, q + 32, q + 48.  Thread (q, rs) reads
  // those vectors from rows rs, rs + 16, ..., eight loads in flight, and keeps
  // four float64 column sums; the 16 row phases are then added in order.
  // (Sixteen loads in flight, issued before the coefficients, measured slower.)
  const int q = tid & 15, rs = tid >> 4;
  const float* et = a.e + (bg * a.n_tiles + ct) * static_cast<size_t>(R) * kT + 4 * q;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  constexpr int kBatch = 8;
  for (int rb = rs; rb < R; rb += 16 * kBatch) {
    float4 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int r = rb + 16 * u;
      v[u] = r < R ? *reinterpret_cast<const float4*>(et + static_cast<size_t>(r) * kT)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int r = rb + 16 * u;
      const double c = r < R ? coef[r] : 0.0;
      s0 = fma(static_cast<double>(v[u].x), c, s0);
      s1 = fma(static_cast<double>(v[u].y), c, s1);
      s2 = fma(static_cast<double>(v[u].z), c, s2);
      s3 = fma(static_cast<double>(v[u].w), c, s3);
    }
  }
  part[rs][q] = s0;
  part[rs][q + 16] = s1;
  part[rs][q + 32] = s2;
  part[rs][q + 48] = s3;
  __syncthreads();
  if (tid < kT) {
    const int j = j0 + tid;
    if (j < pref) {
      double A = part[0][tid];
#pragma unroll
      for (int k = 1; k < 16; ++k) A += part[k][tid];
      a.raw[bg * a.Lmax + j] = static_cast<float>(A);
    }
  }
}

__global__ __launch_bounds__(kThreads) void pool_kernel(ScoreArgs a) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int j = blockIdx.x * kThreads + threadIdx.x;
  const int pref = a.L[b] - a.w;
  if (j >= pref) return;
  const int hp = a.pool / 2;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const float* raw = a.raw + bg * a.Lmax;
  const int lo = max(j - hp, 0), hi = min(j + hp, pref - 1);
  if (a.pool_avg) {
    // positions outside the prefix count as zeros; the divisor is always pool
    double sum = 0.0;
    for (int jn = lo; jn <= hi; ++jn) sum += raw[jn];
    a.scores[bg * a.Lmax + j] = static_cast<float>(sum / a.pool);
  } else {
    float mx = raw[j];
    for (int jn = lo; jn <= hi; ++jn) mx = fmaxf(mx, raw[jn]);
    a.scores[bg * a.Lmax + j] = mx;
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
  bytes += up(units * Lmax * sizeof(float));                         // raw scores
  return bytes;
}

hipError_t launch_score(const ScoreArgs& args, int d, bool bf16, hipStream_t st) {
  // Exponentials larger than the 256 MB last-level cache cannot stay there for
  // K3 anyway: write them with streaming stores (at L = 131072, 8 KV heads,
  // 1.07 GB: K3 reads them back in 199 us instead of 223, K1 unchanged);
  // smaller ones are written normally so that K3 finds them cached
  // (streaming them cost ~2 us per call at L = 8192).
  ScoreArgs a = args;
  const double e_bytes = 4.0 * kT * a.R * a.n_tiles * a.Hkv * a.B;
  a.stream_e = e_bytes > 256.0 * (1 << 20);
  // Packed blocks (P = 4, 6 or 7 row pairs: waves would idle, and every run of
  // 8 units spans at most two tiles) when packing lowers the blocks per CU and
  // still leaves two per CU (two resident blocks overlap each other's barriers
  // and staging).  Measured, d = 128, one scoring call, packed against not
  // (us): P = 7, 4 KV heads: L = 32768 174 / 187 (8 -> 7 blocks per CU),
  // 36864 198 / 210, 65536 352 / 369, but 8192 64.0 / 62.5, 16384 107 / 105,
  // 24576 157 / 153, 28672 175 / 169 (blocks per CU unchanged); P = 6:
  // 16384 85.0 / 99.7, 32768 152 / 184, 8192 60.1 / 59.2 (2 -> 2); P = 4:
  // 16384 60.9 / 66.6, 32768 107 / 117, 8192 43.9 / 40.8 (one block per CU).
  constexpr long long kCUs = 256;
  const int P = (a.R + kWaveRows - 1) / kWaveRows;
  const long long units = static_cast<long long>(a.Hkv) * a.B;
  const long long plain = static_cast<long long>(a.n_tiles) * units;
  const long long packed = (static_cast<long long>(P) * a.n_tiles + 7) / 8 * units;
  const bool pack = a.row_chunks == 1 && (P == 4 || P == 6 || P == 7) && packed >= 2 * kCUs &&
                    (packed + kCUs - 1) / kCUs < (plain + kCUs - 1) / kCUs;
  a.pack_pairs = pack ? P : 0;
  if (pack) {
    const dim3 g1((P * a.n_tiles + 7) / 8, a.Hkv, a.B);
    if (bf16) {
      if (d == 128) score_tiles_kernel<bf16_t, 128, 2><<<g1, kTilesThreads, 0, st>>>(a);
      else          score_tiles_kernel<bf16_t, 64, 2><<<g1, kTilesThreads, 0, st>>>(a);
    } else {
      if (d == 128) score_tiles_kernel<float, 128, 2><<<g1, kTilesThreads, 0, st>>>(a);
      else          score_tiles_kernel<float, 64, 2><<<g1, kTilesThreads, 0, st>>>(a);
    }
  } else {
    const dim3 g1(a.n_tiles * a.row_chunks, a.Hkv, a.B);
    if (bf16) {
      if (d == 128) score_tiles_kernel<bf16_t, 128, 1><<<g1, kTilesThreads, 0, st>>>(a);
      else          score_tiles_kernel<bf16_t, 64, 1><<<g1, kTilesThreads, 0, st>>>(a);
    } else {
      if (d == 128) score_tiles_kernel<float, 128, 1><<<g1, kTilesThreads, 0, st>>>(a);
      else          score_tiles_kernel<float, 64, 1><<<g1, kTilesThreads, 0, st>>>(a);
    }
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int waves = a.B * a.Hkv * a.R;
  row_stats_kernel<<<(waves + 3) / 4, kThreads, 0, st>>>(a);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const dim3 g3((a.Lmax + kT - 1) / kT, a.Hkv, a.B);
  score_accum_kernel<<<g3, kThreads, 0, st>>>(a);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const dim3 g4((a.Lmax + kThreads - 1) / kThreads, a.Hkv, a.B);
  pool_kernel<<<g4, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tb

// Per-KV-head top-k of the pooled scores with lower-position tie-break,
// emitted as ascending kept positions followed by the window.
//
// One block of 1024 threads per (sequence, KV head).  Each score is mapped to
// an unsigned key that orders like the float (non-negative: sign bit set;
// negative: all bits flipped; -0 as +0), so the selection is integer work and
// bit-exact for any finite scores (KNorm's are negative):
//   0. one pass over the prefix finds the largest and smallest key; the bits
//      above their highest differing bit are common to every key, so the radix
//      search starts just below them (digits spread over bins from the first
//      pass instead of piling into the one or two bins the exponent's top bits
//      give, which would serialise the LDS atomics);
//   1. radix select with digits of up to 11 bits (at most 3 passes) finds the
//      key tau of the n_sel-th largest score and how many tau-valued positions
//      to take (histogram bins are replicated per lane group to spread
//      same-bin atomics over LDS banks);
//   2. an ordered emit walks the prefix in tiles of 16384 positions (16 per
//      thread, contiguous), with one block-wide exclusive scan of the packed
//      counts (greater-than-tau, equal-to-tau) per tile.  Positions equal to
//      tau are taken lowest index first, so a thread's output offset is
//      (#greater before it) + min(#equal before it, equal-needed).
// A prefix of up to 32768 positions is read from HBM once and kept in LDS for
// every pass; a longer one is re-read (from L2) by each pass and staged
// through the same LDS buffer one emit tile at a time.  Given a workspace,
// longer prefixes are instead split over up to 32 blocks per KV head (the
// second half of this file): one block per head is then 3-4x slower, since a
// single CU streams every pass.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kBits = 11;
constexpr int kBins = 1 << kBits;
constexpr int kPer = 16;                      // positions per thread per emit tile
constexpr int kTileN = kThreads * kPer;       // 16384
constexpr int kCacheN = 32768;                // prefix kept in LDS when it fits

__device__ __forceinline__ uint32_t key_of(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;               // -0 orders as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Block-wide exclusive scan of v (1024 threads); also returns the total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* s_wave,
                                                         uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const uint32_t t = lane < kWaves ? s_wave[lane] : 0u;
    uint32_t x = t;
#pragma unroll
    for (int off = 1; off < kWaves; off <<= 1) {
      const uint32_t y = __shfl_up(x, off);
      if (lane >= off) x += y;
    }
    if (lane < kWaves) s_wave[kWaves + lane] = x - t;   // exclusive wave offsets
    if (lane == kWaves - 1) s_wave[2 * kWaves] = x;     // block total
  }
  __syncthreads();
  const uint32_t res = s_wave[kWaves + wave] + incl - v;
  total = s_wave[2 * kWaves];
  __syncthreads();
  return res;
}

// Block-wide max and min of 32-bit keys (every thread gets both).
__device__ __forceinline__ void block_max_min(uint32_t& mx, uint32_t& mn, uint32_t* s_wave) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    mx = max(mx, static_cast<uint32_t>(__shfl_xor(mx, off)));
    mn = min(mn, static_cast<uint32_t>(__shfl_xor(mn, off)));
  }
  if (lane == 0) { s_wave[wave] = mx; s_wave[kWaves + wave] = mn; }
  __syncthreads();
  mx = 0u;
  mn = 0xffffffffu;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) { mx = max(mx, s_wave[i]); mn = min(mn, s_wave[kWaves + i]); }
  __syncthreads();
}

// Visit every prefix position j < n once, as f(j, key): each thread takes kU
// positions per round, strided by the block size, all loaded before any is used
// (indices clamped, results masked) so a round's loads are in flight together.
constexpr int kU = 16;
template <typename Load, typename F>
__device__ __forceinline__ void for_each_key(int n, Load load, F f) {
  const int tid = threadIdx.x;
  for (int j0 = 0; j0 < n; j0 += kThreads * kU) {
    uint32_t k[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) k[u] = load(min(j0 + u * kThreads + tid, n - 1));
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int j = j0 + u * kThreads + tid;
      if (j < n) f(j, k[u]);
    }
  }
}

// LDS slot of prefix key j (of the cached prefix or of an emit tile): the low
// 4 bits are XORed with bits 6..9, so the emit's reads (thread t takes keys
// 16 t .. 16 t + 15) hit 64 different banks across a wave, while the
// counting passes' reads (64 consecutive keys per wave) stay conflict-free.
__device__ __forceinline__ int kslot(int j) { return j ^ ((j >> 6) & 15); }

template <bool CACHED>
__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
  const int g = blockIdx.x, b = blockIdx.y;
  const int L = a.L[b], w = a.w, pref = L - w;
  const int n_sel = a.n_keep[b] - w;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const float* sc = a.scores + bg * a.Lmax;
  int32_t* out = a.keep_idx + bg * a.Lmax;
  const int tid = threadIdx.x;

  // Each bin has kRep interleaved copies (lane % kRep picks one), so lanes of a
  // wave that hit the same bin mostly update different LDS banks.
  constexpr int kRep = CACHED ? 2 : 8;
  __shared__ uint32_t s_keys[CACHED ? kCacheN : kTileN];   // the prefix, or one emit tile
  __shared__ uint32_t hist[kBins * kRep];
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  __shared__ uint32_t s_digit, s_rank;

  for (int i = tid; i < w; i += kThreads) out[n_sel + i] = pref + i;
  if (n_sel <= 0) return;
  if (n_sel >= pref) {
    for (int j = tid; j < pref; j += kThreads) out[j] = j;
    return;
  }

  // 0. key range (and the LDS copy of the prefix)
  const auto from_hbm = [&](int j) { return key_of(sc[j]); };
  const auto from_lds = [&](int j) { return s_keys[kslot(j)]; };
  uint32_t kmax = 0u, kmin = 0xffffffffu;
  for_each_key(pref, from_hbm, [&](int j, uint32_t k) {
    if (CACHED) s_keys[kslot(j)] = k;
    kmax = max(kmax, k);
    kmin = min(kmin, k);
  });
  block_max_min(kmax, kmin, s_wave);          // ends with a barrier
  const uint32_t diff = kmax ^ kmin;
  // bits [0, lo) still to resolve; the keys share every bit above them, so
  // their common part is kmax's
  int lo = diff ? 32 - __clz(diff) : 1;
  uint32_t mask = lo >= 32 ? 0u : ~((1u << lo) - 1u);
  uint32_t prefix = kmax & mask;
  uint32_t rank = static_cast<uint32_t>(n_sel);

  // 1. radix select of the n_sel-th largest key among those matching prefix.
  while (lo > 0) {
    const int shift = max(lo - kBits, 0);
    const uint32_t dmask = (1u << (lo - shift)) - 1u;
    for (int i = tid; i < kBins * kRep; i += kThreads) hist[i] = 0u;
    __syncthreads();
    const uint32_t rep = tid % kRep;
    const auto count = [&](int, uint32_t k) {
      if ((k & mask) == prefix) atomicAdd(&hist[((k >> shift) & dmask) * kRep + rep], 1u);
    };
    if (CACHED) for_each_key(pref, from_lds, count);
    else        for_each_key(pref, from_hbm, count);
    __syncthreads();
    // thread t holds bins kBins-1-2t and kBins-2-2t (descending digit order)
    uint32_t c0 = 0u, c1 = 0u;
#pragma unroll
    for (int r = 0; r < kRep; ++r) {
      c0 += hist[(kBins - 1 - 2 * tid) * kRep + r];
      c1 += hist[(kBins - 2 - 2 * tid) * kRep + r];
    }
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(c0 + c1, s_wave, total);
    if (ex < rank && rank <= ex + c0 + c1) {
      if (ex + c0 >= rank) { s_digit = kBins - 1 - 2 * tid; s_rank = rank - ex; }
      else                 { s_digit = kBins - 2 - 2 * tid; s_rank = rank - ex - c0; }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    mask |= dmask << shift;
    rank = s_rank;
    lo = shift;
    __syncthreads();
  }
  const uint32_t tau = prefix;
  const uint32_t need_eq = rank;              // tau-valued positions to keep

  // 2. ordered emit.
  uint32_t gt_run = 0u, eq_run = 0u;
  for (int base = 0; base < pref; base += kTileN) {
    const uint32_t* tk = s_keys + (CACHED ? base : 0);
    if (!CACHED) {
      for_each_key(min(kTileN, pref - base), [&](int i) { return key_of(sc[base + i]); },
                   [&](int i, uint32_t k) { s_keys[kslot(i)] = k; });
      __syncthreads();
    }
    const int j0 = base + tid * kPer;
    uint32_t gt = 0u, eq = 0u, kk[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int j = j0 + q;
      const bool in = j < pref;
      kk[q] = in ? tk[kslot(tid * kPer + q)] : 0u;
      gt += (in && kk[q] > tau) ? 1u : 0u;
      eq += (in && kk[q] == tau) ? 1u : 0u;
    }
    uint32_t total;
    // counts per thread <= 16 and per tile <= 16384 fit the 16-bit halves
    const uint32_t ex = block_exclusive_scan(gt | (eq << 16), s_wave, total);
    uint32_t eq_before = eq_run + (ex >> 16);
    uint32_t pos = gt_run + (ex & 0xffffu) + min(eq_before, need_eq);
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int j = j0 + q;
      if (j < pref && kk[q] > tau) {
        out[pos++] = j;
      } else if (j < pref && kk[q] == tau) {
        if (eq_before < need_eq) out[pos++] = j;
        ++eq_before;
      }
    }
    gt_run += total & 0xffffu;
    eq_run += total >> 16;
  }
}

// ------------------------------------------------- several blocks per KV head
//
// The same selection split over C chunks of the prefix per (sequence, KV head)
// unit, for prefixes too long for one block to go through quickly.  Six
// launches over a (C, Hkv, B) grid; every block of a launch reads only what
// earlier launches wrote (stream order is the only synchronisation):
//   R   chunk key ranges;
//   H1  the radix state S0 from the ranges; the chunk's histogram of digit 1
//       (LDS) added into the unit's global histogram;
//   H2  S1 = S0 with digit 1 resolved from that histogram; histogram of digit 2;
//   H3  S2 = S1 with digit 2 resolved; histogram of digit 3;
//   CNT S3 = S2 with digit 3 resolved: tau and the tau-valued positions to
//       take; the chunk's counts of keys above and equal to tau;
//   EM  ordered emit, each chunk starting at the counts of the chunks before
//       it.
// Every block of a launch resolves the same state from the same histogram, so
// they agree; block 0 stores it for the next launch.  The radix state, digit
// width and tie rule are those of the one-block kernel, so both produce the
// same keep_idx.  Histograms rotate through three buffers: the one being read,
// the one being added into, and the one being cleared for the next launch.

constexpr int kWsRange = 0;                          // [kMaxChunks][2] max, min key
constexpr int kWsCnt = kWsRange + 2 * kSelMaxChunks; // [kMaxChunks][2] #gt, #eq tau
constexpr int kWsState = kWsCnt + 2 * kSelMaxChunks; // [2][4] prefix, mask, lo, rank
constexpr int kWsHist = kWsState + 8;                // [3][kBins]
static_assert(kWsHist + 3 * kBins == kSelWsWords, "select workspace layout");
constexpr int kPerM = 4;                             // positions per thread per emit tile
constexpr int kTileM = kThreads * kPerM;             // 4096
constexpr int kRepM = 4;                             // LDS histogram copies

struct Radix {
  uint32_t prefix, mask, rank;
  int lo;
};

struct Unit {
  int pref, n_sel, c0, c1;                            // chunk [c0, c1) of the prefix
  const float* sc;
  int32_t* out;
  uint32_t* ws;
  bool work;                                          // a radix search is needed
};

__device__ __forceinline__ Unit unit_of(const SelectArgs& a, uint32_t* ws, int C) {
  Unit u;
  const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  u.pref = a.L[b] - a.w;
  u.n_sel = a.n_keep[b] - a.w;
  const int per = ((u.pref + C - 1) / C + 63) & ~63;
  u.c0 = min(c * per, u.pref);
  u.c1 = min(u.c0 + per, u.pref);
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  u.sc = a.scores + bg * a.Lmax;
  u.out = a.keep_idx + bg * a.Lmax;
  u.ws = ws + bg * kSelWsWords;
  u.work = u.n_sel > 0 && u.n_sel < u.pref;
  return u;
}

// Keys of positions [c0, c1), kU per thread in flight, as for_each_key.
template <typename F>
__device__ __forceinline__ void for_each_chunk_key(const Unit& u, F f) {
  for_each_key(u.c1 - u.c0, [&](int i) { return key_of(u.sc[u.c0 + i]); },
               [&](int i, uint32_t k) { f(u.c0 + i, k); });
}

// Clear this block's share of histogram buffer `buf` (C divides kBins).
__device__ __forceinline__ void clear_hist_share(const Unit& u, int C, int buf) {
  const int n = kBins / C;
  uint32_t* h = u.ws + kWsHist + buf * kBins + blockIdx.x * n;
  for (int i = threadIdx.x; i < n; i += kThreads) h[i] = 0u;
}

// S0: the bits common to every prefix key, from the chunk ranges.
__device__ __forceinline__ Radix radix_from_ranges(const Unit& u, int C, uint32_t* s_wave) {
  const int lane = threadIdx.x & 63;
  if (threadIdx.x < 64) {
    uint32_t mx = 0u, mn = 0xffffffffu;
    if (lane < C) { mx = u.ws[kWsRange + 2 * lane]; mn = u.ws[kWsRange + 2 * lane + 1]; }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      mx = max(mx, static_cast<uint32_t>(__shfl_xor(mx, off)));
      mn = min(mn, static_cast<uint32_t>(__shfl_xor(mn, off)));
    }
    if (lane == 0) { s_wave[0] = mx; s_wave[1] = mn; }
  }
  __syncthreads();
  const uint32_t kmax = s_wave[0], diff = kmax ^ s_wave[1];
  __syncthreads();
  Radix r;
  r.lo = diff ? 32 - __clz(diff) : 1;
  r.mask = r.lo >= 32 ? 0u : ~((1u << r.lo) - 1u);
  r.prefix = kmax & r.mask;
  r.rank = static_cast<uint32_t>(u.n_sel);
  return r;
}

__device__ __forceinline__ Radix load_radix(const Unit& u, int slot) {
  const uint32_t* p = u.ws + kWsState + 4 * slot;
  Radix r;
  r.prefix = p[0];
  r.mask = p[1];
  r.lo = static_cast<int>(p[2]);
  r.rank = p[3];
  return r;
}

__device__ __forceinline__ void store_radix(const Unit& u, int slot, const Radix& r) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    uint32_t* p = u.ws + kWsState + 4 * slot;
    p[0] = r.prefix;
    p[1] = r.mask;
    p[2] = static_cast<uint32_t>(r.lo);
    p[3] = r.rank;
  }
}

// Resolve the next digit of r from the unit's global histogram `buf`.
__device__ __forceinline__ Radix radix_resolve(const Unit& u, Radix r, int buf, uint32_t* s_wave,
                                               uint32_t* s_dr) {
  if (r.lo <= 0) return r;
  const int tid = threadIdx.x;
  const int shift = max(r.lo - kBits, 0);
  const uint32_t dmask = (1u << (r.lo - shift)) - 1u;
  const uint32_t* h = u.ws + kWsHist + buf * kBins;
  const uint32_t c0 = h[kBins - 1 - 2 * tid], c1 = h[kBins - 2 - 2 * tid];
  uint32_t total;
  const uint32_t ex = block_exclusive_scan(c0 + c1, s_wave, total);
  if (ex < r.rank && r.rank <= ex + c0 + c1) {
    if (ex + c0 >= r.rank) { s_dr[0] = kBins - 1 - 2 * tid; s_dr[1] = r.rank - ex; }
    else                   { s_dr[0] = kBins - 2 - 2 * tid; s_dr[1] = r.rank - ex - c0; }
  }
  __syncthreads();
  r.prefix |= s_dr[0] << shift;
  r.mask |= dmask << shift;
  r.rank = s_dr[1];
  r.lo = shift;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void select_range_kernel(SelectArgs a, uint32_t* ws, int C) {
  const Unit u = unit_of(a, ws, C);
  if (!u.work) return;
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  uint32_t kmax = 0u, kmin = 0xffffffffu;
  for_each_chunk_key(u, [&](int, uint32_t k) {
    kmax = max(kmax, k);
    kmin = min(kmin, k);
  });
  block_max_min(kmax, kmin, s_wave);
  if (threadIdx.x == 0) {
    u.ws[kWsRange + 2 * blockIdx.x] = kmax;
    u.ws[kWsRange + 2 * blockIdx.x + 1] = kmin;
  }
  clear_hist_share(u, C, 1);
}

// Pass p = 1, 2, 3: state S(p-1), then the histogram of digit p into buffer p % 3.
__global__ __launch_bounds__(kThreads) void select_hist_kernel(SelectArgs a, uint32_t* ws, int C,
                                                               int p) {
  const Unit u = unit_of(a, ws, C);
  if (!u.work) return;
  __shared__ uint32_t hist[kBins * kRepM];
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  __shared__ uint32_t s_dr[2];
  const int tid = threadIdx.x;
  for (int i = tid; i < kBins * kRepM; i += kThreads) hist[i] = 0u;
  Radix r = p == 1 ? radix_from_ranges(u, C, s_wave)
                   : radix_resolve(u, load_radix(u, (p - 2) % 2), (p - 1) % 3, s_wave, s_dr);
  store_radix(u, (p - 1) % 2, r);
  clear_hist_share(u, C, (p + 1) % 3);
  if (r.lo <= 0) return;                      // every digit already resolved
  const int shift = max(r.lo - kBits, 0);
  const uint32_t dmask = (1u << (r.lo - shift)) - 1u;
  const uint32_t rep = tid % kRepM;
  __syncthreads();                            // hist cleared
  for_each_chunk_key(u, [&](int, uint32_t k) {
    if ((k & r.mask) == r.prefix) atomicAdd(&hist[((k >> shift) & dmask) * kRepM + rep], 1u);
  });
  __syncthreads();
  uint32_t* gh = u.ws + kWsHist + (p % 3) * kBins;
  for (int bin = tid; bin < kBins; bin += kThreads) {
    uint32_t v = 0u;
#pragma unroll
    for (int q = 0; q < kRepM; ++q) v += hist[bin * kRepM + q];
    if (v) __hip_atomic_fetch_add(gh + bin, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// S3 (tau, tau-valued positions to take), then the chunk's #gt / #eq counts.
__global__ __launch_bounds__(kThreads) void select_count_kernel(SelectArgs a, uint32_t* ws, int C) {
  const Unit u = unit_of(a, ws, C);
  if (!u.work) return;
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  __shared__ uint32_t s_dr[2];
  const Radix r = radix_resolve(u, load_radix(u, 0), 0, s_wave, s_dr);
  store_radix(u, 1, r);
  const uint32_t tau = r.prefix;
  uint32_t gt = 0u, eq = 0u;
  for_each_chunk_key(u, [&](int, uint32_t k) {
    gt += k > tau ? 1u : 0u;
    eq += k == tau ? 1u : 0u;
  });
  uint32_t tg, te;
  block_exclusive_scan(gt, s_wave, tg);
  block_exclusive_scan(eq, s_wave, te);
  if (threadIdx.x == 0) {
    u.ws[kWsCnt + 2 * blockIdx.x] = tg;
    u.ws[kWsCnt + 2 * blockIdx.x + 1] = te;
  }
}

__global__ __launch_bounds__(kThreads) void select_emit_kernel(SelectArgs a, uint32_t* ws, int C) {
  const Unit u = unit_of(a, ws, C);
  const int tid = threadIdx.x;
  if (blockIdx.x == 0)
    for (int i = tid; i < a.w; i += kThreads) u.out[u.n_sel + i] = u.pref + i;
  if (u.n_sel <= 0) return;
  if (u.n_sel >= u.pref) {
    for (int j = u.c0 + tid; j < u.c1; j += kThreads) u.out[j] = j;
    return;
  }
  __shared__ uint32_t s_keys[kTileM];
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  __shared__ uint32_t s_run[2];
  const Radix r = load_radix(u, 1);
  const uint32_t tau = r.prefix, need_eq = r.rank;
  if (tid < 64) {                             // counts of the chunks before this one
    const int lane = tid;
    uint32_t g = 0u, e = 0u;
    if (lane < static_cast<int>(blockIdx.x)) {
      g = u.ws[kWsCnt + 2 * lane];
      e = u.ws[kWsCnt + 2 * lane + 1];
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      g += __shfl_xor(g, off);
      e += __shfl_xor(e, off);
    }
    if (lane == 0) { s_run[0] = g; s_run[1] = e; }
  }
  __syncthreads();
  uint32_t gt_run = s_run[0], eq_run = s_run[1];
  for (int base = u.c0; base < u.c1; base += kTileM) {
    const int n = min(kTileM, u.c1 - base);
    for_each_key(n, [&](int i) { return key_of(u.sc[base + i]); },
                 [&](int i, uint32_t k) { s_keys[i] = k; });
    __syncthreads();
    uint32_t gt = 0u, eq = 0u, kk[kPerM];
#pragma unroll
    for (int q = 0; q < kPerM; ++q) {
      const int i = tid * kPerM + q;
      const bool in = i < n;
      kk[q] = in ? s_keys[i] : 0u;
      gt += (in && kk[q] > tau) ? 1u : 0u;
      eq += (in && kk[q] == tau) ? 1u : 0u;
    }
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(gt | (eq << 16), s_wave, total);
    uint32_t eq_before = eq_run + (ex >> 16);
    uint32_t pos = gt_run + (ex & 0xffffu) + min(eq_before, need_eq);
#pragma unroll
    for (int q = 0; q < kPerM; ++q) {
      const int i = tid * kPerM + q;
      if (i < n && kk[q] > tau) {
        u.out[pos++] = base + i;
      } else if (i < n && kk[q] == tau) {
        if (eq_before < need_eq) u.out[pos++] = base + i;
        ++eq_before;
      }
    }
    gt_run += total & 0xffffu;
    eq_run += total >> 16;
  }
}

}  // namespace

int select_chunks(int max_pref) {
  int c = 2;
  while (c < kSelMaxChunks && c * 4096 < max_pref) c *= 2;
  return c;
}

hipError_t launch_select_multi(const SelectArgs& a, void* ws, hipStream_t st) {
  int max_pref = 0;
  for (int b = 0; b < a.B; ++b) max_pref = max(max_pref, a.L[b] - a.w);
  const int C = select_chunks(max_pref);
  uint32_t* w = static_cast<uint32_t*>(ws);
  const dim3 grid(C, a.Hkv, a.B);
  select_range_kernel<<<grid, kThreads, 0, st>>>(a, w, C);
  for (int p = 1; p <= 3; ++p) select_hist_kernel<<<grid, kThreads, 0, st>>>(a, w, C, p);
  select_count_kernel<<<grid, kThreads, 0, st>>>(a, w, C);
  select_emit_kernel<<<grid, kThreads, 0, st>>>(a, w, C);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t st) {
  const dim3 grid(a.Hkv, a.B);
  int max_pref = 0;
  for (int b = 0; b < a.B; ++b) max_pref = max(max_pref, a.L[b] - a.w);
  if (max_pref <= kCacheN) select_kernel<true><<<grid, kThreads, 0, st>>>(a);
  else                     select_kernel<false><<<grid, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tb

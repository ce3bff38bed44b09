// Per-KV-head top-k of the pooled scores with lower-position tie-break,
// emitted as ascending kept positions followed by the window.
//
// One block of 1024 threads per (sequence, KV head).  Scores are >= 0, so
// their IEEE bit patterns order like the values; the selection is integer
// work and bit-exact:
//   1. radix select (4 passes of 8 bits, LDS histograms) finds the key tau of
//      the n_sel-th largest score and how many tau-valued positions to take;
//   2. an ordered emit walks the prefix in tiles of 4096 positions (4 per
//      thread, contiguous), with one block-wide exclusive scan of the packed
//      counts (greater-than-tau, equal-to-tau) per tile.  Positions equal to
//      tau are taken lowest index first, so a thread's output offset is
//      (#greater before it) + min(#equal before it, equal-needed).

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kPer = 4;                       // positions per thread per tile
constexpr int kTileN = kThreads * kPer;

__device__ __forceinline__ uint32_t key_of(float f) {
  return __float_as_uint(f) & 0x7fffffffu;    // scores are >= 0 (-0 -> 0)
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

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
  const int g = blockIdx.x, b = blockIdx.y;
  const int L = a.L[b], w = a.w, pref = L - w;
  const int n_sel = a.n_keep[b] - w;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const float* sc = a.scores + bg * a.Lmax;
  int32_t* out = a.keep_idx + bg * a.Lmax;
  const int tid = threadIdx.x;

  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  __shared__ uint32_t s_digit, s_rank;

  for (int i = tid; i < w; i += kThreads) out[n_sel + i] = pref + i;
  if (n_sel <= 0) return;
  if (n_sel >= pref) {
    for (int j = tid; j < pref; j += kThreads) out[j] = j;
    return;
  }

  // 1. radix select of the n_sel-th largest key.
  uint32_t prefix = 0u, mask = 0u, rank = static_cast<uint32_t>(n_sel);
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += kThreads) hist[i] = 0u;
    __syncthreads();
    for (int j = tid; j < pref; j += kThreads) {
      const uint32_t k = key_of(sc[j]);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane holds digits 255-4*lane .. 252-4*lane (descending)
      uint32_t cnt[4], local = 0u;
#pragma unroll
      for (int q = 0; q < 4; ++q) { cnt[q] = hist[255 - (4 * tid + q)]; local += cnt[q]; }
      uint32_t incl = local;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, off);
        if (tid >= off) incl += y;
      }
      const uint32_t excl = incl - local;
      if (excl < rank && rank <= incl) {
        uint32_t accum = excl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (accum + cnt[q] >= rank) {
            s_digit = 255u - static_cast<uint32_t>(4 * tid + q);
            s_rank = rank - accum;
            break;
          }
          accum += cnt[q];
        }
      }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    mask |= 255u << shift;
    rank = s_rank;
    __syncthreads();
  }
  const uint32_t tau = prefix;
  const uint32_t need_eq = rank;              // tau-valued positions to keep

  // 2. ordered emit.
  uint32_t gt_run = 0u, eq_run = 0u;
  for (int base = 0; base < pref; base += kTileN) {
    const int j0 = base + tid * kPer;
    uint32_t gt = 0u, eq = 0u, kk[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int j = j0 + q;
      kk[q] = (j < pref) ? key_of(sc[j]) : 0u;
      const bool in = j < pref;
      gt += (in && kk[q] > tau) ? 1u : 0u;
      eq += (in && kk[q] == tau) ? 1u : 0u;
    }
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(gt | (eq << 16), s_wave, total);
    uint32_t gt_before = gt_run + (ex & 0xffffu);
    uint32_t eq_before = eq_run + (ex >> 16);
    uint32_t pos = gt_before + min(eq_before, need_eq);
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int j = j0 + q;
      if (j >= pref) break;
      if (kk[q] > tau) {
        out[pos++] = j;
      } else if (kk[q] == tau) {
        if (eq_before < need_eq) out[pos++] = j;
        ++eq_before;
      }
    }
    gt_run += total & 0xffffu;
    eq_run += total >> 16;
  }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t st) {
  const dim3 grid(a.Hkv, a.B);
  select_kernel<<<grid, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tb

// Gather of the kept K/V rows into the compact caches.
//
// grid = (ceil(max n_keep / rows_per_block), Hkv, B), block = 256 threads.
// A row of d elements is split over d*elem/16 lanes, 16 bytes each, so each
// wave instruction moves whole contiguous rows; every thread issues all of its
// K and V loads before its stores to keep many requests in flight.  The
// kernel is pure data movement: HBM traffic is one read and one write of each
// kept row of K and V.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

constexpr int kThreads = 256;

template <int ROW_BYTES, int RPB>
__global__ __launch_bounds__(kThreads) void compact_kernel(CompactArgs a) {
  constexpr int LPR = ROW_BYTES / 16;              // lanes per row
  constexpr int ROWS_PER_PASS = kThreads / LPR;
  constexpr int PASSES = RPB / ROWS_PER_PASS;
  const int g = blockIdx.y, b = blockIdx.z;
  const int n = a.n_keep[b];
  const int i0 = blockIdx.x * RPB;
  if (blockIdx.x == 0 && g == 0 && threadIdx.x == 0) a.kv_len[b] = n;
  if (i0 >= n) return;
  const int part = threadIdx.x % LPR, r0 = threadIdx.x / LPR;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const int32_t* keep = a.keep_idx + bg * a.Lmax;
  const char* ks = static_cast<const char*>(a.k) + bg * a.Lmax * ROW_BYTES + part * 16;
  const char* vs = static_cast<const char*>(a.v) + bg * a.Lmax * ROW_BYTES + part * 16;
  char* kd = static_cast<char*>(a.k_cache) + bg * a.cap * ROW_BYTES + part * 16;
  char* vd = static_cast<char*>(a.v_cache) + bg * a.cap * ROW_BYTES + part * 16;
  uint4 kr[PASSES], vr[PASSES];
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int i = i0 + r0 + p * ROWS_PER_PASS;
    if (i < n) {
      // indices are clamped into the prompt so a bad index cannot fault
      const int j = min(max(keep[i], 0), a.Lmax - 1);
      const size_t src = static_cast<size_t>(j) * ROW_BYTES;
      kr[p] = ldg16(ks + src);
      vr[p] = ldg16(vs + src);
    }
  }
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int i = i0 + r0 + p * ROWS_PER_PASS;
    if (i < n) {
      const size_t dst = static_cast<size_t>(i) * ROW_BYTES;
      stg16(kd + dst, kr[p]);
      stg16(vd + dst, vr[p]);
    }
  }
}

template <int ROW_BYTES>
hipError_t launch_rb(const CompactArgs& a, int max_keep, hipStream_t st) {
  constexpr int RPB = 64;
  const dim3 grid((max_keep + RPB - 1) / RPB, a.Hkv, a.B);
  compact_kernel<ROW_BYTES, RPB><<<grid, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int d, int elem_bytes, int max_keep,
                          hipStream_t st) {
  switch (d * elem_bytes) {
    case 128: return launch_rb<128>(a, max_keep, st);
    case 256: return launch_rb<256>(a, max_keep, st);
    case 512: return launch_rb<512>(a, max_keep, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tb

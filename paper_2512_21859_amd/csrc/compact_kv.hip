// Gather of the kept K/V rows into the compact caches.
//
// grid = (ceil(max n_keep / 32), Hkv, B), block = 256 threads; block t fills
// destination rows [32t, 32t + 32) of one (sequence, KV head), i.e. one
// 32-row tile of the contiguous cache or one page of a paged cache.  K and V
// rows are both copied row-major: each row is split into 16-byte pieces, one
// per lane, so a wave instruction moves whole contiguous rows.  Rows past
// n_keep are not written.  All loads of a thread are issued before its
// stores.  HBM traffic is one read and one write of each kept row of K and V.
// The cache writes are streaming (non-temporal) stores: measured at
// L = 131072, 8 KV heads, half the rows kept, 80 us against 104 us with
// ordinary stores (6.7 against 5.2 TB/s); non-temporal loads of the gathered
// rows did not help.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

constexpr int kThreads = 256;
constexpr int kVT = kVTile;

template <typename T, int D, bool PAGED>
__global__ __launch_bounds__(kThreads) void compact_kernel(CompactArgs a) {
  constexpr int ROW_BYTES = D * sizeof(T);
  constexpr int LPR = ROW_BYTES / 16;                 // lanes per row
  constexpr int ROWS_PER_PASS = kThreads / LPR;
  constexpr int PASSES = kVT / ROWS_PER_PASS;
  static_assert(PASSES >= 1 && kVT % ROWS_PER_PASS == 0, "tile shape");
  const int tile = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int n = a.n_keep[b];
  const int i0 = tile * kVT;
  if (tile == 0 && g == 0 && threadIdx.x == 0) a.kv_len[b] = n;
  if (i0 >= n) return;
  const int part = threadIdx.x % LPR, r0 = threadIdx.x / LPR;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const int32_t* keep = a.keep_idx + bg * a.Lmax;
  const char* ks = static_cast<const char*>(a.k) + bg * a.Lmax * ROW_BYTES + part * 16;
  const char* vs = static_cast<const char*>(a.v) + bg * a.Lmax * ROW_BYTES + part * 16;
  const size_t off = cache_tile_off<PAGED>(a, b, g, tile, D);   // element offset of the tile
  char* kd = static_cast<char*>(a.k_cache) + off * sizeof(T) + part * 16;   // tile row 0
  char* vd = static_cast<char*>(a.v_cache) + off * sizeof(T) + part * 16;

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
    const int rr = r0 + p * ROWS_PER_PASS;
    if (i0 + rr < n) {
      stg16_stream(kd + static_cast<size_t>(rr) * ROW_BYTES, kr[p]);
      stg16_stream(vd + static_cast<size_t>(rr) * ROW_BYTES, vr[p]);
    }
  }
}

template <typename T, int D>
hipError_t launch_t(const CompactArgs& a, int max_keep, hipStream_t st) {
  const dim3 grid((max_keep + kVT - 1) / kVT, a.Hkv, a.B);
  if (a.table) compact_kernel<T, D, true><<<grid, kThreads, 0, st>>>(a);
  else         compact_kernel<T, D, false><<<grid, kThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int d, int elem_bytes, int max_keep,
                          hipStream_t st) {
  if (elem_bytes == 2) return d == 128 ? launch_t<uint16_t, 128>(a, max_keep, st)
                                       : launch_t<uint16_t, 64>(a, max_keep, st);
  return d == 128 ? launch_t<float, 128>(a, max_keep, st) : launch_t<float, 64>(a, max_keep, st);
}

}  // namespace tb

// Bandwidth probe for the benchmark (not part of the timebill library): a
// streaming read of a device buffer, the practical HBM read ceiling that the
// decode and compaction rates are compared with.  Each thread reads 16-byte
// vectors in a grid-stride loop with several loads in flight and folds them
// into one word, which the block writes once so the loads cannot be removed.

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kThreads = 256;
constexpr int kUnroll = 8;                   // 16-byte loads in flight per thread

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ p,
                                                               size_t n, unsigned* sink) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kThreads;
  size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x;
  unsigned acc = 0;
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n; i += stride) {
    const u32x4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  __shared__ unsigned s[kThreads];
  s[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned a = 0;
    for (int t = 0; t < kThreads; ++t) a ^= s[t];
    sink[blockIdx.x] = a;
  }
}

}  // namespace

extern "C" __attribute__((visibility("default")))
int tbb_stream_read(const void* p, size_t bytes, unsigned* sink, int blocks, hipStream_t stream) {
  if (!p || !sink || blocks < 1 || bytes % 16 != 0) return 1;
  stream_read_kernel<<<blocks, kThreads, 0, stream>>>(static_cast<const u32x4*>(p), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

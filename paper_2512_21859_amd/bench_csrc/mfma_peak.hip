// Matrix-core throughput probe for the benchmark (not part of the timebill
// library): the practical float64 and bf16 matrix-instruction rates that the
// scoring and prefill kernels are compared with, beside the datasheet peaks.
// Every wave runs `iters` rounds of eight independent accumulation chains of
// one instruction shape on register operands only (no memory traffic in the
// loop); each thread writes one folded value so the products cannot be
// removed.  Flops per instruction: 16 * 16 * 4 * 2 (float64 16x16x4) and
// 16 * 16 * 32 * 2 (bf16 16x16x32).

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef __attribute__((ext_vector_type(4))) double f64x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

constexpr int kThreads = 256;
constexpr int kChains = 8;

__global__ __launch_bounds__(kThreads, 4) void mfma_f64_kernel(int iters, double* sink) {
  const double a = 1.0 + 1e-3 * (threadIdx.x & 63), b = 1e-6;
  f64x4 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[c], 0, 0, 0);
  }
  double s = 0.0;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  sink[static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kThreads, 4) void mfma_bf16_kernel(int iters, double* sink) {
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = static_cast<__bf16>(1.0f + 0.01f * e);
    b[e] = static_cast<__bf16>(1e-4f * (threadIdx.x & 7));
  }
  f32x4 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  sink[static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x] = s;
}

}  // namespace

// kind 0: float64 16x16x4, kind 1: bf16 16x16x32.  `sink` holds blocks * 256
// doubles.  Instructions issued: blocks * 4 waves * iters * 8.
extern "C" __attribute__((visibility("default")))
int tbb_mfma_peak(int kind, int blocks, int iters, double* sink, hipStream_t stream) {
  if (!sink || blocks < 1 || iters < 1 || (kind != 0 && kind != 1)) return 1;
  if (kind == 0) mfma_f64_kernel<<<blocks, kThreads, 0, stream>>>(iters, sink);
  else           mfma_bf16_kernel<<<blocks, kThreads, 0, stream>>>(iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// KNorm scoring: a prefix key scores minus its L2 norm, so the selection that
// keeps the largest scores keeps the smallest norms (the norm-based scorer the
// paper's fixed-ratio baselines cite, Sec. 6.1).
//
// One pass over K, HBM-bound (d * s_e bytes read and 4 bytes written per
// prefix position).  A row is read by d/8 lanes, 8 elements each (16-byte
// loads for bf16); squares of the exact inputs are summed in float64 and the
// lanes of a row are combined by DPP in a fixed order, so the norm is correct
// to the final fp32 rounding.  Each wave takes 4 row groups per round, loaded
// together.

#include "common.h"
#include "kernels.h"

namespace tb {
namespace {

constexpr int kThreads = 256;
constexpr int kRounds = 4;           // row groups per wave per round

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

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void knorm_kernel(KnormArgs a) {
  constexpr int LPR = D / 8;                 // lanes per row (16 or 8)
  constexpr int RPW = 64 / LPR;              // rows per wave per row group
  constexpr int RPB = (kThreads / 64) * RPW * kRounds;   // rows per block per round
  const int g = blockIdx.y, b = blockIdx.z;
  const int pref = a.L[b] - a.w;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LPR, rw = lane / LPR;
  const size_t bg = static_cast<size_t>(b) * a.Hkv + g;
  const T* kh = static_cast<const T*>(a.k) + bg * a.Lmax * D;
  float* out = a.scores + bg * a.Lmax;

  for (int base = blockIdx.x * RPB; base < pref; base += gridDim.x * RPB) {
    float x[kRounds][8];
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {      // unconditional loads of clamped rows
      const int row = base + (r * (kThreads / 64) + wave) * RPW + rw;
      load8<T>(kh + static_cast<size_t>(min(row, pref - 1)) * D + 8 * sub, x[r]);
    }
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const int row = base + (r * (kThreads / 64) + wave) * RPW + rw;
      double s = 0.0;
#pragma unroll
      for (int e = 0; e < 8; ++e) s = fma(static_cast<double>(x[r][e]), static_cast<double>(x[r][e]), s);
      s += dpp_f64<kDppQuadXor1>(s);
      s += dpp_f64<kDppQuadXor2>(s);
      s += dpp_f64<kDppRowHalfMirror>(s);
      if (LPR == 16) s += dpp_f64<kDppRowMirror>(s);
      if (sub == 0 && row < pref) out[row] = static_cast<float>(-sqrt(s));
    }
  }
}

}  // namespace

hipError_t launch_knorm(const KnormArgs& a, int d, bool bf16, hipStream_t st) {
  int max_pref = 0;
  for (int b = 0; b < a.B; ++b) max_pref = max(max_pref, a.L[b] - a.w);
  const int rows_per_block = (kThreads / 64) * (64 / (d / 8)) * kRounds;
  // a few rounds per block; enough blocks for every CU
  const int bx = max(1, min((max_pref + 4 * rows_per_block - 1) / (4 * rows_per_block), 2048));
  const dim3 grid(bx, a.Hkv, a.B);
  if (bf16) {
    if (d == 128) knorm_kernel<bf16_t, 128><<<grid, kThreads, 0, st>>>(a);
    else          knorm_kernel<bf16_t, 64><<<grid, kThreads, 0, st>>>(a);
  } else {
    if (d == 128) knorm_kernel<float, 128><<<grid, kThreads, 0, st>>>(a);
    else          knorm_kernel<float, 64><<<grid, kThreads, 0, st>>>(a);
  }
  return hipGetLastError();
}

}  // namespace tb

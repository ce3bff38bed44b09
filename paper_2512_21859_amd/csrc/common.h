// Shared device helpers for the gfx950 kernels: element types, bf16
// conversion, DPP row reductions and launch-argument structs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tb {

// bf16 is carried as its raw 16-bit pattern.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round-to-nearest-even fp32 -> bf16 (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Element traits: how many elements a 16-byte vector holds and how to widen.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kPer16B = 4;
  __device__ __forceinline__ static void widen(const uint4& v, float* out) {
    out[0] = __uint_as_float(v.x); out[1] = __uint_as_float(v.y);
    out[2] = __uint_as_float(v.z); out[3] = __uint_as_float(v.w);
  }
  __device__ __forceinline__ static float load1(const float* p) { return *p; }
  __device__ __forceinline__ static void store1(float* p, float x) { *p = x; }
};
template <> struct Elem<bf16_t> {
  static constexpr int kPer16B = 8;
  __device__ __forceinline__ static void widen(const uint4& v, float* out) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = __uint_as_float(w[i] << 16);
      out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ static float load1(const bf16_t* p) { return bf16_to_f32(p->bits); }
  __device__ __forceinline__ static void store1(bf16_t* p, float x) { p->bits = f32_to_bf16(x); }
};

// DPP controls (gfx9): quad permutes and row mirrors within 16-lane rows.
constexpr int kDppQuadXor1 = 0xB1;   // [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;   // [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a DPP row; every lane of the row gets the total.
// The order of additions is fixed, so the result is deterministic.
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f32<kDppQuadXor1>(x);
  x += dpp_f32<kDppQuadXor2>(x);
  x += dpp_f32<kDppRowHalfMirror>(x);
  x += dpp_f32<kDppRowMirror>(x);
  return x;
}

__device__ __forceinline__ uint4 ldg16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}
// Streaming (non-temporal) 16-byte store: for outputs written once and not
// read back soon, so they do not displace cached data on their way to HBM.
__device__ __forceinline__ void stg16_stream(void* p, const uint4& v) {
  typedef unsigned int u32x4n __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4n, v), static_cast<u32x4n*>(p));
}

}  // namespace tb

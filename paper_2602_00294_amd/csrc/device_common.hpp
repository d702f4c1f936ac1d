// Small device helpers shared by the HIP kernels of this library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sata {

// bfloat16 storage type: the upper 16 bits of an IEEE binary32.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float((uint32_t)x.bits << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  bf16_t r;
  if ((u & 0x7fffffffu) > 0x7f800000u) {
    r.bits = (uint16_t)((u >> 16) | 0x40);
  } else {
    u += 0x7fffu + ((u >> 16) & 1u);
    r.bits = (uint16_t)(u >> 16);
  }
  return r;
}

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f32_to_bf16(x); }

// Value of one monomial feature from its packed table entry: byte j (< 7) is
// index i_{j+1}, byte 7 the degree p.  x points at the row's coordinates.
__device__ __forceinline__ float feature_value(uint64_t pk, float w, const float* x) {
  const int p = (int)(pk >> 56);
  float r = w;
  for (int j = 0; j < p; ++j) r *= x[(pk >> (8 * j)) & 0xff];
  return r;
}

// Truncated exponential series f_P(s) = sum_{p<P} s^p/p!, Horner form.
__device__ __forceinline__ float taylor_horner(float s, int P) {
  float r = 1.0f;
  for (int p = P - 1; p >= 1; --p) r = 1.0f + r * s * (1.0f / (float)p);
  return r;
}

}  // namespace sata

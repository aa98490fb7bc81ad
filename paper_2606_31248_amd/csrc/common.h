// Internal helpers shared by the HIP kernels of libstrata (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "strata.h"

namespace strata {

// ---- bfloat16 storage -------------------------------------------------------
// bf16 values are kept as their 16-bit patterns; widening is exact.
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float32 -> bfloat16 with round-to-nearest-even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Two floats -> packed pair of bf16 (low half = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
}

// ---- border-clamped neighbourhood window (NATTEN rule, dilation 1) ---------
__device__ __forceinline__ int win_start(int i, int L, int k) {
  int s = i - (k >> 1);
  s = s < 0 ? 0 : s;
  return s > L - k ? L - k : s;
}

}  // namespace strata

// ---- error reporting inside the library -------------------------------------
namespace strata {
strata_status set_error(strata_status st, const char* fmt, ...);
strata_status check_launch(const char* what);
}  // namespace strata

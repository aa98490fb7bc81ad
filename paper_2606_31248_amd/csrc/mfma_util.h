// Device helpers shared by the MFMA neighbourhood-attention kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace strata {
namespace mfma {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2 f = {a, b};
  bf16x2 h = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// Two floats -> packed float16 pair (nearest-even), saturating at +-65504.
__device__ __forceinline__ uint32_t pack2h(float a, float b) {
  f32x2 f = {__builtin_amdgcn_fmed3f(a, -65504.f, 65504.f), __builtin_amdgcn_fmed3f(b, -65504.f, 65504.f)};
  f16x2 h = __builtin_convertvector(f, f16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// Two floats -> packed float16 pair, round to nearest even, no saturation (the
// caller keeps the values inside the float16 range).
__device__ __forceinline__ uint32_t pack2h_rne(float a, float b) {
  f16x2 h = __builtin_convertvector((f32x2{a, b}), f16x2);
  return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Rotate 4 pairs held as 4 packed bf16x2 words by phases (c0,s0,c1,s1),(c2,s2,c3,s3),
// multiply by `mul`, and return them as 4 packed float16x2 words.
__device__ __forceinline__ uint4 rotate8h(uint4 x, float4 p01, float4 p23, float mul) {
  uint32_t w[4] = {x.x, x.y, x.z, x.w};
  float cs_[8] = {p01.x, p01.y, p01.z, p01.w, p23.x, p23.y, p23.z, p23.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float a = lo_bf16(w[t]), b = hi_bf16(w[t]);
    float c = cs_[2 * t], s = cs_[2 * t + 1];
    r[t] = pack2h(fmaf(a, c, -b * s) * mul, fmaf(a, s, b * c) * mul);
  }
  return make_uint4(r[0], r[1], r[2], r[3]);
}

// Rotate 4 pairs held as packed bf16x2 words by float16 phases (c, s) in
// packed float16 arithmetic (one multiply and one fused multiply-add per pair);
// returns packed float16x2 words.  The inputs, times `mul` in float32, are
// clamped to +-46000 so that no rotated value leaves the float16 range.
__device__ __forceinline__ uint4 rotate8h_pk(uint4 x, uint4 ph, float mul = 1.f) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  const uint32_t p[4] = {ph.x, ph.y, ph.z, ph.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const float a = __builtin_amdgcn_fmed3f(lo_bf16(w[t]) * mul, -46000.f, 46000.f);
    const float b = __builtin_amdgcn_fmed3f(hi_bf16(w[t]) * mul, -46000.f, 46000.f);
    const f16x2 ab = __builtin_convertvector((f32x2{a, b}), f16x2);
    const f16x2 cs = __builtin_bit_cast(f16x2, p[t]);
    const f16x2 aa = {ab.x, ab.x}, bb = {ab.y, ab.y}, ns = {-cs.y, cs.x};
    r[t] = __builtin_bit_cast(uint32_t, aa * cs + bb * ns);  // (a c - b s, a s + b c)
  }
  return make_uint4(r[0], r[1], r[2], r[3]);
}

// bf16 x 8 -> float16 x 8 by round-toward-zero: exact for bf16 values whose
// magnitude lies in float16's normal range, saturating at +-65504 above it;
// smaller values keep float16's subnormal spacing 2^-24.
__device__ __forceinline__ uint4 bf16x8_to_f16x8(uint4 x) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) r[t] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo_bf16(w[t]), hi_bf16(w[t])));
  return make_uint4(r[0], r[1], r[2], r[3]);
}

// bf16 x 8 -> float16 x 8, times `mul` (no rotation).
__device__ __forceinline__ uint4 scale8h(uint4 x, float mul) {
  uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) r[t] = pack2h(lo_bf16(w[t]) * mul, hi_bf16(w[t]) * mul);
  return make_uint4(r[0], r[1], r[2], r[3]);
}

__device__ __forceinline__ i16x4 tr_read(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
}

__device__ __forceinline__ uint4 ld16(const char* p) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void st16(char* p, uint4 v) {
  *reinterpret_cast<u32x4*>(p) = u32x4{v.x, v.y, v.z, v.w};
}

// Direct global -> LDS copy of 16 bytes per lane: lane i of the wave writes
// wave_dst + 16 i (wave_dst must be the same for the whole wave).
__device__ __forceinline__ void copy16_to_lds(const uint16_t* src, char* wave_dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_void*)wave_dst, 16, 0, 0);
}

// Cross-row exchanges without LDS (gfx950 v_permlane16/32_swap): with both
// operands equal, the two results of a swap are, in some order, the lane's own
// value and the value of lane l^16 (resp. l^32).
__device__ __forceinline__ float max_over_rows(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float sum_over_rows(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sum of squares of the 8 bf16 values of a 16-byte piece, added to acc (the
// products are exact in float32).
__device__ __forceinline__ float sumsq8(uint4 x, float acc) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int t = 0; t < 4; ++t)
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[t]), __builtin_bit_cast(bf16x2, w[t]), acc,
                                          false);
  return acc;
}

// Sum over each aligned group of 8 consecutive lanes (every lane of the group
// active): two quad permutations, then the mirror inside each half row.
__device__ __forceinline__ float sum_over_8_lanes(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));  // row_half_mirror
  return x;
}

// Sum over each aligned group of 16 consecutive lanes (a row; every lane of it
// active): the 8-lane sums, then the mirror across the row pairs the halves.
__device__ __forceinline__ float sum_over_16_lanes(float x) {
  x = sum_over_8_lanes(x);
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));  // row_mirror
  return x;
}

// Logistic sigmoid 1 / (1 + e^-g) of the output gate (hardware exp2 and
// reciprocal; 0 and 1 at the extremes).
__device__ __forceinline__ float sigmoid_fast(float g) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * g));
}

// Output-gate factors of 4 consecutive channels held as 4 bf16 in a uint2.
__device__ __forceinline__ f32x4 sigmoid4_bf16(uint2 g) {
  return f32x4{sigmoid_fast(lo_bf16(g.x)), sigmoid_fast(hi_bf16(g.x)), sigmoid_fast(lo_bf16(g.y)),
               sigmoid_fast(hi_bf16(g.y))};
}

__device__ __forceinline__ float psum8(uint32_t a, uint32_t b, float acc) {
  const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3F803F80u);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), one, acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, b), one, acc, false);
}

}  // namespace mfma
}  // namespace strata

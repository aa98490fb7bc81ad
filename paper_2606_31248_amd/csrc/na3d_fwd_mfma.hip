// MFMA neighbourhood-attention forward for gfx950 (bf16 in/out, head_dim 64).
//
// Work decomposition
//   workgroup : one (tile, head), an 8 x 8 block of (y, x) query positions and
//               ZQ query levels; 8 waves, one workgroup per CU.
//   wave      : a 4 x 4 (y, x) sub-block = 16 queries, on ZQ/2 of the levels
//               (waves 0-3 take the even levels of the block, waves 4-7 the odd
//               ones, so both halves have work at every key level).
//   key sweep : the workgroup walks the key levels its queries need, each once.
//               K and V of the (8+ky-1) x (8+kx-1) key box of a level are copied
//               global -> LDS by the direct-to-LDS load (no registers), one level
//               ahead of the compute, into a double buffer; each thread then
//               rotates the K pieces its own copies brought (StereoRoPE) and
//               rounds them to float16, and one barrier publishes the level.
//
// Per (query level, key level) a wave multiplies the keys of its 4x4 sub-block's
// box -- (3+ky) x (3+kx) keys, in 16-key chunks -- with its 16 queries:
//   S^T (16 keys x 16 queries) = K . Q^T     v_mfma_f32_16x16x32_f16, the
//                                           accumulator seeded with the window
//                                           mask (0 or -inf),
//   online softmax on S^T in registers (a lane owns one query column); the
//   running maximum only moves when it grows by more than 2^8, so most steps
//   rescale nothing; cross-row maxima use v_permlane16/32_swap,
//   O^T (64 d x 16 queries) += V^T . P^T    bf16 MFMA; V^T fragments come from
//                                           the row-major V tile through the LDS
//                                           transpose read, P^T is the S^T
//                                           accumulator packed to bf16 in place;
//   row sums of the packed P with v_dot2c_f32_bf16 (the same rounded weights the
//   P.V product uses).
// The rotated Q and K are rounded to float16, not bf16, for the Q.K^T contraction
// (same MFMA rate): bf16 rounding of the rotated operands alone costs up to ~0.5%
// of an output, beyond the parity bound; float16 keeps it near 0.05%.  Rotated
// values beyond the float16 range (|x| > 65504) saturate.  P and V stay bf16.
// The logit scale and log2(e) are folded into Q so the softmax uses exp2.
//
// K rows are 128 bytes with their 16-byte columns XOR-swizzled by
// ((x >> 1) + 5 y) & 7 of the key's box position: the 16 keys of any chunk of an
// interior sub-block then sit in 16 distinct bank groups.  V rows are padded to
// 160 bytes, which spreads the 8-byte transpose reads and lets them take
// immediate offsets.  The two halves of the double buffer are distinct LDS objects, so the
// compiler can tell the reads of one from the copies into the other and does not
// wait for the copies before reading.
#include "common.h"
#include "kernels.h"

namespace strata {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kBY = 8, kBX = 8;  // query block of a workgroup (y, x)
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kD = 64;           // head_dim
constexpr int kKRow = 128;       // LDS bytes per key row of K (16-byte columns swizzled)
constexpr int kVRow = 160;       // LDS bytes per key row of V (128 + 32 pad)
constexpr int kLdsMax = 160 * 1024;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLazy = 8.0f;    // rescale only when the maximum grows by > 2^8

template <int KZ, int KY, int KX, int ZQ>
struct Cfg {
  static constexpr int LY = kBY + KY - 1, LX = kBX + KX - 1;  // staged key box per level
  static constexpr int NUY = 3 + KY, NUX = 3 + KX;            // key box of one 4x4 sub-block
  static constexpr int NU = NUY * NUX;
  static constexpr int NC = (NU + 15) / 16;                   // 16-key chunks
  static constexpr int NS = (NC + 1) / 2;                     // 32-key PV steps
  static constexpr int KEYS = LY * LX;
  static constexpr int KSLOTS = KEYS * (kKRow / 16);          // 16-byte slots of a K tile (8 per key)
  static constexpr int VSLOTS = KEYS * (kVRow / 16);
  static constexpr int KBYTES = KEYS * kKRow, VBYTES = KEYS * kVRow;
  static constexpr int BUF = KBYTES + VBYTES;                 // one level: K and V
  static constexpr int ITK = (KSLOTS + kThreads - 1) / kThreads;
  static constexpr int ITV = (VSLOTS + kThreads - 1) / kThreads;
  // per-thread copy offsets live in LDS when they fit, else in registers; the
  // rotary phases of the key box (float16 pairs, one 16-byte slot per K slot)
  // too, else they are read from memory for every key level
  static constexpr int GOFF_BYTES = (ITK + ITV) * kThreads * 4;
  static constexpr bool GOFF_LDS = 2 * BUF + GOFF_BYTES <= kLdsMax;
  static constexpr int PH_BYTES = KSLOTS * 16;
  static constexpr bool PH_LDS = GOFF_LDS && 2 * BUF + GOFF_BYTES + PH_BYTES <= kLdsMax;
  static constexpr int QL = ZQ / 2;                           // query levels per wave
  static_assert(ZQ % 2 == 0, "ZQ must be even");
  static_assert(2 * BUF <= kLdsMax, "key tiles exceed LDS");
};

struct Args {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;   // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  uint16_t* out;
  float* lse;
  int heads, Z, H, W;
  int n_zb, n_yb, n_xb;
  float qscale;       // scale * log2(e)
};

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
// returns packed float16x2 words.  Inputs are clamped to +-46000 so that no
// rotated value leaves the float16 range.
__device__ __forceinline__ uint4 rotate8h_pk(uint4 x, uint4 ph) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  const uint32_t p[4] = {ph.x, ph.y, ph.z, ph.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const float a = __builtin_amdgcn_fmed3f(lo_bf16(w[t]), -46000.f, 46000.f);
    const float b = __builtin_amdgcn_fmed3f(hi_bf16(w[t]), -46000.f, 46000.f);
    const f16x2 ab = __builtin_convertvector((f32x2{a, b}), f16x2);
    const f16x2 cs = __builtin_bit_cast(f16x2, p[t]);
    const f16x2 aa = {ab.x, ab.x}, bb = {ab.y, ab.y}, ns = {-cs.y, cs.x};
    r[t] = __builtin_bit_cast(uint32_t, aa * cs + bb * ns);  // (a c - b s, a s + b c)
  }
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

__device__ __forceinline__ float psum8(uint32_t a, uint32_t b, float acc) {
  const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3F803F80u);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), one, acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, b), one, acc, false);
}

template <int KZ, int KY, int KX, int ZQ>
__global__ void __launch_bounds__(kThreads, 1) na3d_fwd_mfma_kernel(Args a) {
  using C = Cfg<KZ, KY, KX, ZQ>;
  // double buffer of key tiles (distinct objects, see above), copy offsets, phases
  __shared__ __attribute__((aligned(16))) char tK0[C::KBYTES];
  __shared__ __attribute__((aligned(16))) char tV0[C::VBYTES];
  __shared__ __attribute__((aligned(16))) char tK1[C::KBYTES];
  __shared__ __attribute__((aligned(16))) char tV1[C::VBYTES];
  __shared__ __attribute__((aligned(16))) int sgoff[C::GOFF_LDS ? C::GOFF_BYTES / 4 : 1];
  __shared__ __attribute__((aligned(16))) char sph[C::PH_LDS ? C::PH_BYTES : 16];

  // ---- block coordinates (XCD-aware: neighbouring blocks share an L2) -------
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int xb = bid % a.n_xb;
  const int yb = (bid / a.n_xb) % a.n_yb;
  const int zb = (bid / (a.n_xb * a.n_yb)) % a.n_zb;
  const int bh = bid / (a.n_xb * a.n_yb * a.n_zb);
  const int b = bh / a.heads;
  const int H = a.H, W = a.W, Z = a.Z;
  const int by0 = yb * kBY, bx0 = xb * kBX, z0 = zb * ZQ;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;
  const int sb = wave & 3, grp = wave >> 2;  // xy sub-block, level parity

  // staged key box of the workgroup, and the key box of this wave's sub-block
  const int ty0 = win_start(min(by0, H - 1), H, KY);
  const int tx0 = win_start(min(bx0, W - 1), W, KX);
  const int sy0 = by0 + 4 * (sb >> 1), sx0 = bx0 + 4 * (sb & 1);
  const int uy0 = win_start(min(sy0, H - 1), H, KY);
  const int ux0 = win_start(min(sx0, W - 1), W, KX);
  // this lane's query column (clamped into the grid; stores are masked later)
  const int qy_raw = sy0 + (qn >> 2), qx_raw = sx0 + (qn & 3);
  const int qy = min(qy_raw, H - 1), qx = min(qx_raw, W - 1);
  const int wys = win_start(qy, H, KY), wxs = win_start(qx, W, KX);

  // column swizzle of the K tile (see the header comment)
  auto kswz = [&](int key) { return ((key % C::LX >> 1) + 5 * (key / C::LX)) & 7; };

  // ---- per-lane tile offsets and window mask, identical for every key level ----
  uint32_t kaddr[C::NC], vaddr[C::NC];
  f32x4 bias[C::NC];
#pragma unroll
  for (int c = 0; c < C::NC; ++c) {
    {  // K fragment (A operand): row = key 16c + qn, 16 bytes at column g (xor 64 bytes: g+4)
      int u = 16 * c + qn;
      int key = 0;
      if (u < C::NU) key = (uy0 - ty0 + u / C::NUX) * C::LX + (ux0 - tx0 + u % C::NUX);
      kaddr[c] = key * kKRow + ((g ^ kswz(key)) << 4);
    }
    {  // V^T fragment by transpose read: source row = key 16c + 4g + qn/4, element 4*(qn%4)
      int u = 16 * c + 4 * g + (qn >> 2);
      int key = 0;
      if (u < C::NU) key = (uy0 - ty0 + u / C::NUX) * C::LX + (ux0 - tx0 + u % C::NUX);
      vaddr[c] = key * kVRow + (qn & 3) * 8;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int u = 16 * c + 4 * g + i;
      int ky = uy0 + u / C::NUX, kx = ux0 + u % C::NUX;
      bool ok = u < C::NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX;
      bias[c][i] = ok ? 0.f : -INFINITY;
    }
  }

  // ---- direct-to-LDS copy map: slot s = it*512 + tid of a tile ---------------
  // K: 8 slots per key, slot column c holds data column c ^ swizzle(key);
  // V: 10 slots per key (8 data + 2 pad).
  // goff: element offset inside a key level, or -1 for pad / past-the-end slots.
  // Each thread only reads back its own offsets: no barrier needed.
  const int64_t HW = (int64_t)H * W;
  int goffK_r[C::GOFF_LDS ? 1 : C::ITK], goffV_r[C::GOFF_LDS ? 1 : C::ITV];
  auto goffK = [&](int it) {
    return C::GOFF_LDS ? sgoff[it * kThreads + tid] : goffK_r[C::GOFF_LDS ? 0 : it];
  };
  auto goffV = [&](int it) {
    return C::GOFF_LDS ? sgoff[(C::ITK + it) * kThreads + tid] : goffV_r[C::GOFF_LDS ? 0 : it];
  };
#pragma unroll
  for (int it = 0; it < C::ITK; ++it) {
    int s = it * kThreads + tid, key = s >> 3, c = (s & 7) ^ kswz(key);
    int gy = min(ty0 + key / C::LX, H - 1), gx = min(tx0 + key % C::LX, W - 1);
    int off = s < C::KSLOTS ? (gy * W + gx) * kD + c * 8 : -1;
    if (C::GOFF_LDS) sgoff[it * kThreads + tid] = off;
    else goffK_r[C::GOFF_LDS ? 0 : it] = off;
  }
#pragma unroll
  for (int it = 0; it < C::ITV; ++it) {
    int s = it * kThreads + tid, key = s / 10, c = s - key * 10;
    int gy = min(ty0 + key / C::LX, H - 1), gx = min(tx0 + key % C::LX, W - 1);
    int off = (s < C::VSLOTS && c < 8) ? (gy * W + gx) * kD + c * 8 : -1;
    if (C::GOFF_LDS) sgoff[(C::ITK + it) * kThreads + tid] = off;
    else goffV_r[C::GOFF_LDS ? 0 : it] = off;
  }
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * 16 : nullptr;
  const int64_t bh_base = (int64_t)bh * Z * HW;  // token index of (b, h, 0, 0, 0)

  auto issue_copy = [&](int p, char* tk, char* tv) {
    const uint16_t* kp = a.k + (bh_base + (int64_t)p * HW) * kD;
    const uint16_t* vp = a.v + (bh_base + (int64_t)p * HW) * kD;
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      const int o = goffK(it);
      if (o >= 0) copy16_to_lds(kp + o, tk + (it * kThreads + wave * 64) * 16);
    }
#pragma unroll
    for (int it = 0; it < C::ITV; ++it) {
      const int o = goffV(it);
      if (o >= 0) copy16_to_lds(vp + o, tv + (it * kThreads + wave * 64) * 16);
    }
  };

  // phases of this thread's K slots, as float16 (cos, sin) pairs, staged once
  if (C::PH_LDS && csb) {
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      const int o = goffK(it);
      if (o < 0) continue;
      const float4* pp = csb + (o >> 6) * 16 + ((o & 63) >> 2);
      const float4 p0 = pp[0], p1 = pp[1];
      st16(sph + (it * kThreads + tid) * 16,
           make_uint4(pack2h(p0.x, p0.y), pack2h(p0.z, p0.w), pack2h(p1.x, p1.y), pack2h(p1.z, p1.w)));
    }
  }
  // Rotate (or convert) this thread's K slots of one tile in place, bf16 -> float16.
  // A thread's copies land in its own slots, so its own wait suffices: no barrier.
  auto rotate_k = [&](char* tk) {
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      const int o = goffK(it);
      if (o < 0) continue;
      char* ad = tk + (it * kThreads + tid) * 16;
      uint4 x = ld16(ad);
      if (csb) {
        if (C::PH_LDS) {
          x = rotate8h_pk(x, ld16(sph + (it * kThreads + tid) * 16));
        } else {
          const float4* pp = csb + (o >> 6) * 16 + ((o & 63) >> 2);
          x = rotate8h(x, pp[0], pp[1], 1.f);
        }
      } else {
        x = scale8h(x, 1.f);
      }
      st16(ad, x);
    }
  };

  // ---- queries: load, rotate, scale, keep as the B operand of K.Q^T ----------
  f16x8 qf[C::QL][2];
  float m[C::QL], l[C::QL];
  f32x4 o[C::QL][4];
  const float4* csq = csb ? csb + ((int64_t)qy * W + qx) * 16 : nullptr;
#pragma unroll
  for (int j = 0; j < C::QL; ++j) {
    int zq = min(z0 + grp + 2 * j, Z - 1);
    const uint4* src = reinterpret_cast<const uint4*>(a.q + (bh_base + zq * HW + (int64_t)qy * W + qx) * kD);
    uint4 x0 = src[g], x1 = src[4 + g];
    uint4 r0, r1;
    if (csq) {
      r0 = rotate8h(x0, csq[2 * g], csq[2 * g + 1], a.qscale);
      r1 = rotate8h(x1, csq[8 + 2 * g], csq[8 + 2 * g + 1], a.qscale);
    } else {
      r0 = scale8h(x0, a.qscale);
      r1 = scale8h(x1, a.qscale);
    }
    qf[j][0] = __builtin_bit_cast(f16x8, r0);
    qf[j][1] = __builtin_bit_cast(f16x8, r1);
    m[j] = -INFINITY;
    l[j] = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) o[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // one (query level j, key level) update with the key tiles tk, tv
  auto update = [&](int j, const char* tk, const char* tv) {
    f32x4 s[C::NC];
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      f16x8 k0 = __builtin_bit_cast(f16x8, ld16(tk + kaddr[c]));
      f16x8 k1 = __builtin_bit_cast(f16x8, ld16(tk + (kaddr[c] ^ 64u)));
      f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(k0, qf[j][0], bias[c], 0, 0, 0);
      s[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(k1, qf[j][1], acc, 0, 0, 0);
    }
    float mx = fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3]));
#pragma unroll
    for (int c = 1; c < C::NC; ++c)
      mx = fmaxf(fmaxf(mx, fmaxf(s[c][0], s[c][1])), fmaxf(s[c][2], s[c][3]));
    mx = max_over_rows(mx);
    if (__any(mx > m[j] + kLazy)) {  // rare: move the running maximum, rescale
      const float mn = fmaxf(m[j], mx);
      const float alpha = __builtin_amdgcn_exp2f(m[j] - mn);
      m[j] = mn;
      l[j] *= alpha;
#pragma unroll
      for (int t = 0; t < 4; ++t) o[j][t] *= alpha;
    }
    const float mj = m[j];
    uint32_t pk[C::NC][2];
    float ls = l[j];
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      pk[c][0] = pack2(__builtin_amdgcn_exp2f(s[c][0] - mj), __builtin_amdgcn_exp2f(s[c][1] - mj));
      pk[c][1] = pack2(__builtin_amdgcn_exp2f(s[c][2] - mj), __builtin_amdgcn_exp2f(s[c][3] - mj));
      ls = psum8(pk[c][0], pk[c][1], ls);
    }
    l[j] = ls;
#pragma unroll
    for (int st = 0; st < C::NS; ++st) {
      const int c0 = 2 * st, c1 = 2 * st + 1;
      const bool two = c1 < C::NC;
      bf16x8 pf = __builtin_bit_cast(bf16x8, make_uint4(pk[c0][0], pk[c0][1], two ? pk[c1][0] : 0u, two ? pk[c1][1] : 0u));
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        i16x4 lo = tr_read(tv + vaddr[c0] + 32 * t);
        i16x4 hi = two ? tr_read(tv + vaddr[c1] + 32 * t) : i16x4{0, 0, 0, 0};
        uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        bf16x8 vf = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
        o[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[j][t], 0, 0, 0);
      }
    }
  };

  // all query levels of this wave whose window holds key level p
  auto compute = [&](int p, const char* tk, const char* tv) {
#pragma unroll
    for (int j = 0; j < C::QL; ++j) {
      const int zq = z0 + grp + 2 * j;
      if (zq >= Z) continue;
      const int zs = win_start(zq, Z, KZ);
      if (p < zs || p >= zs + KZ) continue;
      update(j, tk, tv);
    }
  };

  // ---- key levels needed by the block's query levels, double-buffered -------
  // Level p+1 is copied while level p is computed; then each thread waits for
  // its own copies, rotates its own K slots, and one barrier publishes the level.
  // The barrier also retires every read of the tiles the next copy overwrites.
  const int zlast = min(z0 + ZQ, Z) - 1;
  const int kp_lo = win_start(z0, Z, KZ);
  const int kp_hi = win_start(zlast, Z, KZ) + KZ;

  issue_copy(kp_lo, tK0, tV0);
  __builtin_amdgcn_s_waitcnt(0);
  rotate_k(tK0);
  __syncthreads();
  for (int p = kp_lo; p < kp_hi; p += 2) {
    // level p in tiles 0, level p+1 (if any) in tiles 1
    const bool more1 = p + 1 < kp_hi;
    if (more1) issue_copy(p + 1, tK1, tV1);
    compute(p, tK0, tV0);
    if (more1) {
      __builtin_amdgcn_s_waitcnt(0);
      rotate_k(tK1);
      __syncthreads();
      const bool more2 = p + 2 < kp_hi;
      if (more2) issue_copy(p + 2, tK0, tV0);
      compute(p + 1, tK1, tV1);
      if (more2) {
        __builtin_amdgcn_s_waitcnt(0);
        rotate_k(tK0);
        __syncthreads();
      }
    }
  }

  // ---- normalise and store --------------------------------------------------------
  const bool in_grid = qy_raw < H && qx_raw < W;
#pragma unroll
  for (int j = 0; j < C::QL; ++j) {
    const int zq = z0 + grp + 2 * j;
    const float lt = sum_over_rows(l[j]);
    if (zq >= Z || !in_grid) continue;
    const float inv = 1.f / lt;
    const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
    uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
#pragma unroll
    for (int t = 0; t < 4; ++t)  // d = 16t + 4g + i
      dst[4 * t + g] = make_uint2(pack2(o[j][t][0] * inv, o[j][t][1] * inv),
                                  pack2(o[j][t][2] * inv, o[j][t][3] * inv));
    if (a.lse && g == 0) a.lse[tok] = (m[j] + __log2f(lt)) * kLn2;
  }
}

template <int KZ, int KY, int KX, int ZQ>
bool launch(const strata_na3d_desc& d, const void* q, const void* k, const void* v, const float* cs,
            void* out, float* lse, hipStream_t s) {
  Args a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.heads = d.heads;
  a.Z = d.Z;
  a.H = d.H;
  a.W = d.W;
  a.n_zb = (d.Z + ZQ - 1) / ZQ;
  a.n_yb = (d.H + kBY - 1) / kBY;
  a.n_xb = (d.W + kBX - 1) / kBX;
  a.qscale = d.scale * kLog2e;
  int64_t blocks = (int64_t)d.B * d.heads * a.n_zb * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  hipLaunchKernelGGL((na3d_fwd_mfma_kernel<KZ, KY, KX, ZQ>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
  return true;
}

}  // namespace

bool launch_na3d_fwd_mfma(const strata_na3d_desc& d, const void* q, const void* k, const void* v,
                          const float* cs, void* out, float* lse, hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  // element offsets inside one key level are int32
  if ((int64_t)d.H * d.W * kD >= (int64_t)1 << 31) return false;
  if (d.kz == 3 && d.ky == 7 && d.kx == 7) return launch<3, 7, 7, 8>(d, q, k, v, cs, out, lse, s);
  if (d.kz == 5 && d.ky == 9 && d.kx == 9) return launch<5, 9, 9, 2>(d, q, k, v, cs, out, lse, s);
  return false;
}

}  // namespace strata

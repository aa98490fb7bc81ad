// bf16 MFMA neighbourhood-attention forward for gfx950 (head_dim 64).
//
// Work decomposition
//   workgroup : one (tile, head), an 8 x 8 block of (y, x) query positions and
//               ZB consecutive query levels; 4 waves of 64 lanes.
//   wave      : a 4 x 4 (y, x) sub-block = 16 queries, for each of the ZB levels.
//   key sweep : the workgroup walks the key levels its queries need, one at a
//               time.  For each key level it stages the rotated K and the V of
//               the (8+ky-1) x (8+kx-1) key box into LDS, then every wave updates
//               the queries of each level whose z-window holds that key level.
//
// Per (query level, key level) a wave multiplies the keys of its 4x4 block's
// box -- (3+ky) x (3+kx) keys, in 16-key chunks -- with its 16 queries:
//   S^T (16 keys x 16 queries) = K . Q^T     v_mfma_f32_16x16x32_f16, the
//                                           accumulator is seeded with the
//                                           window mask (0 or -inf),
//   online softmax on S^T in registers (each lane owns one query column),
//   O^T (64 d x 16 queries) += V^T . P^T    V^T fragments come straight from
//                                           the row-major V tile through the
//                                           LDS transpose read; P^T is the S^T
//                                           accumulator packed to bf16 in place.
// The rotation of StereoRoPE is applied to Q when it is loaded into registers
// and to K while it is staged, in float32.  The rotated Q and K are rounded to
// float16, not bf16, for the Q.K^T contraction (v_mfma_f32_16x16x32_f16, same
// rate): bf16 rounding of the rotated operands alone costs up to ~0.5% of an
// output, beyond the parity bound, while float16 keeps it near 0.05%.  Inputs
// beyond the float16 range (|x| > 65504 after rotation and scaling) saturate.
// P and V stay bf16.  The logit scale and log2(e) are folded into Q so the
// softmax uses exp2.
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

constexpr int kBY = 8, kBX = 8;      // query block of a workgroup (y, x)
constexpr int kThreads = 256;        // 4 waves
constexpr int kD = 64;               // head_dim
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int KZ, int KY, int KX, int ZB>
struct Cfg {
  static constexpr int LY = kBY + KY - 1, LX = kBX + KX - 1;  // staged key box per level
  static constexpr int NUY = 3 + KY, NUX = 3 + KX;            // key box of one 4x4 sub-block
  static constexpr int NU = NUY * NUX;
  static constexpr int NC = (NU + 15) / 16;                   // 16-key chunks
  static constexpr int NS = (NC + 1) / 2;                     // 32-key PV steps
  static constexpr int KEYS = LY * LX;
  static constexpr int CHUNKS16 = KEYS * (kD * 2 / 16);       // 16-byte pieces per level per tensor
  static constexpr int LDS_U4 = 2 * CHUNKS16;                 // K then V
};

struct Args {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;   // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  uint16_t* out;
  float* lse;
  int B, heads, Z, H, W;
  int n_zb, n_yb, n_xb;
  float qscale;       // scale * log2(e)
};

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2 f = {a, b};
  bf16x2 h = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Two floats -> packed float16 pair (nearest-even), saturating at +-65504.
__device__ __forceinline__ uint32_t pack2h(float a, float b) {
  f32x2 f = {__builtin_amdgcn_fmed3f(a, -65504.f, 65504.f), __builtin_amdgcn_fmed3f(b, -65504.f, 65504.f)};
  f16x2 h = __builtin_convertvector(f, f16x2);
  return __builtin_bit_cast(uint32_t, h);
}

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
    float y0 = fmaf(a, c, -b * s) * mul;
    float y1 = fmaf(a, s, b * c) * mul;
    r[t] = pack2h(y0, y1);
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

__device__ __forceinline__ i16x4 tr_read(const char* lds_base, uint32_t byte_off) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(lds_base + byte_off));
}

template <int KZ, int KY, int KX, int ZB>
__global__ void __launch_bounds__(kThreads, 2) na3d_fwd_mfma_kernel(Args a) {
  using C = Cfg<KZ, KY, KX, ZB>;
  __shared__ uint4 lds[C::LDS_U4];
  uint4* ldsK = lds;
  const char* ldsV = reinterpret_cast<const char*>(lds + C::CHUNKS16);

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
  const int by0 = yb * kBY, bx0 = xb * kBX, z0 = zb * ZB;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;

  // staged key box of the workgroup, and the key box of this wave's sub-block
  const int ty0 = win_start(min(by0, H - 1), H, KY);
  const int tx0 = win_start(min(bx0, W - 1), W, KX);
  const int sy0 = by0 + 4 * (wave >> 1), sx0 = bx0 + 4 * (wave & 1);
  const int uy0 = win_start(min(sy0, H - 1), H, KY);
  const int ux0 = win_start(min(sx0, W - 1), W, KX);
  // this lane's query column (clamped into the grid; stores are masked later)
  const int qy_raw = sy0 + (qn >> 2), qx_raw = sx0 + (qn & 3);
  const int qy = min(qy_raw, H - 1), qx = min(qx_raw, W - 1);
  const int wys = win_start(qy, H, KY), wxs = win_start(qx, W, KX);

  // ---- per-lane LDS addresses and window mask, identical for every key level ----
  uint32_t kaddr[C::NC], vaddr[C::NC];
  f32x4 bias[C::NC];
#pragma unroll
  for (int c = 0; c < C::NC; ++c) {
    // K fragment (A operand): row = key 16c + qn, 16 bytes at column g (and g+4)
    {
      int u = 16 * c + qn;
      int key = 0;
      if (u < C::NU) key = (uy0 - ty0 + u / C::NUX) * C::LX + (ux0 - tx0 + u % C::NUX);
      kaddr[c] = key * 128 + ((g ^ (key & 7)) << 4);
    }
    // V^T fragment through the transpose read: source row = key 16c + 4g + qn/4,
    // 8 bytes at element 4*(qn%4) of each 16-element d tile
    {
      int u = 16 * c + 4 * g + (qn >> 2);
      int key = 0;
      if (u < C::NU) key = (uy0 - ty0 + u / C::NUX) * C::LX + (ux0 - tx0 + u % C::NUX);
      int hb = (qn & 3) >> 1;
      vaddr[c] = key * 128 + ((hb ^ (key & 7)) << 4) + ((qn & 1) << 3);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int u = 16 * c + 4 * g + i;
      int ky = uy0 + u / C::NUX, kx = ux0 + u % C::NUX;
      bool ok = u < C::NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX;
      bias[c][i] = ok ? 0.f : -INFINITY;
    }
  }

  // ---- queries: load, rotate, scale, keep as the B operand of K.Q^T ----------
  const int64_t HW = (int64_t)H * W;
  const int64_t bh_base = (int64_t)bh * Z * HW;  // token index of (b, h, 0, 0, 0)
  f16x8 qf[ZB][2];
  float m[ZB], l[ZB];
  f32x4 o[ZB][4];
  const float4* csq = a.cs ? a.cs + ((int64_t)b * HW + (int64_t)qy * W + qx) * 16 : nullptr;
#pragma unroll
  for (int j = 0; j < ZB; ++j) {
    int zq = min(z0 + j, Z - 1);
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

  // ---- key levels needed by the block's query levels --------------------------
  const int zlast = min(z0 + ZB, Z) - 1;
  const int kp_lo = win_start(z0, Z, KZ);
  const int kp_hi = win_start(zlast, Z, KZ) + KZ;

  for (int p = kp_lo; p < kp_hi; ++p) {
    __syncthreads();  // every wave is done with the previous level's tiles
    // stage K (rotated, float16) and V (bf16) of key level p: 16 bytes per thread per step
    const int64_t lvl = bh_base + (int64_t)p * HW;
    for (int idx = tid; idx < 2 * C::CHUNKS16; idx += kThreads) {
      const bool isV = idx >= C::CHUNKS16;
      const int ci = isV ? idx - C::CHUNKS16 : idx;
      const int key = ci >> 3, col = ci & 7;
      const int gy = ty0 + key / C::LX, gx = tx0 + key % C::LX;
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (gy < H && gx < W) {
        const int64_t tok = lvl + (int64_t)gy * W + gx;
        if (isV) {
          val = reinterpret_cast<const uint4*>(a.v + tok * kD)[col];
        } else {
          val = reinterpret_cast<const uint4*>(a.k + tok * kD)[col];
          if (a.cs) {
            const float4* ph = a.cs + ((int64_t)b * HW + (int64_t)gy * W + gx) * 16 + 2 * col;
            val = rotate8h(val, ph[0], ph[1], 1.f);
          } else {
            val = scale8h(val, 1.f);
          }
        }
      }
      lds[(isV ? C::CHUNKS16 : 0) + key * 8 + (col ^ (key & 7))] = val;
    }
    __syncthreads();

#pragma unroll
    for (int j = 0; j < ZB; ++j) {
      const int zq = z0 + j;
      if (zq >= Z) continue;
      const int zs = win_start(zq, Z, KZ);
      if (p < zs || p >= zs + KZ) continue;

      // S^T = K . Q^T, seeded with the window mask
      f32x4 s[C::NC];
#pragma unroll
      for (int c = 0; c < C::NC; ++c) {
        const char* kb = reinterpret_cast<const char*>(ldsK);
        f16x8 k0 = __builtin_bit_cast(f16x8, *reinterpret_cast<const uint4*>(kb + kaddr[c]));
        f16x8 k1 = __builtin_bit_cast(f16x8, *reinterpret_cast<const uint4*>(kb + (kaddr[c] ^ 64u)));
        f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(k0, qf[j][0], bias[c], 0, 0, 0);
        s[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(k1, qf[j][1], acc, 0, 0, 0);
      }
      // online softmax (log2 domain); each lane owns one query, 4 keys per chunk
      float mx = -INFINITY;
#pragma unroll
      for (int c = 0; c < C::NC; ++c)
        mx = fmaxf(fmaxf(mx, fmaxf(s[c][0], s[c][1])), fmaxf(s[c][2], s[c][3]));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m[j], mx);
      const float alpha = __builtin_amdgcn_exp2f(m[j] - mn);
      m[j] = mn;
      float ls = 0.f;
      uint32_t pk[C::NC][2];
#pragma unroll
      for (int c = 0; c < C::NC; ++c) {
        float p0 = __builtin_amdgcn_exp2f(s[c][0] - mn);
        float p1 = __builtin_amdgcn_exp2f(s[c][1] - mn);
        float p2 = __builtin_amdgcn_exp2f(s[c][2] - mn);
        float p3 = __builtin_amdgcn_exp2f(s[c][3] - mn);
        ls += (p0 + p1) + (p2 + p3);
        pk[c][0] = pack2(p0, p1);
        pk[c][1] = pack2(p2, p3);
      }
      l[j] = fmaf(l[j], alpha, ls);
#pragma unroll
      for (int t = 0; t < 4; ++t) o[j][t] *= alpha;
      // O^T += V^T . P^T over 32-key steps (chunks 2s, 2s+1)
#pragma unroll
      for (int st = 0; st < C::NS; ++st) {
        const int c0 = 2 * st, c1 = 2 * st + 1;
        uint4 pb = make_uint4(pk[c0][0], pk[c0][1], c1 < C::NC ? pk[c1][0] : 0u, c1 < C::NC ? pk[c1][1] : 0u);
        bf16x8 pf = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          i16x4 lo = tr_read(ldsV, vaddr[c0] ^ (uint32_t)(t << 5));
          i16x4 hi = c1 < C::NC ? tr_read(ldsV, vaddr[c1] ^ (uint32_t)(t << 5)) : i16x4{0, 0, 0, 0};
          uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
          bf16x8 vf = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
          o[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[j][t], 0, 0, 0);
        }
      }
    }
  }

  // ---- normalise and store --------------------------------------------------------
  const bool in_grid = qy_raw < H && qx_raw < W;
#pragma unroll
  for (int j = 0; j < ZB; ++j) {
    const int zq = z0 + j;
    if (zq >= Z) continue;
    float lt = l[j];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const float inv = 1.f / lt;
    if (in_grid) {
      const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
      uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
#pragma unroll
      for (int t = 0; t < 4; ++t)   // d = 16t + 4g + i
        dst[4 * t + g] = make_uint2(pack2(o[j][t][0] * inv, o[j][t][1] * inv),
                                    pack2(o[j][t][2] * inv, o[j][t][3] * inv));
      if (a.lse && g == 0) a.lse[tok] = (m[j] + __log2f(lt)) * kLn2;
    }
  }
}

template <int KZ, int KY, int KX, int ZB>
void launch(const strata_na3d_desc& d, const void* q, const void* k, const void* v, const float* cs,
            void* out, float* lse, hipStream_t s) {
  Args a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.B = d.B;
  a.heads = d.heads;
  a.Z = d.Z;
  a.H = d.H;
  a.W = d.W;
  a.n_zb = (d.Z + ZB - 1) / ZB;
  a.n_yb = (d.H + kBY - 1) / kBY;
  a.n_xb = (d.W + kBX - 1) / kBX;
  a.qscale = d.scale * kLog2e;
  int64_t blocks = (int64_t)d.B * d.heads * a.n_zb * a.n_yb * a.n_xb;
  hipLaunchKernelGGL((na3d_fwd_mfma_kernel<KZ, KY, KX, ZB>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
}

}  // namespace

bool launch_na3d_fwd_mfma(const strata_na3d_desc& d, const void* q, const void* k, const void* v,
                          const float* cs, void* out, float* lse, hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  int64_t blocks = (int64_t)d.B * d.heads * ((d.Z + 3) / 4) * ((d.H + kBY - 1) / kBY) * ((d.W + kBX - 1) / kBX);
  if (blocks >= (int64_t)1 << 31) return false;
  if (d.kz == 3 && d.ky == 7 && d.kx == 7) {
    launch<3, 7, 7, 4>(d, q, k, v, cs, out, lse, s);
    return true;
  }
  if (d.kz == 5 && d.ky == 9 && d.kx == 9) {
    launch<5, 9, 9, 4>(d, q, k, v, cs, out, lse, s);
    return true;
  }
  return false;
}

}  // namespace strata

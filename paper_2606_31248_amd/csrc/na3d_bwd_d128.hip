// MFMA neighbourhood-attention backward for head_dim 128 (the decoder's NA3D,
// App. B.3), bf16 in/out, window 9 x 9 x 9, StereoRoPE fused.  Options (App.
// B.5): QK RMSNorm in both passes (factors at the Q/K loads, the norm's
// Jacobian applied to dQ and dK at the store); a two-term upstream gradient
// (the gated dA = hi + lo) in both passes: one more MFMA per k-step for Y and
// per tile for dV, the dK/dV pass then staging the query box in two windows
// of 128 rows (three 32 KB tiles).
//
// The same two passes and arithmetic as at head_dim 64, with 128-wide rows:
//
// dQ (query-stationary; an 8 x 8 block of (y, x) queries and ZQ levels per
// workgroup, a 4 x 4 sub-block on all ZQ levels per wave, one wave per SIMD
// so that the S/Y chunks, dO and Q of a level fit in its registers).  Per (query level, key level):
//   S^T = K~ . Q~^T             four float16 MFMAs per 16-key chunk, seeded
//                               with the window mask; P^T = exp2(S^T - LSE)
//                               from the forward's log-sum-exp;
//   Y^T = V . dO^T - D          four bf16 MFMAs per chunk (V rows as the A
//                               operand), seeded with -D;
//   dS^T = P^T * Y^T (float32), then float16 with a per-query power-of-two
//   scale 2^(15-E), E bounding |Y| over the key levels seen so far (the
//   accumulator is rescaled exactly when E grows);
//   dQ~^T (128 d x 16 queries) += K~^T . dS^T, eight 16-row float16 MFMA tiles
//                               whose K~^T fragments come from the rotated K
//                               tile by the LDS transpose read.
// One key level of the 16 x 16 key box (K~ 64 KB in 256-byte rows with their
// 16-byte columns XOR-swizzled, V 72 KB in 288-byte rows) fills the LDS, so it
// is single-buffered: copy, rotate in place, barrier, compute, barrier.  The
// window mask is kept as bits (one per lane and key of a chunk), not as float
// seeds, which leaves registers for the S and Y chunks of a level.
//
// dK, dV (key-stationary; a 4 x 4 block of (y, x) keys and ZK levels per
// workgroup, one wave per key level).  The queries that can see any key of the
// block form a 16 x 16 box per level; its Q~ (float16) and dO (bf16) rows,
// 256 bytes each with swizzled columns, are staged per level (128 KB, single
// buffer) with LSE and -D.  Per (key level, query level) a wave walks the box
// in steps of 32 queries:
//   X = Q~ . K~^T seeded with -LSE (or -inf outside the window), P = exp2(X);
//   Y = dO . V^T - D;
//   dV^T (128 d x 16 keys) += dO^T . P and dK~^T += Q~^T . dS, eight tiles
//   each, from transpose reads of the staged rows; dS in float16 with the
//   per-key scale 2^(15-E).
// Stores: dQ = R^T (scale 2^(E-15) dQ~), dK = R^T (scale 2^(E-15) dK~), dV.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

#include <algorithm>

namespace strata {
namespace {

using namespace mfma;

constexpr int kD = 128;
constexpr int kCS4 = kD / 4;  // float4 entries of the phase table per position
constexpr int kLdsMax = 160 * 1024;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMinExp = -100;  // lower bound of the dS exponent (keeps 2^(15-E) finite)

struct Args {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;      // [B, H, W, 32] float4 = two (cos, sin) pairs; nullptr: no rotation
  const uint16_t* dout;
  const float* lse;      // natural log
  const float* dvec;     // D = rowsum(dO * O)
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  int heads, Z, H, W;
  int n_zb, n_yb, n_xb;
  float scale, qscale;   // scale, scale * log2(e)
  float eps;             // QK RMSNorm (with NORM)
  const uint16_t* dout_lo;  // low term of a two-term upstream gradient (with LO)
};

// ============================================================================ dQ
constexpr int kQBY = 8, kQBX = 8;
constexpr int kQWaves = 4, kQThreads = 64 * kQWaves;  // one wave per SIMD: up to 512 registers each
constexpr int kQGroups = kQWaves / 4;                 // level groups (waves 4g..4g+3 take levels = g mod kQGroups)
constexpr int kKRow = 256, kVRow = 288;

template <int KZ, int KY, int KX, int ZQ>
struct QCfg {
  static constexpr int LY = kQBY + KY - 1, LX = kQBX + KX - 1;
  static constexpr int NUY = 3 + KY, NUX = 3 + KX, NU = NUY * NUX;
  static constexpr int NC = (NU + 15) / 16, NS = (NC + 1) / 2;
  static constexpr int KEYS = LY * LX;
  static constexpr int KSLOTS = KEYS * (kKRow / 16), VSLOTS = KEYS * (kVRow / 16);
  static constexpr int KBYTES = KEYS * kKRow, VBYTES = KEYS * kVRow;
  static constexpr int ITK = (KSLOTS + kQThreads - 1) / kQThreads;
  static constexpr int ITV = (VSLOTS + kQThreads - 1) / kQThreads;
  static constexpr int QL = ZQ / kQGroups;
  static_assert(ZQ % kQGroups == 0 && NC <= 16, "layout");
  static_assert(KBYTES + VBYTES <= kLdsMax, "key tiles exceed LDS");
};

template <int KZ, int KY, int KX, int ZQ, bool NORM, bool LO>
__global__ void __launch_bounds__(kQThreads, 1) na3d_bwd_dq_d128_kernel(Args a) {
  using C = QCfg<KZ, KY, KX, ZQ>;
  __shared__ __attribute__((aligned(16))) char tK[C::KBYTES];
  __shared__ __attribute__((aligned(16))) char tV[C::VBYTES];

  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int xb = bid % a.n_xb;
  const int yb = (bid / a.n_xb) % a.n_yb;
  const int zb = (bid / (a.n_xb * a.n_yb)) % a.n_zb;
  const int bh = bid / (a.n_xb * a.n_yb * a.n_zb);
  const int b = bh / a.heads;
  const int H = a.H, W = a.W, Z = a.Z;
  const int by0 = yb * kQBY, bx0 = xb * kQBX, z0 = zb * ZQ;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;
  const int sb = wave & 3, grp = wave >> 2;

  const int ty0 = win_start(min(by0, H - 1), H, KY);
  const int tx0 = win_start(min(bx0, W - 1), W, KX);
  const int sy0 = by0 + 4 * (sb >> 1), sx0 = bx0 + 4 * (sb & 1);
  const int uy0 = win_start(min(sy0, H - 1), H, KY);
  const int ux0 = win_start(min(sx0, W - 1), W, KX);
  const int qy_raw = sy0 + (qn >> 2), qx_raw = sx0 + (qn & 3);
  const int qy = min(qy_raw, H - 1), qx = min(qx_raw, W - 1);
  const int wys = win_start(qy, H, KY), wxs = win_start(qx, W, KX);

  auto kswz = [&](int key) { return ((key % C::LX >> 1) + 5 * (key / C::LX)) & 7; };
  auto key_row = [&](int u) {
    return u < C::NU ? (uy0 - ty0 + u / C::NUX) * C::LX + (ux0 - tx0 + u % C::NUX) : 0;
  };

  // lane addresses: K fragment (A of S^T), V row (A of Y^T), K~^T transpose read;
  // window mask bit 4c + i: key 16c + 4g + i is in this lane's query window
  uint32_t kaddr[C::NC], vrow[C::NC], ktaddr[C::NC];
  uint64_t mbits = 0;
#pragma unroll
  for (int c = 0; c < C::NC; ++c) {
    {
      const int key = key_row(16 * c + qn);
      kaddr[c] = key * kKRow + ((g ^ kswz(key)) << 4);
      vrow[c] = key * kVRow + 16 * g;
    }
    {
      const int key = key_row(16 * c + 4 * g + (qn >> 2));
      ktaddr[c] = key * kKRow + ((((qn >> 1) & 1) ^ kswz(key)) << 4) + 8 * (qn & 1);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = 16 * c + 4 * g + i;
      const int ky = uy0 + u / C::NUX, kx = ux0 + u % C::NUX;
      if (u < C::NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX) mbits |= 1ull << (4 * c + i);
    }
  }

  // copy map (recomputed per level: registers are scarce here): element
  // offsets inside a key level, -1 for pad and past-the-end slots
  auto goffK = [&](int it) {
    const int s = it * kQThreads + tid, key = s >> 4, c = (s & 15) ^ kswz(key);
    const int gy = min(ty0 + key / C::LX, H - 1), gx = min(tx0 + key % C::LX, W - 1);
    return s < C::KSLOTS ? (gy * W + gx) * kD + c * 8 : -1;
  };
  auto goffV = [&](int it) {
    const int s = it * kQThreads + tid, key = s / 18, c = s - key * 18;
    const int gy = min(ty0 + key / C::LX, H - 1), gx = min(tx0 + key % C::LX, W - 1);
    return (s < C::VSLOTS && c < 16) ? (gy * W + gx) * kD + c * 8 : -1;
  };
  const int64_t HW = (int64_t)H * W;
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * kCS4 : nullptr;
  const int64_t bh_base = (int64_t)bh * Z * HW;

  auto issue_copy = [&](int p) {
    const uint16_t* kp = a.k + (bh_base + (int64_t)p * HW) * kD;
    const uint16_t* vp = a.v + (bh_base + (int64_t)p * HW) * kD;
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      const int o = goffK(it);
      if (o >= 0) copy16_to_lds(kp + o, tK + (it * kQThreads + wave * 64) * 16);
    }
#pragma unroll
    for (int it = 0; it < C::ITV; ++it) {
      const int o = goffV(it);
      if (o >= 0) copy16_to_lds(vp + o, tV + (it * kQThreads + wave * 64) * 16);
    }
  };
  auto rotate_k = [&]() {
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      const int o = goffK(it);
      if (o < 0) continue;
      char* ad = tK + (it * kQThreads + tid) * 16;
      uint4 x = ld16(ad);
      // (a key row is 16 consecutive slots, all in the tile)
      const float mul = NORM ? __builtin_amdgcn_rsqf(sum_over_16_lanes(sumsq8(x, 0.f)) * (1.f / kD) + a.eps) : 1.f;
      if (csb) {  // packed float16 rotation, phases converted from the float32 table
        const float4* pp = csb + (o >> 7) * kCS4 + ((o & 127) >> 2);
        const float4 p0 = pp[0], p1 = pp[1];
        x = rotate8h_pk(x, make_uint4(pack2h_rne(p0.x, p0.y), pack2h_rne(p0.z, p0.w), pack2h_rne(p1.x, p1.y),
                                      pack2h_rne(p1.z, p1.w)), mul);
      } else {
        x = scale8h(x, mul);
      }
      st16(ad, x);
    }
  };

  // queries: Q~ (float16, times scale log2 e) and dO (bf16) as B operands
  f16x8 qf[C::QL][4];
  bf16x8 gf[C::QL][4], gl[LO ? C::QL : 1][4];  // dO (hi and low terms)
  float rq[NORM ? C::QL : 1];                  // QK RMSNorm factor of the query
  float lse2[C::QL], nd[C::QL];
  int ex[C::QL];
  f32x4 o[C::QL][8];
  const float4* csq = csb ? csb + ((int64_t)qy * W + qx) * kCS4 : nullptr;
#pragma unroll
  for (int j = 0; j < C::QL; ++j) {
    const int zq = min(z0 + grp + kQGroups * j, Z - 1);
    const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
    const uint4* src = reinterpret_cast<const uint4*>(a.q + tok * kD);
    const uint4* gsrc = reinterpret_cast<const uint4*>(a.dout + tok * kD);
    uint4 x[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) x[kk] = src[4 * kk + g];
    float mul = a.qscale;
    if constexpr (NORM) {  // the 4 lanes of a query row hold its 128 values
      float ss = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) ss = sumsq8(x[kk], ss);
      rq[j] = __builtin_amdgcn_rsqf(sum_over_rows(ss) * (1.f / kD) + a.eps);
      mul *= rq[j];
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint4 r = csq ? rotate8h(x[kk], csq[8 * kk + 2 * g], csq[8 * kk + 2 * g + 1], mul) : scale8h(x[kk], mul);
      qf[j][kk] = __builtin_bit_cast(f16x8, r);
      gf[j][kk] = __builtin_bit_cast(bf16x8, gsrc[4 * kk + g]);
      if constexpr (LO) gl[j][kk] = __builtin_bit_cast(bf16x8, reinterpret_cast<const uint4*>(a.dout_lo + tok * kD)[4 * kk + g]);
    }
    lse2[j] = a.lse[tok] * kLog2e;
    nd[j] = -a.dvec[tok];
    ex[j] = kMinExp;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto update_dq = [&](int j) {
    // dS = P Y per chunk in float32 (P = exp2(S^T - LSE) <= 1), and the bound of |Y|
    f32x4 ds[C::NC];
    float my = 0.f;
    const f32x4 ndv = {nd[j], nd[j], nd[j], nd[j]};
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      f32x4 acc;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = ((mbits >> (4 * c + i)) & 1ull) ? 0.f : -INFINITY;
      f32x4 yy = ndv;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const f16x8 kf = __builtin_bit_cast(f16x8, ld16(tK + (kaddr[c] ^ (64u * kk))));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[j][kk], acc, 0, 0, 0);
        const bf16x8 vv = __builtin_bit_cast(bf16x8, ld16(tV + vrow[c] + 64 * kk));
        yy = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vv, gf[j][kk], yy, 0, 0, 0);
        if constexpr (LO) yy = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vv, gl[j][kk], yy, 0, 0, 0);
      }
      my = fmaxf(fmaxf(my, fmaxf(fabsf(yy[0]), fabsf(yy[1]))), fmaxf(fabsf(yy[2]), fabsf(yy[3])));
#pragma unroll
      for (int i = 0; i < 4; ++i) ds[c][i] = __builtin_amdgcn_exp2f(acc[i] - lse2[j]) * yy[i];
    }
    my = max_over_rows(my);
    const int e = max(__builtin_amdgcn_frexp_expf(my), kMinExp);
    if (__any(e > ex[j])) {  // the bound grew: rescale the accumulator exactly
      const int en = max(ex[j], e);
      const float f = __builtin_amdgcn_ldexpf(1.f, ex[j] - en);
#pragma unroll
      for (int t = 0; t < 8; ++t) o[j][t] *= f;
      ex[j] = en;
    }
    const float sc = __builtin_amdgcn_ldexpf(1.f, 15 - ex[j]);  // |dS| 2^(15-E) < 2^15
    uint32_t dk[C::NC][2];
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      dk[c][0] = pack2h_rne(ds[c][0] * sc, ds[c][1] * sc);
      dk[c][1] = pack2h_rne(ds[c][2] * sc, ds[c][3] * sc);
    }
#pragma unroll
    for (int st = 0; st < C::NS; ++st) {
      const int c0 = 2 * st, c1 = 2 * st + 1;
      const bool two = c1 < C::NC;
      const int cc = two ? c1 : c0;
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(dk[c0][0], dk[c0][1], two ? dk[cc][0] : 0u, two ? dk[cc][1] : 0u));
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const i16x4 lo = tr_read(tK + (ktaddr[c0] ^ (32u * t)));
        const i16x4 hi = two ? tr_read(tK + (ktaddr[cc] ^ (32u * t))) : i16x4{0, 0, 0, 0};
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        const f16x8 kt = __builtin_bit_cast(f16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
        o[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kt, df, o[j][t], 0, 0, 0);
      }
    }
  };

  const int zlast = min(z0 + ZQ, Z) - 1;
  const int kp_lo = win_start(z0, Z, KZ);
  const int kp_hi = win_start(zlast, Z, KZ) + KZ;
  for (int p = kp_lo; p < kp_hi; ++p) {
    issue_copy(p);
    __builtin_amdgcn_s_waitcnt(0);
    rotate_k();
    __syncthreads();  // the level is published
#pragma unroll
    for (int j = 0; j < C::QL; ++j) {
      const int zq = z0 + grp + kQGroups * j;
      if (zq >= Z) continue;
      const int zs = win_start(zq, Z, KZ);
      if (p < zs || p >= zs + KZ) continue;
      update_dq(j);
    }
    __syncthreads();  // every read of the level is done before the next copy
  }

  // dQ = R^T (scale 2^(E-15) dQ~); the lane holds d = 16t + 4g + i
  const bool in_grid = qy_raw < H && qx_raw < W;
#pragma unroll
  for (int j = 0; j < C::QL; ++j) {
    const int zq = z0 + grp + kQGroups * j;
    if (zq >= Z || !in_grid) continue;
    const float f = a.scale * __builtin_amdgcn_ldexpf(1.f, ex[j] - 15);
    const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
    uint2* dst = reinterpret_cast<uint2*>(a.dq + tok * kD);
    f32x4 x[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      x[t] = o[j][t] * f;
      if (csq) {
        const float4 ph = csq[4 * t + g];  // pairs 8t+2g and 8t+2g+1
        const float r0 = fmaf(x[t][0], ph.x, x[t][1] * ph.y), r1 = fmaf(x[t][1], ph.x, -x[t][0] * ph.y);
        const float r2 = fmaf(x[t][2], ph.z, x[t][3] * ph.w), r3 = fmaf(x[t][3], ph.z, -x[t][2] * ph.w);
        x[t] = f32x4{r0, r1, r2, r3};
      }
    }
    if constexpr (NORM) {
      // the gradient of q^ = r q carried back through the norm:
      // dq = r (dq^ - q^ mean(dq^ q^)), q^ from the raw row in float32
      const uint2* qr = reinterpret_cast<const uint2*>(a.q + tok * kD);
      f32x4 qh[8];
      float c = 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint2 w = qr[4 * t + g];
        qh[t] = f32x4{lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y)} * rq[j];
#pragma unroll
        for (int i = 0; i < 4; ++i) c = fmaf(x[t][i], qh[t][i], c);
      }
      c = sum_over_rows(c) * (1.f / kD);
#pragma unroll
      for (int t = 0; t < 8; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) x[t][i] = rq[j] * fmaf(-qh[t][i], c, x[t][i]);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) dst[4 * t + g] = make_uint2(pack2(x[t][0], x[t][1]), pack2(x[t][2], x[t][3]));
  }
}

// ======================================================================== dK, dV
constexpr int kRow = 256;  // staged query row (Q~ float16 or dO bf16)

// queries whose (border-clamped) window holds position j of an axis of extent L
__host__ __device__ __forceinline__ int inv_lo(int j, int k) { return j < k ? 0 : j - (k >> 1); }
__host__ __device__ __forceinline__ int inv_hi(int j, int L, int k) { return j >= L - k ? L - 1 : j + (k >> 1); }
__device__ __forceinline__ int rswz(int u) { return (((u >> 1) & 3) << 1) | ((u >> 3) & 1); }

// The query box is staged in row windows of RW rows: the whole box (Q~ and dO,
// 2 x 64 KB) without the low term; with it, three tiles of 128 rows (96 KB)
// and two windows per level.
template <int KZ, int KY, int KX, int ZK, bool LO>
struct KvCfg {
  static constexpr int kThreads = 64 * ZK;
  static constexpr int MQY = 4 + 3 * (KY / 2), MQX = 4 + 3 * (KX / 2);  // largest query box
  static constexpr int MQ = (MQY * MQX + 31) / 32 * 32;                  // rows, whole 32-query steps
  static constexpr int RW = LO ? 128 : MQ;                               // rows per staged window
  static constexpr int NW = (MQ + RW - 1) / RW;                          // windows of the largest box
  static constexpr int TBYTES = RW * kRow;
  static constexpr int SLOTS = RW * (kRow / 16);
  static constexpr int IT = (SLOTS + kThreads - 1) / kThreads;
  static constexpr int IS = (MQ + kThreads - 1) / kThreads;
  static_assert(RW % 32 == 0 && SLOTS % kThreads == 0, "windows of whole steps, whole copy passes");
  static_assert((LO ? 3 : 2) * TBYTES + 2 * MQ * 4 + MQ * 2 <= kLdsMax, "query tiles exceed LDS");
};

template <int KZ, int KY, int KX, int ZK, bool NORM, bool LO>
__global__ void __launch_bounds__(64 * ZK, 1) na3d_bwd_dkdv_d128_kernel(Args a) {
  using C = KvCfg<KZ, KY, KX, ZK, LO>;
  constexpr int kThreads = C::kThreads;
  __shared__ __attribute__((aligned(16))) char tQ[C::TBYTES];
  __shared__ __attribute__((aligned(16))) char tG[C::TBYTES];
  __shared__ __attribute__((aligned(16))) char tL[LO ? C::TBYTES : 16];  // low term of dO (LO)
  __shared__ __attribute__((aligned(16))) float sL[C::MQ];
  __shared__ __attribute__((aligned(16))) float sD[C::MQ];
  __shared__ __attribute__((aligned(16))) unsigned short smask[C::MQ];

  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int xb = bid % a.n_xb;
  const int yb = (bid / a.n_xb) % a.n_yb;
  const int zb = (bid / (a.n_xb * a.n_yb)) % a.n_zb;
  const int bh = bid / (a.n_xb * a.n_yb * a.n_zb);
  const int b = bh / a.heads;
  const int H = a.H, W = a.W, Z = a.Z;
  const int y0 = 4 * yb, x0 = 4 * xb, z0 = ZK * zb;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;

  // the query box of the block (the same on every level)
  const int qy0 = inv_lo(y0, KY), qy1 = inv_hi(min(y0 + 3, H - 1), H, KY);
  const int qx0 = inv_lo(x0, KX), qx1 = inv_hi(min(x0 + 3, W - 1), W, KX);
  const int nqx = qx1 - qx0 + 1;
  const int nq = (qy1 - qy0 + 1) * nqx;
  const int npairs = (nq + 31) >> 5;
  const int64_t HW = (int64_t)H * W;
  const int64_t bh_base = (int64_t)bh * Z * HW;
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * kCS4 : nullptr;

  // window-mask bits per box query (bit 4 dy + dx: key (y0+dy, x0+dx) in the
  // query's (y, x) window); LSE / D entries past the box are zero
  for (int u = tid; u < C::MQ; u += kThreads) {
    unsigned bits = 0;
    if (u < nq) {
      const int qy = qy0 + u / nqx, qx = qx0 + u % nqx;
      const int wy = win_start(qy, H, KY), wx = win_start(qx, W, KX);
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const int yy = y0 + (t >> 2), xx = x0 + (t & 3);
        if (yy >= wy && yy < wy + KY && xx >= wx && xx < wx + KX) bits |= 1u << t;
      }
    } else {
      sL[u] = 0.f;
      sD[u] = 0.f;
    }
    smask[u] = (unsigned short)bits;
  }
  // copy map of window w: tile row r = s / 16 holds box query u = w RW + r,
  // slot column s % 16 holds data column (s % 16) ^ sigma(r) (sigma of the row
  // inside its 32-row step, which is also sigma(u)); Q and dO share it.
  // goff: element offset inside a level; -1: a row past the box but inside the
  // last 32-query step (written as zeros); -2: past that (untouched)
  int goff[C::NW][C::IT];
#pragma unroll
  for (int w = 0; w < C::NW; ++w)
#pragma unroll
    for (int it = 0; it < C::IT; ++it) {
      const int s = it * kThreads + tid, r = s >> 4, u = w * C::RW + r, dc = (s & 15) ^ rswz(r);
      goff[w][it] = u < nq ? ((qy0 + u / nqx) * W + qx0 + u % nqx) * kD + dc * 8 : (u < npairs * 32 ? -1 : -2);
    }
  int soff[C::IS];
  float pl[C::IS], pd[C::IS];
#pragma unroll
  for (int is = 0; is < C::IS; ++is) {
    const int u = is * kThreads + tid;
    soff[is] = u < nq ? (qy0 + u / nqx) * W + qx0 + u % nqx : -1;
    pl[is] = 0.f;
    pd[is] = 0.f;
  }

  // stage window w of level p (and, with the first window, its LSE / D)
  auto issue = [&](int p, int w) {
    const int64_t lev = bh_base + (int64_t)p * HW;
    const uint16_t* qp = a.q + lev * kD;
    const uint16_t* gp = a.dout + lev * kD;
    const uint16_t* lp = LO ? a.dout_lo + lev * kD : nullptr;
#pragma unroll
    for (int it = 0; it < C::IT; ++it) {
      const int o = goff[w][it];
      if (o >= 0) {
        copy16_to_lds(qp + o, tQ + (it * kThreads + wave * 64) * 16);
        copy16_to_lds(gp + o, tG + (it * kThreads + wave * 64) * 16);
        if constexpr (LO) copy16_to_lds(lp + o, tL + (it * kThreads + wave * 64) * 16);
      } else if (o == -1) {  // rows past the box inside the last step: zeros
        const uint4 z = make_uint4(0u, 0u, 0u, 0u);
        st16(tQ + (it * kThreads + tid) * 16, z);
        st16(tG + (it * kThreads + tid) * 16, z);
        if constexpr (LO) st16(tL + (it * kThreads + tid) * 16, z);
      }
    }
    if (w == 0) {
#pragma unroll
      for (int is = 0; is < C::IS; ++is) {
        if (soff[is] < 0) continue;
        pl[is] = a.lse[lev + soff[is]];
        pd[is] = a.dvec[lev + soff[is]];
      }
    }
  };
  // wait for this thread's copies, rotate its own Q slots in place, store its
  // LSE / D entries (first window)
  auto finish = [&](int w) {
    __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
    for (int it = 0; it < C::IT; ++it) {
      const int o = goff[w][it];
      if (o < 0) continue;
      char* ad = tQ + (it * kThreads + tid) * 16;
      const uint4 x = ld16(ad);
      // (a query row is 16 consecutive slots, all in or all past the box)
      const float mul = NORM ? __builtin_amdgcn_rsqf(sum_over_16_lanes(sumsq8(x, 0.f)) * (1.f / kD) + a.eps) : 1.f;
      if (csb) {  // packed float16 rotation, phases converted from the float32 table
        const float4* pp = csb + (o >> 7) * kCS4 + ((o & 127) >> 2);
        const float4 p0 = pp[0], p1 = pp[1];
        st16(ad, rotate8h_pk(x, make_uint4(pack2h_rne(p0.x, p0.y), pack2h_rne(p0.z, p0.w), pack2h_rne(p1.x, p1.y),
                                           pack2h_rne(p1.z, p1.w)), mul));
      } else {
        st16(ad, scale8h(x, mul));
      }
    }
    if (w == 0) {
#pragma unroll
      for (int is = 0; is < C::IS; ++is) {
        if (soff[is] < 0) continue;
        const int u = is * kThreads + tid;
        sL[u] = pl[is] * kLog2e;
        sD[u] = -pd[is];
      }
    }
  };

  // this wave's keys: K~ (times scale log2 e) and V as B operands
  const int ky_raw = y0 + (qn >> 2), kx_raw = x0 + (qn & 3);
  const int ky = min(ky_raw, H - 1), kx = min(kx_raw, W - 1);
  const int kz = z0 + wave;
  const bool wave_on = kz < Z;
  const int64_t ktok = bh_base + (int64_t)min(kz, Z - 1) * HW + (int64_t)ky * W + kx;
  const float4* csk = csb ? csb + ((int64_t)ky * W + kx) * kCS4 : nullptr;
  f16x8 kf[4];
  bf16x8 vf[4];
  float rk = 1.f;  // QK RMSNorm factor of this lane's key
  {
    const uint4* src = reinterpret_cast<const uint4*>(a.k + ktok * kD);
    const uint4* vs = reinterpret_cast<const uint4*>(a.v + ktok * kD);
    uint4 x[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) x[kk] = src[4 * kk + g];
    if constexpr (NORM) {  // the 4 lanes of a key row hold its 128 values
      float ss = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) ss = sumsq8(x[kk], ss);
      rk = __builtin_amdgcn_rsqf(sum_over_rows(ss) * (1.f / kD) + a.eps);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const float mul = a.qscale * rk;
      const uint4 r = csk ? rotate8h(x[kk], csk[8 * kk + 2 * g], csk[8 * kk + 2 * g + 1], mul) : scale8h(x[kk], mul);
      kf[kk] = __builtin_bit_cast(f16x8, r);
      vf[kk] = __builtin_bit_cast(bf16x8, vs[4 * kk + g]);
    }
  }
  f32x4 accK[8], accV[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    accK[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    accV[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  int ex = kMinExp;

  // A rows: chunk c, row 16c + qn, column g (k-step kk: xor 64 kk bytes)
  const uint32_t aoff = qn * kRow + ((g ^ rswz(qn)) << 4);
  // transpose reads: row 32 st + 4g + qn/4 (+16 for the second chunk), the 8
  // bytes holding elements 4 (qn % 4) .. +3 of each 16-wide d block (xor 32 t)
  const int trow = 4 * g + (qn >> 2);
  const uint32_t toff = trow * kRow + ((((qn >> 1) & 1) ^ rswz(trow)) << 4) + 8 * (qn & 1);

  auto compute = [&](int w) {
    const int st0 = w * (C::RW / 32), st1 = min(npairs, st0 + C::RW / 32);
    for (int st = st0; st < st1; ++st) {
      f32x4 x[2], y[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = 2 * st + h;                 // chunk of the box (mask, LSE, D)
        const int cl = 2 * (st - st0) + h;        // chunk of the staged window
        const char* rq = tQ + cl * (16 * kRow);
        const char* rg = tG + cl * (16 * kRow);
        const int u4 = 16 * c + 4 * g;
        const float4 l4 = *reinterpret_cast<const float4*>(sL + u4);
        const float4 d4 = *reinterpret_cast<const float4*>(sD + u4);
        const uint2 m4 = *reinterpret_cast<const uint2*>(smask + u4);
        f32x4 xs;
        xs[0] = ((m4.x >> qn) & 1u) ? -l4.x : -INFINITY;
        xs[1] = ((m4.x >> (16 + qn)) & 1u) ? -l4.y : -INFINITY;
        xs[2] = ((m4.y >> qn) & 1u) ? -l4.z : -INFINITY;
        xs[3] = ((m4.y >> (16 + qn)) & 1u) ? -l4.w : -INFINITY;
        f32x4 ys = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const f16x8 qa = __builtin_bit_cast(f16x8, ld16(rq + (aoff ^ (64u * kk))));
          const bf16x8 ga = __builtin_bit_cast(bf16x8, ld16(rg + (aoff ^ (64u * kk))));
          xs = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa, kf[kk], xs, 0, 0, 0);
          ys = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ga, vf[kk], ys, 0, 0, 0);
          if constexpr (LO) {
            const bf16x8 la = __builtin_bit_cast(bf16x8, ld16(tL + cl * (16 * kRow) + (aoff ^ (64u * kk))));
            ys = __builtin_amdgcn_mfma_f32_16x16x32_bf16(la, vf[kk], ys, 0, 0, 0);
          }
        }
        x[h] = xs;
        y[h] = ys;
      }
      float my = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
        my = fmaxf(fmaxf(my, fmaxf(fabsf(y[h][0]), fabsf(y[h][1]))), fmaxf(fabsf(y[h][2]), fabsf(y[h][3])));
      my = max_over_rows(my);
      const int e = max(__builtin_amdgcn_frexp_expf(my), kMinExp);
      if (__any(e > ex)) {  // the bound grew: rescale the dK~ accumulator exactly
        const int en = max(ex, e);
        const float f = __builtin_amdgcn_ldexpf(1.f, ex - en);
#pragma unroll
        for (int t = 0; t < 8; ++t) accK[t] *= f;
        ex = en;
      }
      const float sc = __builtin_amdgcn_ldexpf(1.f, 15 - ex);
      uint32_t pb[2][2], db[2][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float p0 = __builtin_amdgcn_exp2f(x[h][0]), p1 = __builtin_amdgcn_exp2f(x[h][1]);
        const float p2 = __builtin_amdgcn_exp2f(x[h][2]), p3 = __builtin_amdgcn_exp2f(x[h][3]);
        pb[h][0] = pack2(p0, p1);
        pb[h][1] = pack2(p2, p3);
        db[h][0] = pack2h_rne(p0 * sc * y[h][0], p1 * sc * y[h][1]);
        db[h][1] = pack2h_rne(p2 * sc * y[h][2], p3 * sc * y[h][3]);
      }
      const bf16x8 pf = __builtin_bit_cast(bf16x8, make_uint4(pb[0][0], pb[0][1], pb[1][0], pb[1][1]));
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(db[0][0], db[0][1], db[1][0], db[1][1]));
      const char* tq0 = tQ + (st - st0) * (32 * kRow);
      const char* tg0 = tG + (st - st0) * (32 * kRow);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t o0 = toff ^ (32u * t);
        const uint2 g_lo = __builtin_bit_cast(uint2, tr_read(tg0 + o0));
        const uint2 g_hi = __builtin_bit_cast(uint2, tr_read(tg0 + 16 * kRow + o0));
        const bf16x8 gt = __builtin_bit_cast(bf16x8, make_uint4(g_lo.x, g_lo.y, g_hi.x, g_hi.y));
        accV[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gt, pf, accV[t], 0, 0, 0);
        if constexpr (LO) {
          const char* tl0 = tL + (st - st0) * (32 * kRow);
          const uint2 l_lo = __builtin_bit_cast(uint2, tr_read(tl0 + o0));
          const uint2 l_hi = __builtin_bit_cast(uint2, tr_read(tl0 + 16 * kRow + o0));
          const bf16x8 lt = __builtin_bit_cast(bf16x8, make_uint4(l_lo.x, l_lo.y, l_hi.x, l_hi.y));
          accV[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lt, pf, accV[t], 0, 0, 0);
        }
        const uint2 q_lo = __builtin_bit_cast(uint2, tr_read(tq0 + o0));
        const uint2 q_hi = __builtin_bit_cast(uint2, tr_read(tq0 + 16 * kRow + o0));
        const f16x8 qt = __builtin_bit_cast(f16x8, make_uint4(q_lo.x, q_lo.y, q_hi.x, q_hi.y));
        accK[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qt, df, accK[t], 0, 0, 0);
      }
    }
  };
  auto active = [&](int p) {
    const int zs = win_start(p, Z, KZ);
    return wave_on && kz >= zs && kz < zs + KZ;
  };

  // query levels that see the block's key levels, one at a time
  const int zk_last = min(z0 + ZK, Z) - 1;
  const int p_lo = inv_lo(z0, KZ), p_hi = inv_hi(zk_last, Z, KZ);
  const int nwin = (npairs * 32 + C::RW - 1) / C::RW;
  for (int p = p_lo; p <= p_hi; ++p)
    for (int w = 0; w < nwin; ++w) {
      issue(p, w);
      finish(w);
      __syncthreads();  // the window is published
      if (active(p)) compute(w);
      __syncthreads();  // every read of the window is done before the next copy
    }

  // dV, and dK = R^T (scale 2^(E-15) dK~); the lane holds d = 16t + 4g + i.
  // With QK RMSNorm that is the gradient of k^ = r k, carried back through the
  // norm: dk = r (dk^ - k^ mean(dk^ k^)), k^ from the raw row in float32.
  const float f = a.scale * __builtin_amdgcn_ldexpf(1.f, ex - 15);
  f32x4 xk[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    xk[t] = accK[t] * f;
    if (csk) {
      const float4 p = csk[4 * t + g];  // pairs 8t+2g and 8t+2g+1
      const float r0 = fmaf(xk[t][0], p.x, xk[t][1] * p.y), r1 = fmaf(xk[t][1], p.x, -xk[t][0] * p.y);
      const float r2 = fmaf(xk[t][2], p.z, xk[t][3] * p.w), r3 = fmaf(xk[t][3], p.z, -xk[t][2] * p.w);
      xk[t] = f32x4{r0, r1, r2, r3};
    }
  }
  if constexpr (NORM) {
    const uint2* kr = reinterpret_cast<const uint2*>(a.k + ktok * kD);
    f32x4 kh[8];
    float c = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint2 w = kr[4 * t + g];
      kh[t] = f32x4{lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y)} * rk;
#pragma unroll
      for (int i = 0; i < 4; ++i) c = fmaf(xk[t][i], kh[t][i], c);
    }
    c = sum_over_rows(c) * (1.f / kD);
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) xk[t][i] = rk * fmaf(-kh[t][i], c, xk[t][i]);
  }
  if (!wave_on || ky_raw >= H || kx_raw >= W) return;
  uint2* dkd = reinterpret_cast<uint2*>(a.dk + ktok * kD);
  uint2* dvd = reinterpret_cast<uint2*>(a.dv + ktok * kD);
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    dvd[4 * t + g] = make_uint2(pack2(accV[t][0], accV[t][1]), pack2(accV[t][2], accV[t][3]));
    dkd[4 * t + g] = make_uint2(pack2(xk[t][0], xk[t][1]), pack2(xk[t][2], xk[t][3]));
  }
}

// widest query box (per axis) over the 4-wide key blocks of an axis of extent L
int max_box(int L, int k) {
  int mx = 0;
  for (int j0 = 0; j0 < L; j0 += 4) {
    const int n = inv_hi(std::min(j0 + 3, L - 1), L, k) - inv_lo(j0, k) + 1;
    mx = std::max(mx, n);
  }
  return mx;
}

bool supported(const strata_na3d_desc& d) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  if (!(d.kz == 9 && d.ky == 9 && d.kx == 9)) return false;
  return (int64_t)d.H * d.W * kD < (int64_t)1 << 31;  // int32 offsets inside a level
}

Args make_args(const strata_na3d_desc& d, const void* q, const void* k, const void* v, const float* cs,
               const void* dout, const float* lse, const float* dvec) {
  Args a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse = lse;
  a.dvec = dvec;
  a.heads = d.heads;
  a.Z = d.Z;
  a.H = d.H;
  a.W = d.W;
  a.scale = d.scale;
  a.qscale = d.scale * kLog2e;
  return a;
}

}  // namespace

bool launch_na3d_bwd_dq_d128(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                             const void* v, const float* cs, const void* dout, const float* lse,
                             const float* dvec, void* dq, hipStream_t s) {
  if (!supported(d)) return false;
  Args a = make_args(d, q, k, v, cs, dout, lse, dvec);
  a.dq = static_cast<uint16_t*>(dq);
  a.eps = o.eps;
  a.dout_lo = static_cast<const uint16_t*>(o.dout_lo);
  // two query levels per wave, one with the two-term dO (its low term's
  // fragments would not fit beside two levels' state)
  const int zq = o.dout_lo ? 1 : 2;
  a.n_zb = (d.Z + zq - 1) / zq;
  a.n_yb = (d.H + kQBY - 1) / kQBY;
  a.n_xb = (d.W + kQBX - 1) / kQBX;
  const int64_t blocks = (int64_t)d.B * d.heads * a.n_zb * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  const dim3 grid((unsigned)blocks), block(kQThreads);
  if (o.qk_norm && o.dout_lo)
    hipLaunchKernelGGL((na3d_bwd_dq_d128_kernel<9, 9, 9, 1, true, true>), grid, block, 0, s, a);
  else if (o.qk_norm)
    hipLaunchKernelGGL((na3d_bwd_dq_d128_kernel<9, 9, 9, 2, true, false>), grid, block, 0, s, a);
  else if (o.dout_lo)
    hipLaunchKernelGGL((na3d_bwd_dq_d128_kernel<9, 9, 9, 1, false, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((na3d_bwd_dq_d128_kernel<9, 9, 9, 2, false, false>), grid, block, 0, s, a);
  return true;
}

bool launch_na3d_bwd_dkdv_d128(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                               const void* v, const float* cs, const void* dout, const float* lse,
                               const float* dvec, void* dk, void* dv, hipStream_t s) {
  if (!supported(d)) return false;
  constexpr int ZK = 8;
  using C = KvCfg<9, 9, 9, ZK, false>;
  if (max_box(d.H, 9) > C::MQY || max_box(d.W, 9) > C::MQX) return false;
  Args a = make_args(d, q, k, v, cs, dout, lse, dvec);
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.eps = o.eps;
  a.n_zb = (d.Z + ZK - 1) / ZK;
  a.n_yb = (d.H + 3) / 4;
  a.n_xb = (d.W + 3) / 4;
  const int64_t blocks = (int64_t)d.B * d.heads * a.n_zb * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  a.dout_lo = static_cast<const uint16_t*>(o.dout_lo);
  const dim3 grid((unsigned)blocks), block(C::kThreads);
  if (o.qk_norm && o.dout_lo)
    hipLaunchKernelGGL((na3d_bwd_dkdv_d128_kernel<9, 9, 9, ZK, true, true>), grid, block, 0, s, a);
  else if (o.qk_norm)
    hipLaunchKernelGGL((na3d_bwd_dkdv_d128_kernel<9, 9, 9, ZK, true, false>), grid, block, 0, s, a);
  else if (o.dout_lo)
    hipLaunchKernelGGL((na3d_bwd_dkdv_d128_kernel<9, 9, 9, ZK, false, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((na3d_bwd_dkdv_d128_kernel<9, 9, 9, ZK, false, false>), grid, block, 0, s, a);
  return true;
}

}  // namespace strata

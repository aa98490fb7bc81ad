// MFMA neighbourhood-attention forward for head_dim 128 (the decoder's NA3D,
// App. B.3: one head of 128 channels, window 9 x 9 x 9), bf16 in/out,
// StereoRoPE fused into the Q/K loads.
//
// Same decomposition and arithmetic as the head_dim-64 query-stationary kernel:
// a workgroup takes an 8 x 8 block of (y, x) query positions and ZQ query
// levels of one (tile, head) with 8 waves; a wave takes a 4 x 4 sub-block on
// ZQ/2 of the levels (waves 0-3 the even ones, 4-7 the odd ones).  Per (query
// level, key level):
//   S^T (16 keys x 16 queries) = K . Q^T   four 16x16x32 float16 MFMAs per
//                                          16-key chunk (128 = 4 x 32), the
//                                          accumulator seeded with the mask;
//   online softmax against a lazy reference (from 0; it moves only past 2^8
//   growth, or below -2^6 on the first key level), row sums of the packed
//   bf16 weights by v_dot2c;
//   O^T (128 d x 16 queries) += V^T . P^T  eight 16-row bf16 MFMA tiles, V^T
//                                          fragments from the LDS transpose
//                                          read.
// What head_dim 128 changes: one key level of the 16 x 16 key box is 64 KB of
// float16 K (256-byte rows, 16-byte columns XOR-swizzled as for head_dim 64)
// and 72 KB of bf16 V (288-byte rows: 256 + a 32-byte pad that spreads the
// transpose reads), so the tiles are single-buffered: each key level is copied
// (direct to LDS), rotated in place in packed float16 by the thread whose
// copies brought it -- phases converted from the float32 table, which stays
// in the L2 -- published by a
// barrier, computed, and retired by a second barrier before the next copy.
// The rotated Q and K are float16 (logit scale and log2(e) folded into Q); P
// and V are bf16.  Options (App. B.5): QK RMSNorm scales each query and key by
// (mean square + eps)^(-1/2) in float32 before the float16 rounding -- a
// query's factor from the 4 lanes holding its row, a key's from the 16
// consecutive lanes whose copies brought it; the sigmoid gate (one logit per
// token-head or per channel) multiplies the normalised output at the store.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

namespace strata {
namespace {

using namespace mfma;

constexpr int kBY = 8, kBX = 8;
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kD = 128;
constexpr int kKRow = 256;  // LDS bytes per key row of K (16 columns of 16 bytes, swizzled)
constexpr int kVRow = 288;  // LDS bytes per key row of V (256 + 32 pad)
constexpr int kCS4 = kD / 4;  // float4 entries of the phase table per position (two pairs each)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLazy = 8.0f;   // move the softmax reference only when a logit exceeds it by > 2^8
constexpr float kLow = -64.0f;  // ... or down, on a level's first key level

template <int KZ, int KY, int KX, int ZQ>
struct Cfg {
  static constexpr int LY = kBY + KY - 1, LX = kBX + KX - 1;  // staged key box per level
  static constexpr int NUY = 3 + KY, NUX = 3 + KX;            // key box of a 4x4 sub-block
  static constexpr int NU = NUY * NUX;
  static constexpr int NC = (NU + 15) / 16;                   // 16-key chunks
  static constexpr int NS = (NC + 1) / 2;                     // 32-key P.V steps
  static constexpr int KEYS = LY * LX;
  static constexpr int KSLOTS = KEYS * (kKRow / 16), VSLOTS = KEYS * (kVRow / 16);
  static constexpr int KBYTES = KEYS * kKRow, VBYTES = KEYS * kVRow;
  static constexpr int ITK = (KSLOTS + kThreads - 1) / kThreads;
  static constexpr int ITV = (VSLOTS + kThreads - 1) / kThreads;
  static constexpr int QL = ZQ / 2;
  static_assert(ZQ % 2 == 0, "ZQ must be even");
  static_assert(KBYTES + VBYTES <= 160 * 1024, "key tiles exceed LDS");
};

struct Args {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;  // [B, H, W, 32] float4 = two (cos, sin) pairs; nullptr: no rotation
  uint16_t* out;
  float* lse;        // optional
  int heads, Z, H, W;
  int n_zb, n_yb, n_xb;
  float qscale;      // scale * log2(e)
  float eps;         // QK RMSNorm
  const uint16_t* gate;
  int gate_dim;
};

template <int KZ, int KY, int KX, int ZQ, bool NORM, bool GATE>
__global__ void __launch_bounds__(kThreads, 1) na3d_fwd_d128_kernel(Args a) {
  using C = Cfg<KZ, KY, KX, ZQ>;
  __shared__ __attribute__((aligned(16))) char tK[C::KBYTES];
  __shared__ __attribute__((aligned(16))) char tV[C::VBYTES];

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

  // ---- per-lane tile addresses and window mask (the same at every level) ---
  uint32_t kaddr[C::NC], vaddr[C::NC];
  f32x4 bias[C::NC];
#pragma unroll
  for (int c = 0; c < C::NC; ++c) {
    {  // K fragment: row = key 16c + qn, column g (k-step kk: column g + 4kk, i.e. xor 64 kk bytes)
      const int key = key_row(16 * c + qn);
      kaddr[c] = key * kKRow + ((g ^ kswz(key)) << 4);
    }
    // V^T transpose read: source row = key 16c + 4g + qn/4, 8 bytes at d = 4 (qn % 4) (+ 16 d per tile)
    vaddr[c] = key_row(16 * c + 4 * g + (qn >> 2)) * kVRow + (qn & 3) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = 16 * c + 4 * g + i;
      const int ky = uy0 + u / C::NUX, kx = ux0 + u % C::NUX;
      const bool ok = u < C::NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX;
      bias[c][i] = ok ? 0.f : -INFINITY;
    }
  }

  // ---- direct-to-LDS copy map: element offsets inside a key level, -1 for --
  // ---- pad and past-the-end slots ------------------------------------------
  int goffK[C::ITK], goffV[C::ITV];
#pragma unroll
  for (int it = 0; it < C::ITK; ++it) {
    const int s = it * kThreads + tid, key = s >> 4, c = (s & 15) ^ kswz(key);
    const int gy = min(ty0 + key / C::LX, H - 1), gx = min(tx0 + key % C::LX, W - 1);
    goffK[it] = s < C::KSLOTS ? (gy * W + gx) * kD + c * 8 : -1;
  }
#pragma unroll
  for (int it = 0; it < C::ITV; ++it) {
    const int s = it * kThreads + tid, key = s / 18, c = s - key * 18;
    const int gy = min(ty0 + key / C::LX, H - 1), gx = min(tx0 + key % C::LX, W - 1);
    goffV[it] = (s < C::VSLOTS && c < 16) ? (gy * W + gx) * kD + c * 8 : -1;
  }
  const int64_t HW = (int64_t)H * W;
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * kCS4 : nullptr;
  const int64_t bh_base = (int64_t)bh * Z * HW;

  auto issue_copy = [&](int p) {
    const uint16_t* kp = a.k + (bh_base + (int64_t)p * HW) * kD;
    const uint16_t* vp = a.v + (bh_base + (int64_t)p * HW) * kD;
#pragma unroll
    for (int it = 0; it < C::ITK; ++it)
      if (goffK[it] >= 0) copy16_to_lds(kp + goffK[it], tK + (it * kThreads + wave * 64) * 16);
#pragma unroll
    for (int it = 0; it < C::ITV; ++it)
      if (goffV[it] >= 0) copy16_to_lds(vp + goffV[it], tV + (it * kThreads + wave * 64) * 16);
  };
  // rotate (or convert) this thread's K slots in place, bf16 -> float16; its own
  // copies land in its own slots, so its own wait suffices
  auto rotate_k = [&]() {
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      const int o = goffK[it];
      if (o < 0) continue;
      char* ad = tK + (it * kThreads + tid) * 16;
      uint4 x = ld16(ad);
      // (a key row is 16 consecutive slots, all in the tile: every lane of the row takes part)
      const float mul = NORM ? __builtin_amdgcn_rsqf(sum_over_16_lanes(sumsq8(x, 0.f)) * (1.f / kD) + a.eps) : 1.f;
      if (csb) {  // packed float16 rotation, phases of pairs 4c..4c+3 of the key's position
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

  // ---- queries: load, rotate, scale (float16 B operands of K.Q^T) ----------
  f16x8 qf[C::QL][4];
  float m[C::QL], l[C::QL];
  bool mset[C::QL];  // wave-uniform: the reference m has moved from 0 somewhere in the wave
  f32x4 o[C::QL][8];
  const float4* csq = csb ? csb + ((int64_t)qy * W + qx) * kCS4 : nullptr;
#pragma unroll
  for (int j = 0; j < C::QL; ++j) {
    const int zq = min(z0 + grp + 2 * j, Z - 1);
    const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
    const uint4* src = reinterpret_cast<const uint4*>(a.q + tok * kD);
    uint4 x[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) x[kk] = src[4 * kk + g];  // d = 32 kk + 8 g .. + 7
    float mul = a.qscale;
    if constexpr (NORM) {  // the 4 lanes of a query row hold its 128 values
      float ss = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) ss = sumsq8(x[kk], ss);
      mul *= __builtin_amdgcn_rsqf(sum_over_rows(ss) * (1.f / kD) + a.eps);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint4 r = csq ? rotate8h(x[kk], csq[8 * kk + 2 * g], csq[8 * kk + 2 * g + 1], mul) : scale8h(x[kk], mul);
      qf[j][kk] = __builtin_bit_cast(f16x8, r);
    }
    m[j] = 0.f;
    l[j] = 0.f;
    mset[j] = false;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // one (query level j, key level) update from the staged tiles; `first`: the
  // query level's first key level (nothing accumulated yet)
  auto update = [&](int j, bool first) {
    f32x4 s[C::NC];
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      f32x4 acc = bias[c];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const f16x8 kf = __builtin_bit_cast(f16x8, ld16(tK + (kaddr[c] ^ (64u * kk))));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[j][kk], acc, 0, 0, 0);
      }
      s[c] = acc;
    }
    float mx = fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3]));
#pragma unroll
    for (int c = 1; c < C::NC; ++c) mx = fmaxf(fmaxf(mx, fmaxf(s[c][0], s[c][1])), fmaxf(s[c][2], s[c][3]));
    mx = max_over_rows(mx);
    // lazy reference: starts at 0, moves past 2^kLazy growth or, on the first
    // key level, below kLow; while 0 across the wave nothing is subtracted
    const bool move = mx > m[j] + kLazy || (first && mx < kLow);
    if (__any(move)) {  // rare: move the reference, rescale
      const float mn = move ? mx : m[j];
      if (!first) {  // nothing accumulated before the first key level
        const float alpha = __builtin_amdgcn_exp2f(m[j] - mn);
        l[j] *= alpha;
#pragma unroll
        for (int t = 0; t < 8; ++t) o[j][t] *= alpha;
      }
      m[j] = mn;
      mset[j] = true;
    }
    if (mset[j]) {
#pragma unroll
      for (int c = 0; c < C::NC; ++c) s[c] -= m[j];
    }
    uint32_t pk[C::NC][2];
    float ls = l[j];
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      pk[c][0] = pack2(__builtin_amdgcn_exp2f(s[c][0]), __builtin_amdgcn_exp2f(s[c][1]));
      pk[c][1] = pack2(__builtin_amdgcn_exp2f(s[c][2]), __builtin_amdgcn_exp2f(s[c][3]));
      ls = psum8(pk[c][0], pk[c][1], ls);
    }
    l[j] = ls;
#pragma unroll
    for (int st = 0; st < C::NS; ++st) {
      const int c0 = 2 * st, c1 = 2 * st + 1;
      const bool two = c1 < C::NC;
      const bf16x8 pf = __builtin_bit_cast(
          bf16x8, make_uint4(pk[c0][0], pk[c0][1], two ? pk[two ? c1 : c0][0] : 0u, two ? pk[two ? c1 : c0][1] : 0u));
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const i16x4 lo = tr_read(tV + vaddr[c0] + 32 * t);
        const i16x4 hi = two ? tr_read(tV + vaddr[two ? c1 : c0] + 32 * t) : i16x4{0, 0, 0, 0};
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        const bf16x8 vf = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
        o[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[j][t], 0, 0, 0);
      }
    }
  };

  // ---- key levels needed by the block's query levels, one at a time --------
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
      const int zq = z0 + grp + 2 * j;
      if (zq >= Z) continue;
      const int zs = win_start(zq, Z, KZ);
      if (p < zs || p >= zs + KZ) continue;
      update(j, p == zs);
    }
    __syncthreads();  // every read of the level is done before the next copy
  }

  // ---- normalise and store ---------------------------------------------------
  const bool in_grid = qy_raw < H && qx_raw < W;
#pragma unroll
  for (int j = 0; j < C::QL; ++j) {
    const int zq = z0 + grp + 2 * j;
    const float lt = sum_over_rows(l[j]);
    if (zq >= Z || !in_grid) continue;
    float inv = 1.f / lt;
    const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
    uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
    if constexpr (GATE)
      if (a.gate_dim == 1) inv *= sigmoid_fast(bf16_to_f32(a.gate[tok]));
#pragma unroll
    for (int t = 0; t < 8; ++t) {  // d = 16t + 4g + i
      f32x4 r = o[j][t] * inv;
      if constexpr (GATE)
        if (a.gate_dim != 1) r *= sigmoid4_bf16(reinterpret_cast<const uint2*>(a.gate + tok * kD)[4 * t + g]);
      dst[4 * t + g] = make_uint2(pack2(r[0], r[1]), pack2(r[2], r[3]));
    }
    if (a.lse && g == 0) a.lse[tok] = (m[j] + __log2f(lt)) * kLn2;
  }
}

}  // namespace

bool launch_na3d_fwd_d128(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                          const void* v, const float* cs, void* out, float* lse, hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  if (!(d.kz == 9 && d.ky == 9 && d.kx == 9)) return false;
  if ((int64_t)d.H * d.W * kD >= (int64_t)1 << 31) return false;  // int32 offsets inside a key level
  constexpr int ZQ = 2;
  Args a = {};
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
  a.eps = o.eps;
  a.gate = static_cast<const uint16_t*>(o.gate);
  a.gate_dim = o.gate_dim;
  const int64_t blocks = (int64_t)d.B * d.heads * a.n_zb * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  const dim3 grid((unsigned)blocks), block(kThreads);
  if (o.qk_norm && o.gate)
    hipLaunchKernelGGL((na3d_fwd_d128_kernel<9, 9, 9, ZQ, true, true>), grid, block, 0, s, a);
  else if (o.qk_norm)
    hipLaunchKernelGGL((na3d_fwd_d128_kernel<9, 9, 9, ZQ, true, false>), grid, block, 0, s, a);
  else if (o.gate)
    hipLaunchKernelGGL((na3d_fwd_d128_kernel<9, 9, 9, ZQ, false, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((na3d_fwd_d128_kernel<9, 9, 9, ZQ, false, false>), grid, block, 0, s, a);
  return true;
}

}  // namespace strata

// Neighbourhood-attention forward for gfx950 with a level sweep over a group of
// query levels: odd windows (KZ, KY, KX) up to 9 x 9 x 9 (dispatched for 3x7x7
// and 5x9x9), any number of levels, head_dim 64, bf16 in/out, StereoRoPE fused
// into the Q/K loads (Sec. 3.2, 3.3).
//
// Work decomposition
//   workgroup : one tile, an 8 x 8 block of (y, x) query positions, a group of
//               G consecutive query levels, and a run of heads processed one
//               after the other; 4 waves (one per SIMD), one workgroup per CU.
//   wave      : a 4 x 4 (y, x) sub-block = 16 queries, on the G levels of the
//               group (G accumulators in registers for the whole head).
//   key sweep : per head the workgroup walks the key levels that the group's
//               query windows reach, each once (G + KZ - 1 of them for an
//               interior group).  K and V of the (8 + KY - 1) x (8 + KX - 1)
//               key box of a level are copied global -> LDS by the direct copy,
//               the K pieces rotated in place (StereoRoPE in packed float16,
//               phases of the box staged once in LDS, at half length so that a
//               rotated pair never overflows float16) and the V pieces converted
//               to float16.  A wave reads the K and V
//               fragments of its sub-block's (3 + KY) x (3 + KX) key box once per
//               key level and applies them to every query level of the group
//               whose window holds that key level (a wave-uniform test: the
//               border-clamped windows make the pattern depend on the group's
//               place in the column).
//   buffers   : NBUF = 1 (what both dispatched windows use): after every wave
//               has its fragments in registers a barrier frees the buffer and
//               the copies of the next level go into it (two barriers per
//               level).  NBUF = 2 (the next level copied into a second buffer,
//               the key loop unrolled by two so the buffers stay distinct LDS
//               objects) does not fit 16 x 16 key boxes and, at 3x7x7, spills
//               registers with the loop body duplicated.
//
// Per (query level, key level) -- the same update as the 8-level sweep:
//   S^T (16 keys x 16 queries) = K . Q^T   16x16x32 float16 MFMAs seeded with
//                                         the window mask (0 or -inf);
//   lazy softmax reference m (moves only when a logit exceeds it by 15, or on
//   a level's first key level when nothing reaches -8); P = exp2(S^T - m) as
//   float16 (2^-8 <= max P <= 2^15); O^T += V^T . P^T and the row sums
//   L += 1 . P^T on float16 MFMAs (bf16 weights would cost up to ~2% of the
//   output RMS in the worst outputs).
// The queries of all G levels are rotated once per head (float32 phases, the
// scale times 2 log2(e), one float16 rounding); their rows for the next head
// are loaded during the last key level.
//
// Options (App. B.5): QK RMSNorm scales every query and key in float32 before
// its float16 rounding; the sigmoid gate multiplies the normalised output.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

namespace strata {
namespace {

using namespace mfma;

constexpr int kThreads = 256;
constexpr int kD = 64;
constexpr int kKRow = 128, kVRow = 160;  // LDS bytes per key row (K swizzled; V padded)
constexpr int kLdsMax = 160 * 1024;
constexpr float kLazy = 15.0f;   // m moves up when a logit exceeds it by 15 (P <= 2^15)
constexpr float kLow = -8.0f;    // ... or down, on a level's first key level (max P >= 2^-8)
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLog2e = 1.4426950408889634f;

template <int KZ, int KY, int KX, int G, int NBUF>
struct LsgCfg {
  static constexpr int LY = 8 + KY - 1, LX = 8 + KX - 1;    // staged key box per level
  static constexpr int NUY = 3 + KY, NUX = 3 + KX, NU = NUY * NUX;  // key box of a 4x4 sub-block
  static constexpr int NC = (NU + 15) / 16;                 // 16-key chunks
  static constexpr int NS = (NC + 1) / 2;                   // 32-key P.V steps
  static constexpr int KEYS = LY * LX;
  static constexpr int KSLOTS = KEYS * (kKRow / 16), VSLOTS = KEYS * (kVRow / 16);
  static constexpr int ITK = (KSLOTS + kThreads - 1) / kThreads;
  static constexpr int ITV = (VSLOTS + kThreads - 1) / kThreads;
  static constexpr int KTILE = ITK * kThreads * 16, VTILE = ITV * kThreads * 16;
  static constexpr int LDS = NBUF * (KTILE + VTILE) + KTILE;  // + the phases of the box
  static_assert(LDS <= kLdsMax, "key tiles exceed LDS");
  static constexpr int CPC = (ITK + ITV + NC - 1) / NC;  // copies issued beside each chunk of one update
  static_assert(KZ % 2 == 1 && KY % 2 == 1 && KX % 2 == 1, "odd windows");
};

struct LsgArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;  // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  uint16_t* out;
  float* lse;        // optional
  int heads, Z, H, W;
  int n_yb, n_xb, n_zg, n_hg, hpw;
  float qscale;      // 2 scale log2(e) (K enters at half length)
  float eps;
  const uint16_t* gate;
  int gate_dim;
};

template <int I>
struct IC {
  static constexpr int v = I;
};
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(IC<I>{});
    static_for<N, I + 1>(f);
  }
}

// Rotate 4 pairs of K held as packed bf16x2 words by packed float16 phases
// (c, s): round-toward-zero to float16, then (a c - b s, a s + b c) in packed
// float16 with the halves of the phase word taken through the operand selects.
__device__ __forceinline__ uint4 rotate_k8(uint4 x, uint4 ph, float mul = 1.f) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  const uint32_t p[4] = {ph.x, ph.y, ph.z, ph.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint32_t ab =
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo_bf16(w[t]) * mul, hi_bf16(w[t]) * mul));
    uint32_t tt;
    asm("v_pk_mul_f16 %1, %2, %3 op_sel_hi:[0,1]\n\t"
        "v_pk_fma_f16 %0, %2, %3, %1 op_sel:[1,1,0] op_sel_hi:[1,0,1] neg_lo:[0,1,0]"
        : "=v"(r[t]), "=&v"(tt) : "v"(ab), "v"(p[t]));
  }
  return make_uint4(r[0], r[1], r[2], r[3]);
}

template <int KZ, int KY, int KX, int G, int NBUF, bool NORM, bool GATE>
__global__ void __launch_bounds__(kThreads, 1) na3d_fwd_lsg_kernel(LsgArgs a) {
  using C = LsgCfg<KZ, KY, KX, G, NBUF>;
  constexpr int NC = C::NC, NS = C::NS, ITK = C::ITK, ITV = C::ITV;
  constexpr int LX = C::LX, NUX = C::NUX, NU = C::NU, KEYS = C::KEYS;
  __shared__ __attribute__((aligned(16))) char tK0[C::KTILE];
  __shared__ __attribute__((aligned(16))) char tV0[C::VTILE];
  __shared__ __attribute__((aligned(16))) char tK1[NBUF == 2 ? C::KTILE : 16];
  __shared__ __attribute__((aligned(16))) char tV1[NBUF == 2 ? C::VTILE : 16];
  __shared__ __attribute__((aligned(16))) char sph[C::KTILE];

  // ---- block coordinates (XCD-aware: neighbouring blocks share an L2) -------
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int xb = bid % a.n_xb;
  const int yb = (bid / a.n_xb) % a.n_yb;
  const int zg = (bid / (a.n_xb * a.n_yb)) % a.n_zg;
  const int hg = (bid / (a.n_xb * a.n_yb * a.n_zg)) % a.n_hg;
  const int b = bid / (a.n_xb * a.n_yb * a.n_zg * a.n_hg);
  const int h_lo = hg * a.hpw;
  const int h_hi = min(h_lo + a.hpw, a.heads);
  const int H = a.H, W = a.W, Z = a.Z;
  const int64_t HW = (int64_t)H * W;
  const int by0 = yb * 8, bx0 = xb * 8;
  const int z0 = zg * G;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, qn = lane & 15;

  // query levels of the group: first key level of each window (wave-uniform);
  // a level past the column gets a start that no key level reaches
  int zsj[G];
#pragma unroll
  for (int j = 0; j < G; ++j) zsj[j] = z0 + j < Z ? win_start(z0 + j, Z, KZ) : (1 << 20);
  const int kp_lo = zsj[0];
  const int kp_hi = win_start(min(z0 + G, Z) - 1, Z, KZ) + KZ - 1;

  const int ty0 = win_start(min(by0, H - 1), H, KY);
  const int tx0 = win_start(min(bx0, W - 1), W, KX);
  const int sy0 = by0 + 4 * (wave >> 1), sx0 = bx0 + 4 * (wave & 1);
  const int uy0 = win_start(min(sy0, H - 1), H, KY);
  const int ux0 = win_start(min(sx0, W - 1), W, KX);
  const int qy_raw = sy0 + (qn >> 2), qx_raw = sx0 + (qn & 3);
  const int qy = min(qy_raw, H - 1), qx = min(qx_raw, W - 1);
  const bool in_grid = qy_raw < H && qx_raw < W;

  // (the row step NUX / 2 keeps the 16 keys of a chunk, which span two or three
  // rows of the sub-block's key box, in 16 distinct bank groups: 5 for 10-wide
  // boxes, 6 for 12-wide ones)
  auto kswz = [&](int key) { return ((key % LX >> 1) + (NUX / 2) * (key / LX)) & 7; };
  auto key_row = [&](int u) { return u < NU ? (uy0 - ty0 + u / NUX) * LX + (ux0 - tx0 + u % NUX) : 0; };

  // ---- LDS addresses of this lane's fragments and its window mask ----------
  const int wys = win_start(qy, H, KY), wxs = win_start(qx, W, KX);
  uint32_t kaddr[NC], vaddr[NC];
  f32x4 bias[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    {
      const int key = key_row(16 * c + qn);
      kaddr[c] = key * kKRow + ((g ^ kswz(key)) << 4);
    }
    vaddr[c] = key_row(16 * c + 4 * g + (qn >> 2)) * kVRow + (qn & 3) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = 16 * c + 4 * g + i;
      const int ky = uy0 + u / NUX, kx = ux0 + u % NUX;
      const bool ok = u < NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX;
      bias[c][i] = ok ? 0.f : -INFINITY;
    }
  }

  // ---- copy offsets and the half-length phases of this thread's K slots ------
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * 16 : nullptr;
  auto pos_of = [&](int key) { return min(ty0 + key / LX, H - 1) * W + min(tx0 + key % LX, W - 1); };
  uint32_t koff[ITK], voff[ITV];
#pragma unroll
  for (int it = 0; it < ITK; ++it) {
    const int s = it * kThreads + tid;
    const int key = min(s >> 3, KEYS - 1);  // pad slots copy a valid row into the pad
    const int c = (s & 7) ^ kswz(key);
    const int pos = pos_of(key);
    koff[it] = (uint32_t)(pos * kD + c * 8) * 2u;
    uint4 ph;
    if (csb) {
      const float4* pp = csb + (int64_t)pos * 16 + 2 * c;
      const float4 p0 = pp[0] * 0.5f, p1 = pp[1] * 0.5f;
      ph = make_uint4(pack2h(p0.x, p0.y), pack2h(p0.z, p0.w), pack2h(p1.x, p1.y), pack2h(p1.z, p1.w));
    } else {
      const uint32_t half = pack2h(0.5f, 0.f);
      ph = make_uint4(half, half, half, half);
    }
    st16(sph + s * 16, ph);
  }
#pragma unroll
  for (int it = 0; it < ITV; ++it) {
    const int s = it * kThreads + tid;
    const int key = min(s / 10, KEYS - 1);
    const int c = s % 10 < 8 ? s % 10 : 0;  // pad columns copy column 0
    voff[it] = (uint32_t)(pos_of(key) * kD + c * 8) * 2u;
  }
  // float32 phases of this lane's query position (pairs 4g..4g+3, 16+4g..),
  // the same for every level and head: loaded once and kept
  const float4* csq = csb ? csb + ((int64_t)qy * W + qx) * 16 : nullptr;
  float4 cqv[4] = {};
  if (csq) {
    cqv[0] = csq[2 * g];
    cqv[1] = csq[2 * g + 1];
    cqv[2] = csq[8 + 2 * g];
    cqv[3] = csq[8 + 2 * g + 1];
  }

  auto level_base = [&](int h, int p) { return (((int64_t)b * a.heads + h) * Z + p) * HW; };
  auto rotate_k = [&](char* tk, char* tv) {
    uint4 y[ITV];
#pragma unroll
    for (int it = 0; it < ITV; ++it) y[it] = ld16(tv + (it * kThreads + tid) * 16);
    uint4 x[ITK];
#pragma unroll
    for (int it = 0; it < ITK; ++it) x[it] = ld16(tk + (it * kThreads + tid) * 16);
    float rn[ITK];
#pragma unroll
    for (int it = 0; it < ITK; ++it)
      rn[it] = NORM ? __builtin_amdgcn_rsqf(sum_over_8_lanes(sumsq8(x[it], 0.f)) * (1.f / kD) + a.eps) : 1.f;
#pragma unroll
    for (int it = 0; it < ITK; ++it)
      st16(tk + (it * kThreads + tid) * 16, rotate_k8(x[it], ld16(sph + (it * kThreads + tid) * 16), rn[it]));
#pragma unroll
    for (int it = 0; it < ITV; ++it) st16(tv + (it * kThreads + tid) * 16, bf16x8_to_f16x8(y[it]));
  };
  auto load_q = [&](int h, int z, uint4& x0, uint4& x1) {
    const uint4* src =
        reinterpret_cast<const uint4*>(a.q + (level_base(h, min(z, Z - 1)) + (int64_t)qy * W + qx) * kD);
    x0 = src[g];
    x1 = src[4 + g];
  };
  auto prep_q = [&](const float4* cq, uint4 x0, uint4 x1, f16x8& q0, f16x8& q1) {
    uint4 r0, r1;
    float mul = a.qscale;
    if constexpr (NORM) mul *= __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(x1, sumsq8(x0, 0.f))) * (1.f / kD) + a.eps);
    if (cq) {
      r0 = rotate8h(x0, cqv[0], cqv[1], mul);
      r1 = rotate8h(x1, cqv[2], cqv[3], mul);
    } else {
      r0 = scale8h(x0, mul);
      r1 = scale8h(x1, mul);
    }
    q0 = __builtin_bit_cast(f16x8, r0);
    q1 = __builtin_bit_cast(f16x8, r1);
  };

  // ---- per query level state (all G live for the whole head) ---------------
  f16x8 qf[G][2];
  float m[G];
  f32x4 lsum[G];
  bool mset[G];
  f32x4 o[G][4];
  uint4 qraw[G][2];
  uint2 gch[GATE ? G : 1][4];
  uint32_t ghd[GATE ? G : 1];
  const f16x8 ones = __builtin_bit_cast(f16x8, make_uint4(0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u));

  struct Frags {
    f16x8 k[NC][2];
    f16x8 v[NS][4];
  };
  auto load_frags = [&](const char* tk, const char* tv, Frags& f) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      f.k[c][0] = __builtin_bit_cast(f16x8, ld16(tk + kaddr[c]));
      f.k[c][1] = __builtin_bit_cast(f16x8, ld16(tk + (kaddr[c] ^ 64u)));
    }
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const int c0 = 2 * st, c1 = 2 * st + 1;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const i16x4 lo = tr_read(tv + vaddr[c0] + 32 * t);
        const i16x4 hi = c1 < NC ? tr_read(tv + vaddr[c1 < NC ? c1 : c0] + 32 * t) : i16x4{0, 0, 0, 0};
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        f.v[st][t] = __builtin_bit_cast(f16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
      }
    }
  };

  // one query level j at one key level; `first`: the level's first key level;
  // hook(c) runs beside the logits of chunk c
  auto update = [&](auto Ji, const Frags& f, bool first, auto&& hook) {
    constexpr int j = decltype(Ji)::v;
    f32x4 s[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      hook(c);
      const f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.k[c][0], qf[j][0], bias[c], 0, 0, 0);
      s[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.k[c][1], qf[j][1], acc, 0, 0, 0);
    }
    {
      float mx = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
      mx = fmaxf(mx, s[0][3]);
#pragma unroll
      for (int c = 1; c < NC; ++c) {
        mx = fmaxf(fmaxf(mx, s[c][0]), s[c][1]);
        mx = fmaxf(fmaxf(mx, s[c][2]), s[c][3]);
      }
      mx = max_over_rows(mx);
      const bool move = mx > m[j] + kLazy || (first && mx < kLow);
      if (__any(move)) {  // rare: move the reference m
        const float mn = move ? mx : m[j];
        if (!first) {
          const float alpha = __builtin_amdgcn_exp2f(m[j] - mn);
          lsum[j] *= alpha;
#pragma unroll
          for (int t = 0; t < 4; ++t) o[j][t] *= alpha;
        }
        m[j] = mn;
        mset[j] = true;
      }
      if (mset[j]) {
#pragma unroll
        for (int c = 0; c < NC; ++c) s[c] -= m[j];
      }
    }
    uint32_t pk[NC][2];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      pk[c][0] = pack2h_rne(__builtin_amdgcn_exp2f(s[c][0]), __builtin_amdgcn_exp2f(s[c][1]));
      pk[c][1] = pack2h_rne(__builtin_amdgcn_exp2f(s[c][2]), __builtin_amdgcn_exp2f(s[c][3]));
    }
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const int c0 = 2 * st, c1 = 2 * st + 1;
      const uint32_t p2 = c1 < NC ? pk[c1 < NC ? c1 : c0][0] : 0u;
      const uint32_t p3 = c1 < NC ? pk[c1 < NC ? c1 : c0][1] : 0u;
      const f16x8 pf = __builtin_bit_cast(f16x8, make_uint4(pk[c0][0], pk[c0][1], p2, p3));
#pragma unroll
      for (int t = 0; t < 4; ++t)
        o[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.v[st][t], pf, o[j][t], 0, 0, 0);
      lsum[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones, pf, lsum[j], 0, 0, 0);
    }
  };

  // normalise and store query level j of head h
  auto finish = [&](auto Ji, int h) {
    constexpr int j = decltype(Ji)::v;
    const int z = z0 + j;
    const float lt = lsum[j][0];
    if (!in_grid || z >= Z) return;
    float inv = 1.f / lt;
    if constexpr (GATE)
      if (a.gate_dim == 1) inv *= sigmoid_fast(__uint_as_float(ghd[j] << 16));
    const int64_t tok = level_base(h, z) + (int64_t)qy * W + qx;
    uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
#pragma unroll
    for (int t = 0; t < 4; ++t) {  // d = 16t + 4g + i
      f32x4 r = o[j][t] * inv;
      if constexpr (GATE)
        if (a.gate_dim != 1) r *= sigmoid4_bf16(gch[j][t]);
      dst[4 * t + g] = make_uint2(pack2(r[0], r[1]), pack2(r[2], r[3]));
    }
    if (a.lse && g == 0) a.lse[tok] = (m[j] + __log2f(lt)) * kLn2;
  };

  // ---- prologue: the first head's first key level and its query rows --------
  {
    const int64_t base = level_base(h_lo, kp_lo);
    const char* kp = reinterpret_cast<const char*>(a.k + base * kD);
    const char* vp = reinterpret_cast<const char*>(a.v + base * kD);
#pragma unroll
    for (int it = 0; it < ITK; ++it)
      copy16_to_lds(reinterpret_cast<const uint16_t*>(kp + koff[it]), tK0 + (it * kThreads + wave * 64) * 16);
#pragma unroll
    for (int it = 0; it < ITV; ++it)
      copy16_to_lds(reinterpret_cast<const uint16_t*>(vp + voff[it]), tV0 + (it * kThreads + wave * 64) * 16);
  }
#pragma unroll
  for (int j = 0; j < G; ++j) load_q(h_lo, z0 + j, qraw[j][0], qraw[j][1]);
  __builtin_amdgcn_s_waitcnt(0);
  rotate_k(tK0, tV0);
  __syncthreads();

  int iter = 0;  // key levels swept so far (buffer parity)
  for (int h = h_lo; h < h_hi; ++h) {
    const bool more_heads = h + 1 < h_hi;
    // queries of every level of the group, rotated and scaled once per head
    {
      static_for<G>([&](auto Ji) {
        constexpr int j = decltype(Ji)::v;
        prep_q(csq, qraw[j][0], qraw[j][1], qf[j][0], qf[j][1]);
        m[j] = 0.f;
        mset[j] = false;
        lsum[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 4; ++t) o[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
      });
    }
    for (int p = kp_lo; p <= kp_hi; ++p, ++iter) {
      const bool last = p == kp_hi;
      const bool has_next = !last || more_heads;
      const int64_t nbase = !last ? level_base(h, p + 1) : level_base(h + 1, kp_lo);
      auto key_level = [&](char* tk, char* tv, char* nk, char* nv) {
#pragma unroll
        for (int c = 0; c < NC; ++c) asm volatile("" : "+v"(kaddr[c]), "+v"(vaddr[c]));
#pragma unroll
        for (int it = 0; it < ITK; ++it) asm volatile("" : "+v"(koff[it]));
#pragma unroll
        for (int it = 0; it < ITV; ++it) asm volatile("" : "+v"(voff[it]));
        const char* const nkp = reinterpret_cast<const char*>(a.k + nbase * kD);
        const char* const nvp = reinterpret_cast<const char*>(a.v + nbase * kD);
        if (last && more_heads) {  // the next head's query rows
#pragma unroll
          for (int j = 0; j < G; ++j) load_q(h + 1, z0 + j, qraw[j][0], qraw[j][1]);
        }
        if constexpr (GATE) {  // gate logits of the levels that end here
          static_for<G>([&](auto Ji) {
            constexpr int j = decltype(Ji)::v;
            if (zsj[j] + KZ - 1 == p) {
              const int64_t tok = level_base(h, z0 + j) + (int64_t)qy * W + qx;
              if (a.gate_dim == 1) {
                ghd[j] = a.gate[tok];
              } else {
                const uint2* src = reinterpret_cast<const uint2*>(a.gate + tok * kD);
#pragma unroll
                for (int t = 0; t < 4; ++t) gch[j][t] = src[4 * t + g];
              }
            }
          });
        }
        Frags f;
        load_frags(tk, tv, f);
        if constexpr (NBUF == 1) {  // every wave holds its fragments: the buffer is free
          __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
          __syncthreads();
        }
        bool copy = has_next;  // the next level's copies ride on the first active update
        static_for<G>([&](auto Ji) {
          constexpr int j = decltype(Ji)::v;
          if ((unsigned)(p - zsj[j]) < (unsigned)KZ) {
            const bool cp = copy;
            update(Ji, f, p == zsj[j], [&](int c) {
              if (cp) {
#pragma unroll
                for (int e = 0; e < C::CPC; ++e) {
                  const int i = C::CPC * c + e;  // copy i: K slot i, then V slot i - ITK
                  if (i < ITK)
                    copy16_to_lds(reinterpret_cast<const uint16_t*>(nkp + koff[i < ITK ? i : 0]),
                                  nk + (i * kThreads + wave * 64) * 16);
                  else if (i - ITK < ITV)
                    copy16_to_lds(reinterpret_cast<const uint16_t*>(nvp + voff[i - ITK < ITV ? i - ITK : 0]),
                                  nv + ((i - ITK) * kThreads + wave * 64) * 16);
                }
              }
            });
            copy = false;
            if (p == zsj[j] + KZ - 1) finish(Ji, h);
          }
        });
        if (has_next) {
          __builtin_amdgcn_s_waitcnt(0);
          rotate_k(nk, nv);
        }
        __syncthreads();
      };
      if constexpr (NBUF == 2) {
        if (iter & 1) key_level(tK1, tV1, tK0, tV0);
        else key_level(tK0, tV0, tK1, tV1);
      } else {
        key_level(tK0, tV0, tK0, tV0);
      }
    }
  }
}

template <int KZ, int KY, int KX, int G, int NBUF, bool NORM, bool GATE>
bool launch_lsg(const strata_na3d_desc& d, const LsgArgs& a0, hipStream_t s) {
  LsgArgs a = a0;
  a.n_zg = (d.Z + G - 1) / G;
  // a run of up to 8 heads per workgroup shares its geometry; a small problem
  // takes fewer, so that the grid still has two workgroups per CU
  while (a.hpw > 1 && (int64_t)d.B * ((d.heads + a.hpw - 1) / a.hpw) * a.n_zg * a.n_yb * a.n_xb < 512)
    a.hpw = (a.hpw + 1) / 2;
  a.n_hg = (d.heads + a.hpw - 1) / a.hpw;
  const int64_t blocks = (int64_t)d.B * a.n_hg * a.n_zg * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  hipLaunchKernelGGL((na3d_fwd_lsg_kernel<KZ, KY, KX, G, NBUF, NORM, GATE>), dim3((unsigned)blocks), dim3(kThreads),
                     0, s, a);
  return true;
}

// four query levels per group; three with the gate at 5x9x9, whose logits of
// four levels would not fit the registers beside the 9-chunk fragments
template <int KZ, int KY, int KX>
bool launch_lsg_opts(const strata_na3d_desc& d, const NaOpts& o, const LsgArgs& a, hipStream_t s) {
  constexpr int GG = KY > 7 ? 3 : 4;
  switch ((o.qk_norm ? 1 : 0) | (o.gate ? 2 : 0)) {
    case 0: return launch_lsg<KZ, KY, KX, 4, 1, false, false>(d, a, s);
    case 1: return launch_lsg<KZ, KY, KX, 4, 1, true, false>(d, a, s);
    case 2: return launch_lsg<KZ, KY, KX, GG, 1, false, true>(d, a, s);
    default: return launch_lsg<KZ, KY, KX, GG, 1, true, true>(d, a, s);
  }
}

}  // namespace

// Grouped level-sweep forward (bf16, head_dim 64) for the windows 3x7x7 (any Z
// but 8, which the 8-level sweep takes) and 5x9x9; false otherwise.  (The
// kernel compiles for 9x9x9 too, but with four query levels per group it
// stages each key level for only ~3 updates: measured 7.94 ms against the
// query-stationary kernel's 6.54 ms on 96 tiles x 16 heads x 24 x 16 x 16.)
bool launch_na3d_fwd_lsg(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k, const void* v,
                         const float* cs, void* out, float* lse, hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  if ((int64_t)d.H * d.W * kD * 2 >= (int64_t)1 << 32) return false;  // byte offsets in 32 bits
  const bool w377 = d.kz == 3 && d.ky == 7 && d.kx == 7;
  const bool w599 = d.kz == 5 && d.ky == 9 && d.kx == 9;
  if (!w377 && !w599) return false;  // 9x9x9: the query-stationary kernel measured faster
  LsgArgs a = {};
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
  a.n_yb = (d.H + 7) / 8;
  a.n_xb = (d.W + 7) / 8;
  a.hpw = d.heads < 8 ? d.heads : 8;
  a.n_hg = (d.heads + a.hpw - 1) / a.hpw;
  a.qscale = 2.f * d.scale * kLog2e;  // K is rotated at half length
  a.eps = o.eps;
  a.gate = static_cast<const uint16_t*>(o.gate);
  a.gate_dim = o.gate_dim;
  if (w377) return launch_lsg_opts<3, 7, 7>(d, o, a, s);
  return launch_lsg_opts<5, 9, 9>(d, o, a, s);
}

}  // namespace strata

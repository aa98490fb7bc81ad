// MFMA neighbourhood attention for gfx950, query-stationary kernels (bf16 in/out,
// head_dim 64): the forward, and the dQ part of the backward.
//
// Work decomposition
//   workgroup : one (tile, head), an 8 x 8 block of (y, x) query positions, NG
//               groups of four waves, one workgroup per CU; it takes the groups
//               of ZQ query levels of its block's column one after another.
//   wave      : a 4 x 4 (y, x) sub-block = 16 queries, on ZQ/NG of a group's
//               levels (wave group g takes the levels g, g + NG, ..., so every
//               group has work at every key level).  NG = 2 (8 waves) for the
//               forward and the 3x7x7 dQ; NG = 3 (12 waves, three per SIMD, one
//               query level each) for the dQ of the 9-wide windows.
//   key sweep : for each group of query levels the workgroup walks the key
//               levels they need, each once (the copies of the next group's
//               first level run during the current group's last).
//               K and V of the (8+ky-1) x (8+kx-1) key box of a level are copied
//               global -> LDS by the direct-to-LDS load (no registers), one level
//               ahead of the compute, into a double buffer; each thread then
//               rotates the K pieces its own copies brought (StereoRoPE, in
//               packed float16 with float16 phases, staged in LDS when they
//               fit, else converted from the float32 table) and one barrier
//               publishes the level.
//
// Per (query level, key level) a wave multiplies the keys of its 4x4 sub-block's
// box -- (3+ky) x (3+kx) keys, in 16-key chunks -- with its 16 queries:
//   S^T (16 keys x 16 queries) = K . Q^T     v_mfma_f32_16x16x32_f16, the
//                                           accumulator seeded with the window
//                                           mask (0 or -inf),
//   online softmax on S^T in registers (a lane owns one query column) against
//   a lazy reference m: it starts at 0 and moves only when a logit exceeds it
//   by more than 2^8 (or, on a query level's first key level, when no logit
//   reaches -2^6), so most steps rescale nothing and, while m is 0 across the
//   wave, subtract nothing; cross-row maxima use v_permlane16/32_swap,
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
// Options: QK RMSNorm (the factor of every query and key, from its sum of
// squares over the lanes that hold it, scales it in float32 before the float16
// rounding; the backward applies the norm's Jacobian to dQ before the store),
// the sigmoid gate applied with the final 1/l (forward), and dO given as two
// bf16 terms hi + lo (backward: one more MFMA pair for Y).
//
// K rows are 128 bytes with their 16-byte columns XOR-swizzled by
// ((x >> 1) + (NUX / 2) y) & 7 of the key's box position (NUX = 3 + kx, the
// width of a sub-block's key box): the 16 keys of any chunk of an interior
// sub-block then sit in 16 distinct bank groups.  In the forward V rows
// are padded to 160 bytes, which spreads the 8-byte transpose reads and lets
// them take immediate offsets; the backward reads V rows as an A operand and
// stages them like K (128 bytes, same swizzle).  The two halves of the double buffer are distinct LDS objects, so the
// compiler can tell the reads of one from the copies into the other and does not
// wait for the copies before reading.
//
// Backward, dQ (same decomposition and key staging; a lane still owns a query),
// 32 keys (two chunks) per step:
//   S^T = K . Q^T as above, seeded with -(lse2 + E - 15) where the query sees
//   the key (window bits, two words per lane) and -inf elsewhere, so that
//   exp2(S^T) is the weight P^T (from the forward's log-sum-exp, no online
//   softmax) times the current dS scale 2^(15 - E);
//   Y^T (16 keys x 16 queries) = V . dO^T - D   bf16 MFMA, V rows read as the A
//                                           operand, dO of the lane's query held
//                                           in registers, seeded with -D;
//   dS^T = P^T * Y^T, and dQ~^T (64 d x 16 queries) += K~^T . dS^T as a float16
//   MFMA whose K~^T fragments come from the rotated K tile by the transpose read.
//   dS is carried in float16 with a per-query power-of-two scale 2^(15 - E): E
//   bounds |Y| of every step seen so far (|dS| <= P |Y|, P <= 1), so the
//   scaled values stay below 2^15; when a step raises E the accumulator is
//   rescaled exactly and the step's logits move by the change.  At the end
//   dQ = R^T (scale 2^(E-15) dQ~).
// The lanes that load a query's dO row also load its O row and form D = <dO, O>
// (stored once for the dK/dV pass), and every lane keeps the largest |dO| it
// loads: at the end each wave takes an integer atomic maximum of that value's
// exponent into a word per (batch, head), by which the balanced dK/dV pass
// scales its float16 copy of dO.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

namespace strata {
namespace {

using namespace mfma;


constexpr int kBY = 8, kBX = 8;  // query block of a workgroup (y, x)
constexpr int kD = 64;           // head_dim
constexpr int kKRow = 128;       // LDS bytes per key row of K (16-byte columns swizzled)
constexpr int kVRow = 160;       // LDS bytes per key row of V (128 + 32 pad)
constexpr int kLdsMax = 160 * 1024;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLazy = 8.0f;    // move the softmax reference only when a logit exceeds it by > 2^8
constexpr float kLow = -64.0f;   // ... or down, on a level's first key level
constexpr int kMinExp = -100;    // lower bound of the dS exponent (keeps 2^(15-E) finite)

// largest |x| over the 8 bf16 values of a 16-byte piece, or m if larger
__device__ __forceinline__ float absmax8(uint4 x, float m) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int t = 0; t < 4; ++t) m = fmaxf(m, fmaxf(fabsf(lo_bf16(w[t])), fabsf(hi_bf16(w[t]))));
  return m;
}

// <x, y> over the 8 bf16 values of two 16-byte pieces, added to acc (the
// products are exact in float32)
__device__ __forceinline__ float dot8(uint4 x, uint4 y, float acc) {
  const uint32_t u[4] = {x.x, x.y, x.z, x.w}, w[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
  for (int t = 0; t < 4; ++t)
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u[t]), __builtin_bit_cast(bf16x2, w[t]), acc,
                                          false);
  return acc;
}

// NG groups of four waves, one wave per 4x4 sub-block in each group; group g
// takes the levels g, g + NG, ... of the block's ZQ levels
template <int KZ, int KY, int KX, int ZQ, bool BWD, int NG>
struct Cfg {
  static constexpr int kThreads = 256 * NG;
  // V rows: the forward reads V^T by transpose reads (160-byte rows spread
  // them); the backward reads V rows as an A operand like K (128-byte rows with
  // K's column swizzle, conflict-free)
  static constexpr int VROW = BWD ? kKRow : kVRow;
  static constexpr int LY = kBY + KY - 1, LX = kBX + KX - 1;  // staged key box per level
  static constexpr int NUY = 3 + KY, NUX = 3 + KX;            // key box of one 4x4 sub-block
  static constexpr int NU = NUY * NUX;
  static constexpr int NC = (NU + 15) / 16;                   // 16-key chunks
  static constexpr int NS = (NC + 1) / 2;                     // 32-key PV steps
  static constexpr int KEYS = LY * LX;
  static constexpr int KSLOTS = KEYS * (kKRow / 16);          // 16-byte slots of a K tile (8 per key)
  static constexpr int VSLOTS = KEYS * (VROW / 16);
  static constexpr int KBYTES = KEYS * kKRow, VBYTES = KEYS * VROW;
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
  static constexpr int QL = ZQ / NG;                          // query levels per wave
  static_assert(ZQ % NG == 0, "ZQ must be a multiple of NG");
  static_assert(2 * BUF <= kLdsMax, "key tiles exceed LDS");
};

struct Args {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;   // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  uint16_t* out;      // forward: O; backward: dQ
  float* lse;         // forward: optional LSE output
  const uint16_t* dout;  // backward: dO
  const float* lse_in;   // backward: LSE of the forward (natural log)
  const float* dvec;     // backward: D = rowsum(dO * O)
  const uint16_t* fo;    // backward: the forward's O; when set, D is formed here
  float* dvec_out;       //   from dO and O and stored for the dK/dV pass
  int* emax;             // backward: per (batch, head) the largest exponent of
                         //   |dO| (atomic max; frexp convention), or nullptr
  int heads, Z, H, W;
  int n_zb, n_yb, n_xb;
  int n_zc, zb_per;   // runs of query-level groups per column, groups per run
  float qscale;       // scale * log2(e)
  float scale;
  // options: QK RMSNorm (factor applied in float32 before the float16
  // rounding), the sigmoid output gate (forward), the low term of a two-term
  // dO (backward)
  int qk_norm;
  float eps;
  const uint16_t* gate;
  int gate_dim;
  const uint16_t* dout_lo;
};

// OPT: bit 0 = QK RMSNorm; bit 1 = the output gate (forward) or the low term of
// a two-term dO (backward)
constexpr int kNorm = 1, kOpt2 = 2;

template <int KZ, int KY, int KX, int ZQ, bool BWD, int OPT, int NG>
__global__ void __launch_bounds__(256 * NG, 1) na3d_mfma_q_kernel(Args a) {
  constexpr bool NORM = (OPT & kNorm) != 0;
  constexpr bool GATE = !BWD && (OPT & kOpt2) != 0;
  constexpr bool LO = BWD && (OPT & kOpt2) != 0;
  using C = Cfg<KZ, KY, KX, ZQ, BWD, NG>;
  constexpr int kThreads = C::kThreads;
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
  const int zc = (bid / (a.n_xb * a.n_yb)) % a.n_zc;
  const int bh = bid / (a.n_xb * a.n_yb * a.n_zc);
  const int b = bh / a.heads;
  const int H = a.H, W = a.W, Z = a.Z;
  const int by0 = yb * kBY, bx0 = xb * kBX;
  // the workgroup takes the groups [zb_lo, zb_hi) of ZQ query levels one after
  // another; z0 is the first level of the current group
  const int zb_lo = zc * a.zb_per, zb_hi = min(zb_lo + a.zb_per, a.n_zb);
  int z0 = zb_lo * ZQ;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;
  const int sb = wave & 3, grp = wave >> 2;  // xy sub-block, level group

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
  // (the row step NUX / 2 keeps the 16 keys of a chunk, which span two or three
  // rows of the sub-block's key box, in 16 distinct bank groups: 5 for 10-wide
  // boxes, 6 for 12-wide ones)
  auto kswz = [&](int key) { return ((key % C::LX >> 1) + (C::NUX / 2) * (key / C::LX)) & 7; };
  // tile row of sub-block key u (u past the box: row 0, masked)
  auto key_row = [&](int u) {
    return u < C::NU ? (uy0 - ty0 + u / C::NUX) * C::LX + (ux0 - tx0 + u % C::NUX) : 0;
  };

  // ---- per-lane tile offsets and window mask, identical for every key level ----
  // forward: vaddr = V^T transpose-read address; backward: vaddr = V row (A
  // operand) address, ktaddr = K~^T transpose-read address
  uint32_t kaddr[C::NC], vaddr[C::NC], ktaddr[BWD ? C::NC : 1];
  // window mask: forward, the accumulator seeds (0 / -inf); backward, bits (bit
  // 4c + i: row 4g + i of chunk c seen by the lane's query), from which each
  // step selects its seeds
  f32x4 bias[BWD ? 1 : C::NC];
  static_assert(!BWD || C::NC <= 16, "window bits of a lane fit two words");
  uint32_t mbits[2] = {0u, 0u};
#pragma unroll
  for (int c = 0; c < C::NC; ++c) {
    {  // K fragment (A operand): row = key 16c + qn, 16 bytes at column g (xor 64 bytes: g+4)
      const int key = key_row(16 * c + qn);
      kaddr[c] = key * kKRow + ((g ^ kswz(key)) << 4);
      if constexpr (BWD) vaddr[c] = kaddr[c];  // V row, the same swizzled layout as K
    }
    {  // transpose reads: source row = key 16c + 4g + qn/4, elements 4*(qn%4) of a 16-wide block
      const int key = key_row(16 * c + 4 * g + (qn >> 2));
      if constexpr (BWD)
        ktaddr[c] = key * kKRow + ((((qn >> 1) & 1) ^ kswz(key)) << 4) + 8 * (qn & 1);
      else
        vaddr[c] = key * kVRow + (qn & 3) * 8;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int u = 16 * c + 4 * g + i;
      int ky = uy0 + u / C::NUX, kx = ux0 + u % C::NUX;
      bool ok = u < C::NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX;
      if constexpr (BWD)
        mbits[c >> 3] |= (ok ? 1u : 0u) << (4 * (c & 7) + i);
      else
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
    // forward: 10 slots per key (8 data + 2 pad); backward: 8, swizzled like K
    int s = it * kThreads + tid, key = BWD ? s >> 3 : s / 10, c = BWD ? (s & 7) ^ kswz(key) : s - key * 10;
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
  // With QK RMSNorm the 8 slots of a key (8 consecutive lanes, all in or all
  // past the tile) add their sums of squares, and the factor scales the values
  // in float32 before they are rounded.
  auto rotate_k = [&](char* tk) {
#pragma unroll
    for (int it = 0; it < C::ITK; ++it) {
      // slots past the tile exist only in the last pass (known per thread)
      if ((it + 1) * kThreads > C::KSLOTS && it * kThreads + tid >= C::KSLOTS) continue;
      char* ad = tk + (it * kThreads + tid) * 16;
      uint4 x = ld16(ad);
      float mul = 1.f;
      if constexpr (NORM) mul = __builtin_amdgcn_rsqf(sum_over_8_lanes(sumsq8(x, 0.f)) * (1.f / kD) + a.eps);
      if (csb) {
        if (C::PH_LDS) {
          x = rotate8h_pk(x, ld16(sph + (it * kThreads + tid) * 16), mul);
        } else {  // the same float16 phases, converted here (|cos|, |sin| <= 1: no saturation)
          const int o = goffK(it);
          const float4* pp = csb + (o >> 6) * 16 + ((o & 63) >> 2);
          const float4 p0 = pp[0], p1 = pp[1];
          x = rotate8h_pk(x, make_uint4(pack2h_rne(p0.x, p0.y), pack2h_rne(p0.z, p0.w), pack2h_rne(p1.x, p1.y),
                                        pack2h_rne(p1.z, p1.w)), mul);
        }
      } else {
        x = scale8h(x, mul);
      }
      st16(ad, x);
    }
  };

  // ---- queries: load, rotate, scale, keep as the B operand of K.Q^T ----------
  // forward: running max m, row sum l, O^T accumulator o;
  // backward: dO^T fragments gf, LSE in log2 units lse2, -D nd, dS exponent ex,
  //           dQ~^T accumulator o
  f16x8 qf[C::QL][2];
  bf16x8 gf[BWD ? C::QL : 1][2], gl[LO ? C::QL : 1][2];  // dO (hi and low terms)
  float rq[BWD && NORM ? C::QL : 1];                     // QK RMSNorm factor of the query
  float m[C::QL], l[C::QL];
  bool mset[C::QL];  // forward, wave-uniform: the reference m has moved from 0 somewhere in the wave
  int ex[C::QL];
  f32x4 o[C::QL][4];
  float gmx = 0.f;  // backward: largest |dO| this lane has loaded
  const float4* csq = csb ? csb + ((int64_t)qy * W + qx) * 16 : nullptr;
  // queries of the group starting at level z0 (and, backward, their dO, LSE, D)
  auto begin_group = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < C::QL; ++j) {
      int zq = min(z0 + grp + NG * j, Z - 1);
      const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
      const uint4* src = reinterpret_cast<const uint4*>(a.q + tok * kD);
      uint4 x0 = src[g], x1 = src[4 + g];
      uint4 r0, r1;
      float mul = a.qscale;
      if constexpr (NORM) {  // the 4 lanes of a query row hold its 64 values
        const float rn = __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(x1, sumsq8(x0, 0.f))) * (1.f / kD) + a.eps);
        mul *= rn;
        if constexpr (BWD) rq[j] = rn;
      }
      if (csq) {
        r0 = rotate8h(x0, csq[2 * g], csq[2 * g + 1], mul);
        r1 = rotate8h(x1, csq[8 + 2 * g], csq[8 + 2 * g + 1], mul);
      } else {
        r0 = scale8h(x0, mul);
        r1 = scale8h(x1, mul);
      }
      qf[j][0] = __builtin_bit_cast(f16x8, r0);
      qf[j][1] = __builtin_bit_cast(f16x8, r1);
      if constexpr (BWD) {
        const uint4* gsrc = reinterpret_cast<const uint4*>(a.dout + tok * kD);
        const uint4 g0 = gsrc[g], g1 = gsrc[4 + g];
        gf[j][0] = __builtin_bit_cast(bf16x8, g0);
        gf[j][1] = __builtin_bit_cast(bf16x8, g1);
        if constexpr (!LO) {  // (the balanced dK/dV pass, which reads it, takes no two-term dO)
          if (a.emax) gmx = absmax8(g1, absmax8(g0, gmx));
        }
        if constexpr (LO) {
          const uint4* lsrc = reinterpret_cast<const uint4*>(a.dout_lo + tok * kD);
          gl[j][0] = __builtin_bit_cast(bf16x8, lsrc[g]);
          gl[j][1] = __builtin_bit_cast(bf16x8, lsrc[4 + g]);
        }
        m[j] = a.lse_in[tok] * kLog2e;  // lse2
        float dj;
        if (a.fo) {  // D = <dO, O> of the row over the 4 lanes that hold it, stored once
          const uint4* osrc = reinterpret_cast<const uint4*>(a.fo + tok * kD);
          dj = sum_over_rows(dot8(osrc[4 + g], g1, dot8(osrc[g], g0, 0.f)));
          if (g == 0 && z0 + grp + NG * j < Z && qy_raw < H && qx_raw < W) a.dvec_out[tok] = dj;
        } else {
          dj = a.dvec[tok];
        }
        l[j] = -dj;  // -D
        ex[j] = kMinExp;
      } else {
        m[j] = 0.f;
        l[j] = 0.f;
        mset[j] = false;
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) o[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  begin_group();

  // one (query level j, key level) update with the key tiles tk, tv; `first`:
  // the query level's first key level (nothing accumulated yet)
  auto update = [&](int j, bool first, const char* tk, const char* tv) {
    f32x4 s[C::NC];
#pragma unroll
    for (int c = 0; c < C::NC; ++c) {
      f16x8 k0 = __builtin_bit_cast(f16x8, ld16(tk + kaddr[c]));
      f16x8 k1 = __builtin_bit_cast(f16x8, ld16(tk + (kaddr[c] ^ 64u)));
      f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(k0, qf[j][0], bias[c], 0, 0, 0);
      s[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(k1, qf[j][1], acc, 0, 0, 0);
    }
    float mx = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
    mx = fmaxf(fmaxf(mx, s[0][3]), s[1][0]);
#pragma unroll
    for (int c = 1; c < C::NC; ++c) {  // three-input maxima
      if (c > 1) mx = fmaxf(fmaxf(mx, s[c][0]), s[c][1]);
      else mx = fmaxf(mx, s[c][1]);
      mx = fmaxf(fmaxf(mx, s[c][2]), s[c][3]);
    }
    mx = max_over_rows(mx);
    // the reference m starts at 0 and moves when a logit exceeds it by more
    // than 2^kLazy, or when a query level's first key level has no logit above
    // kLow (nothing is accumulated yet); while it is 0 across the wave no
    // subtraction is needed
    const bool move = mx > m[j] + kLazy || (first && mx < kLow);
    if (__any(move)) {  // rare: move the reference, rescale
      const float mn = move ? mx : m[j];
      if (!first) {  // nothing is accumulated before the first key level (and a downward
                     // move there would make the factor overflow)
        const float alpha = __builtin_amdgcn_exp2f(m[j] - mn);
        l[j] *= alpha;
#pragma unroll
        for (int t = 0; t < 4; ++t) o[j][t] *= alpha;
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

  // backward: one (query level j, key level) update of dQ~ with the key tiles
  // tk, tv, 32 keys (two chunks) at a time: logits and Y, the exponent bound of
  // |Y| grown to cover them (the accumulator rescaled exactly when it grows), dS
  // in float16 with the current scale, and the dQ MFMAs of the two chunks.  The
  // logits are seeded with -(lse2 + E - 15) where the lane's query sees the key
  // (so that P 2^(15-E) = exp2(S)) and -inf elsewhere, selected by the window
  // bits; a step whose bound grows moves its own logits by the change.
  auto update_dq = [&](int j, const char* tk, const char* tv) {
    const f32x4 nd = {l[j], l[j], l[j], l[j]};
    uint32_t mw[2] = {mbits[0], mbits[1]};
    asm volatile("" : "+v"(mw[0]), "+v"(mw[1]));  // derive the selects step by step
#pragma unroll
    for (int st = 0; st < C::NS; ++st) {
      const int c0 = 2 * st, c1 = 2 * st + 1;
      const bool two = c1 < C::NC;
      // transpose reads of the step's K~^T, issued first: their latency hides
      // under the MFMAs and the softmax below
      uint2 ktl[4], kth[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        ktl[t] = __builtin_bit_cast(uint2, tr_read(tk + (ktaddr[c0] ^ (32u * t))));
        kth[t] = two ? __builtin_bit_cast(uint2, tr_read(tk + (ktaddr[two ? c1 : c0] ^ (32u * t))))
                     : make_uint2(0u, 0u);
      }
      const uint32_t ncj = __float_as_uint(-(m[j] + (float)(ex[j] - 15)));
      f32x4 s2[2], y2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = h == 0 ? c0 : (two ? c1 : c0);
        if (h == 1 && !two) {
          s2[1] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
          y2[1] = f32x4{0.f, 0.f, 0.f, 0.f};
          continue;
        }
        f32x4 seed;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int bit = 4 * c + i;
          const uint32_t sel = (uint32_t)__builtin_amdgcn_sbfe((int)mw[bit >> 5], bit & 31, 1);
          seed[i] = __uint_as_float((sel & ncj) | (~sel & 0xff800000u));
        }
        f16x8 k0 = __builtin_bit_cast(f16x8, ld16(tk + kaddr[c]));
        f16x8 k1 = __builtin_bit_cast(f16x8, ld16(tk + (kaddr[c] ^ 64u)));
        f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(k0, qf[j][0], seed, 0, 0, 0);
        s2[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(k1, qf[j][1], acc, 0, 0, 0);
        bf16x8 v0 = __builtin_bit_cast(bf16x8, ld16(tv + vaddr[c]));
        bf16x8 v1 = __builtin_bit_cast(bf16x8, ld16(tv + (vaddr[c] ^ 64u)));
        f32x4 t0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, gf[j][0], nd, 0, 0, 0);
        y2[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v1, gf[j][1], t0, 0, 0, 0);
        if constexpr (LO) {
          y2[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, gl[j][0], y2[h], 0, 0, 0);
          y2[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v1, gl[j][1], y2[h], 0, 0, 0);
        }
      }
      float my = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
        my = fmaxf(fmaxf(my, fmaxf(fabsf(y2[h][0]), fabsf(y2[h][1]))), fmaxf(fabsf(y2[h][2]), fabsf(y2[h][3])));
      my = max_over_rows(my);
      const int e = max(__builtin_amdgcn_frexp_expf(my), kMinExp);
      if (__any(e > ex[j])) {  // the bound grew: rescale the accumulator exactly
        const int en = max(ex[j], e);
        const float f = __builtin_amdgcn_ldexpf(1.f, ex[j] - en);
#pragma unroll
        for (int t = 0; t < 4; ++t) o[j][t] *= f;
        const float d = (float)(ex[j] - en);  // this step's logits carry the old offset
#pragma unroll
        for (int h = 0; h < 2; ++h) s2[h] += d;
        ex[j] = en;
      }
      uint32_t dk[2][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float p0 = __builtin_amdgcn_exp2f(s2[h][0]), p1 = __builtin_amdgcn_exp2f(s2[h][1]);
        const float p2 = __builtin_amdgcn_exp2f(s2[h][2]), p3 = __builtin_amdgcn_exp2f(s2[h][3]);
        dk[h][0] = pack2h_rne(p0 * y2[h][0], p1 * y2[h][1]);
        dk[h][1] = pack2h_rne(p2 * y2[h][2], p3 * y2[h][3]);
      }
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(dk[0][0], dk[0][1], dk[1][0], dk[1][1]));
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const f16x8 kt = __builtin_bit_cast(f16x8, make_uint4(ktl[t].x, ktl[t].y, kth[t].x, kth[t].y));
        o[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kt, df, o[j][t], 0, 0, 0);
      }
    }
  };

  // all query levels of this wave whose window holds key level p
  auto compute = [&](int p, const char* tk, const char* tv) {
#pragma unroll
    for (int j = 0; j < C::QL; ++j) {
      const int zq = z0 + grp + NG * j;
      if (zq >= Z) continue;
      const int zs = win_start(zq, Z, KZ);
      if (p < zs || p >= zs + KZ) continue;
      if constexpr (BWD) update_dq(j, tk, tv);
      else update(j, p == zs, tk, tv);
    }
  };

  // ---- normalise and store --------------------------------------------------------
  auto end_group = [&]() __attribute__((always_inline)) {
    const bool in_grid = qy_raw < H && qx_raw < W;
#pragma unroll
    for (int j = 0; j < C::QL; ++j) {
      const int zq = z0 + grp + NG * j;
      if constexpr (BWD) {
        // dQ = R^T (scale 2^(E-15) dQ~); lane holds d = 16t + 4g + i.  With QK
        // RMSNorm that is the gradient of q^ = r q, carried back through the
        // norm: dq = r (dq^ - q^ mean(dq^ q^)), q^ from the raw row in float32.
        const float f = a.scale * __builtin_amdgcn_ldexpf(1.f, ex[j] - 15);
        const int64_t tok = bh_base + min(zq, Z - 1) * HW + (int64_t)qy * W + qx;
        f32x4 x[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          x[t] = o[j][t] * f;
          if (csq) {
            const float4 ph = csq[4 * t + g];  // pairs 8t+2g and 8t+2g+1
            const float r0 = fmaf(x[t][0], ph.x, x[t][1] * ph.y), r1 = fmaf(x[t][1], ph.x, -x[t][0] * ph.y);
            const float r2 = fmaf(x[t][2], ph.z, x[t][3] * ph.w), r3 = fmaf(x[t][3], ph.z, -x[t][2] * ph.w);
            x[t] = f32x4{r0, r1, r2, r3};
          }
        }
        if constexpr (NORM) {
          const uint2* qr = reinterpret_cast<const uint2*>(a.q + tok * kD);
          f32x4 qh[4];
          float c = 0.f;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const uint2 w = qr[4 * t + g];
            qh[t] = f32x4{lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y)} * rq[j];
#pragma unroll
            for (int i = 0; i < 4; ++i) c = fmaf(x[t][i], qh[t][i], c);
          }
          c = sum_over_rows(c) * (1.f / kD);
#pragma unroll
          for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) x[t][i] = rq[j] * fmaf(-qh[t][i], c, x[t][i]);
        }
        if (zq >= Z || !in_grid) continue;
        uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
#pragma unroll
        for (int t = 0; t < 4; ++t) dst[4 * t + g] = make_uint2(pack2(x[t][0], x[t][1]), pack2(x[t][2], x[t][3]));
      } else {
        const float lt = sum_over_rows(l[j]);
        if (zq >= Z || !in_grid) continue;
        float inv = 1.f / lt;
        const int64_t tok = bh_base + zq * HW + (int64_t)qy * W + qx;
        uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
        if constexpr (GATE)
          if (a.gate_dim == 1) inv *= sigmoid_fast(bf16_to_f32(a.gate[tok]));
#pragma unroll
        for (int t = 0; t < 4; ++t) {  // d = 16t + 4g + i
          f32x4 r = o[j][t] * inv;
          if constexpr (GATE)
            if (a.gate_dim != 1) r *= sigmoid4_bf16(reinterpret_cast<const uint2*>(a.gate + tok * kD)[4 * t + g]);
          dst[4 * t + g] = make_uint2(pack2(r[0], r[1]), pack2(r[2], r[3]));
        }
        if (a.lse && g == 0) a.lse[tok] = (m[j] + __log2f(lt)) * kLn2;
      }
    }
  };

  // ---- the groups' key levels, double-buffered ----------------------------------
  // Group zb needs the key levels [kp_lo(zb), kp_hi(zb)); the workgroup walks
  // them group after group, copying the next (group, key level) while the
  // current one is computed, so the copies keep running across the end of a
  // group.  Each thread waits for its own copies, rotates its own K slots, and
  // one barrier publishes the level; the barrier also retires every read of the
  // tiles the next copy overwrites.
  auto kp_lo = [&](int zb) { return win_start(zb * ZQ, Z, KZ); };
  auto kp_hi = [&](int zb) { return win_start(min(zb * ZQ + ZQ, Z) - 1, Z, KZ) + KZ; };
  auto next_of = [&](int zb, int p, int& nz, int& np) {
    nz = zb;
    np = p + 1;
    if (np >= kp_hi(zb)) {
      nz = zb + 1;
      np = nz < zb_hi ? kp_lo(nz) : 0;
    }
  };
  auto change_group = [&](int nz, bool more) __attribute__((always_inline)) {
    end_group();
    if (more) {
      z0 = nz * ZQ;
      begin_group();
    }
  };
  int cz = zb_lo, cp = kp_lo(zb_lo);
  issue_copy(cp, tK0, tV0);
  __builtin_amdgcn_s_waitcnt(0);
  rotate_k(tK0);
  __syncthreads();
  for (;;) {
    int nz, np;
    next_of(cz, cp, nz, np);
    bool more = nz < zb_hi;
    if (more) issue_copy(np, tK1, tV1);
    compute(cp, tK0, tV0);
    if (nz != cz) change_group(nz, more);
    if (!more) break;
    __builtin_amdgcn_s_waitcnt(0);
    rotate_k(tK1);
    __syncthreads();
    cz = nz;
    cp = np;
    next_of(cz, cp, nz, np);
    more = nz < zb_hi;
    if (more) issue_copy(np, tK0, tV0);
    compute(cp, tK1, tV1);
    if (nz != cz) change_group(nz, more);
    if (!more) break;
    __builtin_amdgcn_s_waitcnt(0);
    rotate_k(tK0);
    __syncthreads();
    cz = nz;
    cp = np;
  }
  if constexpr (BWD && !LO) {
    if (a.emax) {  // the exponent of the wave's largest |dO|, one atomic per wave
      float wm = max_over_rows(gmx);
#pragma unroll
      for (int o2 = 8; o2 > 0; o2 >>= 1) wm = fmaxf(wm, __shfl_xor(wm, o2));
      if (lane == 0 && wm > 0.f) atomicMax(a.emax + bh, __builtin_amdgcn_frexp_expf(wm));
    }
  }
}

// the empty value of the per-(batch, head) dO exponents before the dQ pass
__global__ void __launch_bounds__(256) emax_init_kernel(int* e, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) e[i] = kEmaxEmpty;
}

Args make_args(const strata_na3d_desc& d, int zq, const void* q, const void* k, const void* v,
               const float* cs) {
  Args a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.heads = d.heads;
  a.Z = d.Z;
  a.H = d.H;
  a.W = d.W;
  a.n_zb = (d.Z + zq - 1) / zq;
  a.n_yb = (d.H + kBY - 1) / kBY;
  a.n_xb = (d.W + kBX - 1) / kBX;
  // a workgroup walks a whole column of query-level groups (the setup is paid
  // once, and the key copies run on across groups) unless that leaves fewer
  // than 1024 workgroups: then the column is cut into runs
  const int64_t cols = (int64_t)d.B * d.heads * a.n_yb * a.n_xb;
  a.n_zc = 1;
  while (a.n_zc < a.n_zb && cols * a.n_zc < 1024) ++a.n_zc;
  a.zb_per = (a.n_zb + a.n_zc - 1) / a.n_zc;
  a.n_zc = (a.n_zb + a.zb_per - 1) / a.zb_per;
  a.qscale = d.scale * kLog2e;
  a.scale = d.scale;
  return a;
}

template <int KZ, int KY, int KX, int ZQ, bool BWD, int NG = 2>
bool launch(const strata_na3d_desc& d, const Args& a, int opt, hipStream_t s) {
  int64_t blocks = (int64_t)d.B * d.heads * a.n_zc * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  const dim3 grid((unsigned)blocks), block(Cfg<KZ, KY, KX, ZQ, BWD, NG>::kThreads);
  switch (opt) {
    case 0: hipLaunchKernelGGL((na3d_mfma_q_kernel<KZ, KY, KX, ZQ, BWD, 0, NG>), grid, block, 0, s, a); break;
    case 1: hipLaunchKernelGGL((na3d_mfma_q_kernel<KZ, KY, KX, ZQ, BWD, 1, NG>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((na3d_mfma_q_kernel<KZ, KY, KX, ZQ, BWD, 2, NG>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((na3d_mfma_q_kernel<KZ, KY, KX, ZQ, BWD, 3, NG>), grid, block, 0, s, a); break;
  }
  return true;
}

bool supported(const strata_na3d_desc& d) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  // element offsets inside one key level are int32
  return (int64_t)d.H * d.W * kD < (int64_t)1 << 31;
}

}  // namespace

bool launch_na3d_fwd_mfma(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                          const void* v, const float* cs, void* out, float* lse, hipStream_t s) {
  if (!supported(d)) return false;
  const bool w377 = d.kz == 3 && d.ky == 7 && d.kx == 7, w599 = d.kz == 5 && d.ky == 9 && d.kx == 9;
  const bool w999 = d.kz == 9 && d.ky == 9 && d.kx == 9;
  if (!w377 && !w599 && !w999) return false;
  Args a = make_args(d, w599 ? 2 : (w999 ? 6 : 8), q, k, v, cs);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.qk_norm = o.qk_norm;
  a.eps = o.eps;
  a.gate = static_cast<const uint16_t*>(o.gate);
  a.gate_dim = o.gate_dim;
  const int opt = (o.qk_norm ? kNorm : 0) | (o.gate ? kOpt2 : 0);
  if (w377) return launch<3, 7, 7, 8, false>(d, a, opt, s);
  if (w999) return launch<9, 9, 9, 6, false>(d, a, opt, s);
  return launch<5, 9, 9, 2, false>(d, a, opt, s);
}

bool na3d_bwd_dq_mfma_takes(const strata_na3d_desc& d) {
  if (!supported(d)) return false;
  const bool w377 = d.kz == 3 && d.ky == 7 && d.kx == 7, w599 = d.kz == 5 && d.ky == 9 && d.kx == 9;
  const bool w999 = d.kz == 9 && d.ky == 9 && d.kx == 9;
  if (!w377 && !w599 && !w999) return false;
  const Args a = make_args(d, w377 ? 4 : 3, nullptr, nullptr, nullptr, nullptr);
  return (int64_t)d.B * d.heads * a.n_zc * a.n_yb * a.n_xb < (int64_t)1 << 31;
}

bool launch_na3d_bwd_dq_mfma(const strata_na3d_desc& d, const BwdOpts& o, const void* q,
                             const void* k, const void* v, const float* cs, const void* dout,
                             const float* lse, float* dvec, const void* out, int* emax, void* dq,
                             hipStream_t s) {
  if (!na3d_bwd_dq_mfma_takes(d)) return false;
  if (out && o.dout_lo) return false;  // D of a two-term dO comes from the gate's pass
  const bool w377 = d.kz == 3 && d.ky == 7 && d.kx == 7;
  const bool w999 = d.kz == 9 && d.ky == 9 && d.kx == 9;
  // 9-wide windows: three groups of four waves, one query level each (12 waves,
  // three per SIMD); 3x7x7: two groups, two levels per wave
  Args a = make_args(d, w377 ? 4 : 3, q, k, v, cs);
  a.out = static_cast<uint16_t*>(dq);
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse_in = lse;
  a.dvec = dvec;
  if (out) {  // D formed from dO and O by this pass and stored to dvec
    a.fo = static_cast<const uint16_t*>(out);
    a.dvec_out = dvec;
  }
  if (emax && !o.dout_lo) {
    const int n = d.B * d.heads;
    hipLaunchKernelGGL(emax_init_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, emax, n);
    a.emax = emax;
  }
  a.qk_norm = o.qk_norm;
  a.eps = o.eps;
  a.dout_lo = static_cast<const uint16_t*>(o.dout_lo);
  const int opt = (o.qk_norm ? kNorm : 0) | (o.dout_lo ? kOpt2 : 0);
  if (w377) return launch<3, 7, 7, 4, true>(d, a, opt, s);
  if (w999) return launch<9, 9, 9, 3, true, 3>(d, a, opt, s);
  return launch<5, 9, 9, 3, true, 3>(d, a, opt, s);
}

}  // namespace strata

// Neighbourhood-attention forward for gfx950 with a level sweep: window 3 x 7 x 7,
// Z = 8 levels (every option, and the stitch of the face step) or Z = 24 (no
// options: the paper's 24-level stack), head_dim 64, bf16 in/out, StereoRoPE
// fused into the Q/K loads.  The whole sweep is unrolled per Z (the 24-level
// kernel is ~170 KB of code and measured 1.97 ms against the grouped sweep's
// 2.92 ms on 24 tiles x 16 heads x 24 x 32 x 32).
//
// Work decomposition
//   workgroup : one tile, an 8 x 8 block of (y, x) query positions, all Z levels,
//               and a run of heads processed one after the other; 4 waves (one
//               per SIMD), one workgroup per CU.  Consecutive heads share every
//               piece of geometry (key box, window masks, copy offsets, rotary
//               phases), so it is set up once and the key-level pipeline runs on
//               from one head into the next without draining.
//   wave      : a 4 x 4 (y, x) sub-block = 16 queries, on all Z levels.
//   key sweep : per head the workgroup walks the Z key levels once.  K and V of
//               the 14 x 14 key box of a level are copied global -> LDS by the
//               direct-to-LDS load one level ahead of the compute (double
//               buffer; the copies are spread over the first two query levels
//               of the current key level); once its query levels are issued,
//               each thread waits for its own copies, rotates the K pieces they
//               brought (StereoRoPE in packed float16, with the float16 phases
//               of the key box staged once in LDS) and converts the V pieces to
//               float16; the barrier at the end of the key level publishes the
//               next one.
//               Queries are rotated in float32 with float32 phases and the logit
//               scale times log2 e, then rounded to float16 once: an exact scale
//               matters, a scale rounded to float16 shifts every logit by up to
//               2^-11 relative, which moves sharp softmax rows visibly.
//
// K rows are 128 bytes with their 16-byte columns XOR-swizzled by
// ((x >> 1) + 5 y) & 7 of the key's box position (the 16 keys of a chunk hit 16
// bank groups); V rows are 160 bytes (8 data columns + 2 pad columns), which
// spreads the transpose reads and lets them take immediate offsets.  Every
// thread owns 7 K slots and 8 V slots of 16 bytes per level, with their global
// offsets in registers; the tiles carry the pad slots of the last pass and V's
// pad columns copy a valid column, so no copy or rotation needs a branch.
//
// At key level p a wave reads the K and V fragments of its sub-block's key box
// from LDS once and applies them to every query level whose window holds p
// (two to four of them).  Per (query level, key level):
//   S^T (16 keys x 16 queries) = K . Q^T   two 16x16x32 float16 MFMAs of the
//                                         rotated, scaled K and the rotated Q,
//                                         the accumulator seeded with the window
//                                         mask (0 or -inf);
//   P = exp2(S^T - m) packed to float16 in place;
//   O^T (64 d x 16 queries) += V^T . P^T  float16 MFMA, V^T fragments by the
//                                         LDS transpose read of V converted to
//                                         float16 when it is staged;
//   L (16 x 16 queries)     += 1 . P^T    the row sums, by one more float16 MFMA
//                                         against a tile of ones (every row of
//                                         L holds the sum, so each lane has its
//                                         query's sum without a reduction).
// P.V runs in float16 rather than bf16: rounding the weights P to bf16 (8
// significant bits) moved outputs by up to 2.2% of their RMS beyond their own
// storage rounding on the 8-tile workload (checked on every output, and
// reproduced by a CPU emulation of these roundings), float16 weights (11 bits)
// by 0.7%.  The reference m starts at 0 for every query and moves up when a
// logit exceeds it by more than 15 (O and the row sum are then rescaled), so
// P <= 2^15 stays inside float16; on a query level's first key level it moves
// down when no logit reaches -8 (nothing is accumulated yet), so the largest
// weight is at least 2^-8 and the small ones keep their relative size; while m
// is 0 for the whole wave (the common case for logits of moderate size) no
// subtraction is done.
// Every accumulator chain uses one MFMA shape only (the last 16-key chunk of
// the P.V product is padded with zero weights rather than switching to a
// 16x16x16 MFMA): gfx950 gives wrong sums when an accumulator is handed from
// one MFMA shape to another without wait states, which the compiler does not
// insert.
//
// Input range: V is converted to float16 by round-toward-zero (exact for bf16
// values of magnitude 2^-14 .. 65504, saturating above, float16's subnormal
// spacing below).  K is converted to float16 with round-toward-zero before its
// rotation (bf16 values up to +-65504 convert exactly, larger ones saturate) and
// rotated by phases of half length (c/2, s/2), so a rotated pair stays below
// 65504 sqrt(2) / 2 and never overflows; the queries carry the factor 2 instead:
// 2 scale log2(e) q is rounded to float16, saturating at +-65504.
//
// Options (App. B.5).  QK RMSNorm: the factor (mean square + eps)^(-1/2) of a
// query comes from the sums of squares of the 4 lanes holding its row, that of
// a key from the 8 lanes whose copies brought its row; each scales its vector
// in float32 before the float16 rounding.  (The normalised logits are bounded
// by scale log2(e) head_dim, which would allow a constant reference m; measured,
// that variant is slower than the lazy reference above, so the softmax is the
// same with and without the norm.)  Output gate: the logits of a query level
// are loaded at the start of its last key level (later loads leave their
// latency exposed, measured) and sigmoid(g) multiplies the normalised output
// at the store.
//
// Stitch (App. F, Eq. stitch).  When the batch is the regular tiling of one
// face, a query cell that no other tile covers is stored straight into the face
// (its stitch is the tile's own value, 0 where its weight is 0, with -0 turned
// into +0 as the stitch's multiply-add from +0 does); the other cells go to the
// tile output for the overlap stitch.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

namespace strata {
namespace {

using namespace mfma;

constexpr int kThreads = 256;
constexpr int KZ = 3, KY = 7, KX = 7;
constexpr int kBY = 8, kBX = 8;
constexpr int kD = 64;
constexpr int LY = kBY + KY - 1, LX = kBX + KX - 1;       // staged key box per level (14 x 14)
constexpr int NUY = 3 + KY, NUX = 3 + KX, NU = NUY * NUX;  // key box of a 4x4 sub-block (10 x 10)
constexpr int NC = (NU + 15) / 16;                         // 16-key chunks (7)
constexpr int NS = (NC + 1) / 2;                           // 32-key P.V steps (4)
constexpr int KEYS = LY * LX;
constexpr int kKRow = 128, kVRow = 160;                    // LDS bytes per key row
constexpr int KSLOTS = KEYS * (kKRow / 16), VSLOTS = KEYS * (kVRow / 16);  // 16-byte slots
constexpr int ITK = (KSLOTS + kThreads - 1) / kThreads;    // K slots per thread (7)
constexpr int ITV = (VSLOTS + kThreads - 1) / kThreads;    // V slots per thread (8)
constexpr int KTILE = ITK * kThreads * 16;                 // tile bytes incl. pad slots
constexpr int VTILE = ITV * kThreads * 16;
constexpr float kLazy = 15.0f;    // m moves up when a logit exceeds it by 15 (P <= 2^15)
constexpr float kLow = -8.0f;     // ... or down, on a level's first key level (max P >= 2^-8)
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLog2e = 1.4426950408889634f;

static_assert(3 * KTILE + 2 * VTILE <= 160 * 1024, "LDS budget");
static_assert(ITK <= NC + 1 && ITV <= NC + 1, "copies are spread over the chunks of two query levels");

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

// first key level of query level z (border-clamped window along the levels)
template <int Z>
__host__ __device__ constexpr int zstart(int z) {
  return z - KZ / 2 < 0 ? 0 : (z - KZ / 2 > Z - KZ ? Z - KZ : z - KZ / 2);
}
// query levels whose window holds key level p: the consecutive range [zlo, zhi]
template <int Z>
__host__ __device__ constexpr int zlo(int p) {
  int z = 0;
  while (zstart<Z>(z) + KZ <= p) ++z;
  return z;
}
template <int Z>
__host__ __device__ constexpr int zhi(int p) {
  int z = Z - 1;
  while (zstart<Z>(z) > p) --z;
  return z;
}

struct ZArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;   // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  uint16_t* out;
  float* lse;         // optional
  int heads, H, W;
  int n_yb, n_xb, n_hg, hpw;
  float qscale;       // 2 scale log2(e) (K enters at half length)
  // options: QK RMSNorm (eps) and the sigmoid output gate
  float eps;
  const uint16_t* gate;
  int gate_dim;
  // stitch into the face: the tiles of the batch form an nty x ntx regular
  // tiling with strides (sy, sx) of a face [heads Z, Hf, Wf, 64]; cells that
  // one tile alone covers go to the face, the others to `out`
  uint16_t* face;
  const float* window;  // [H, W] stitch weights
  int nty, ntx, sy, sx, Hf, Wf;
};

// A bf16 pair with each -0 half turned into +0: the stitch of a cell covered by
// one tile returns w v / w, which is v for every value except -0 (its fused
// multiply-add starts from +0).  Magnitude m = bits & 0x7fff; m + 0x7fff sets
// bit 15 exactly when m > 0, and the sign survives only there.
__device__ __forceinline__ uint32_t plus_zero2(uint32_t w) {
  const uint32_t m = w & 0x7fff7fffu;
  const uint32_t keep = ((m + 0x7fff7fffu) & 0x80008000u) | 0x7fff7fffu;
  return w & keep;
}

// The stitch of a bf16 pair that one tile alone covers with weight w > 0, as
// the stitch computes it: fma(w, v, +0) / w, correctly rounded, to bf16.
__device__ __forceinline__ uint32_t stitch_one2(uint32_t v, float w) {
  const float lo = __builtin_fmaf(w, lo_bf16(v), 0.f) / w;
  const float hi = __builtin_fmaf(w, hi_bf16(v), 0.f) / w;
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// Rotate 4 pairs of K held as packed bf16x2 words by packed float16 phases
// (c, s): round-toward-zero to float16 (exact for bf16 values inside the
// float16 range, saturating outside it), then in packed float16, the products
// taking the halves of the phase word through the operand selects,
//   t = (a c, a s),   r = (b, b) * (s, c) * (-1, 1) + t = (a c - b s, a s + b c).
// With `mul` (the QK RMSNorm factor) the values are scaled in float32 first.
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

template <int Z, bool NORM, bool GATE, bool STITCH>
__global__ void __launch_bounds__(kThreads, 1) na3d_fwd_zs_kernel(ZArgs a) {
  __shared__ __attribute__((aligned(16))) char tK0[KTILE];
  __shared__ __attribute__((aligned(16))) char tV0[VTILE];
  __shared__ __attribute__((aligned(16))) char tK1[KTILE];
  __shared__ __attribute__((aligned(16))) char tV1[VTILE];
  __shared__ __attribute__((aligned(16))) char sph[KTILE];

  // ---- block coordinates (XCD-aware: neighbouring blocks share an L2) -------
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int xb = bid % a.n_xb;
  const int yb = (bid / a.n_xb) % a.n_yb;
  const int hg = (bid / (a.n_xb * a.n_yb)) % a.n_hg;
  const int b = bid / (a.n_xb * a.n_yb * a.n_hg);
  const int h_lo = hg * a.hpw;
  const int h_hi = min(h_lo + a.hpw, a.heads);
  const int H = a.H, W = a.W;
  const int64_t HW = (int64_t)H * W;
  const int by0 = yb * kBY, bx0 = xb * kBX;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, qn = lane & 15;

  const int ty0 = win_start(min(by0, H - 1), H, KY);
  const int tx0 = win_start(min(bx0, W - 1), W, KX);
  const int sy0 = by0 + 4 * (wave >> 1), sx0 = bx0 + 4 * (wave & 1);
  const int uy0 = win_start(min(sy0, H - 1), H, KY);
  const int ux0 = win_start(min(sx0, W - 1), W, KX);
  const int qy_raw = sy0 + (qn >> 2), qx_raw = sx0 + (qn & 3);
  const int qy = min(qy_raw, H - 1), qx = min(qx_raw, W - 1);
  const bool in_grid = qy_raw < H && qx_raw < W;
  // stitch: a cell no other tile of the tiling covers (sy <= H <= 2 sy, and
  // likewise along x) takes this tile's value, or 0 where its weight is 0
  bool direct = false, wzero = false, wexact = true;
  float wcell = 0.f;
  int64_t fcell = 0;
  if constexpr (STITCH) {
    const int ta = b / a.ntx, tb = b - ta * a.ntx;
    const bool one_y = !(ta > 0 && qy < H - a.sy) && !(ta < a.nty - 1 && qy >= a.sy);
    const bool one_x = !(tb > 0 && qx < W - a.sx) && !(tb < a.ntx - 1 && qx >= a.sx);
    direct = one_y && one_x;
    fcell = (int64_t)(ta * a.sy + qy) * a.Wf + (tb * a.sx + qx);
    wcell = a.window[qy * W + qx];
    wzero = wcell == 0.f;
    // for 2^-8 <= w <= 1, fl(fl(w v) / w) rounds back to v for every bf16 v (no
    // overflow, and an underflowing product keeps more than 8 significant bits),
    // so the tile value is stored as it is; other weights take the stitch's own
    // arithmetic
    wexact = wzero || (wcell >= 0x1p-8f && wcell <= 1.f);
  }

  auto kswz = [&](int key) { return ((key % LX >> 1) + 5 * (key / LX)) & 7; };
  auto key_row = [&](int u) {
    return u < NU ? (uy0 - ty0 + u / NUX) * LX + (ux0 - tx0 + u % NUX) : 0;
  };

  // ---- LDS addresses of this lane's fragments and its window mask ----------
  const int wys = win_start(qy, H, KY), wxs = win_start(qx, W, KX);
  uint32_t kaddr[NC], vaddr[NC];
  f32x4 bias[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    {  // K fragment (A operand): row = key 16c + qn, 16 bytes at column g (xor 64 bytes: g+4)
      const int key = key_row(16 * c + qn);
      kaddr[c] = key * kKRow + ((g ^ kswz(key)) << 4);
    }
    // V^T transpose read: row = key 16c + 4g + qn/4, 8 bytes at d = 4 (qn % 4) (+ 32 t: + 16 t)
    vaddr[c] = key_row(16 * c + 4 * g + (qn >> 2)) * kVRow + (qn & 3) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = 16 * c + 4 * g + i;
      const int ky = uy0 + u / NUX, kx = ux0 + u % NUX;
      const bool ok = u < NU && ky >= wys && ky < wys + KY && kx >= wxs && kx < wxs + KX;
      bias[c][i] = ok ? 0.f : -INFINITY;
    }
  }

  // ---- copy offsets (bytes inside a key level) and the rotary phases of this --
  // ---- thread's K slots ------------------------------------------------------
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * 16 : nullptr;
  auto pos_of = [&](int key) {  // grid position of a staged key (rows past the grid repeat the last)
    return min(ty0 + key / LX, H - 1) * W + min(tx0 + key % LX, W - 1);
  };
  uint32_t koff[ITK], voff[ITV];
#pragma unroll
  for (int it = 0; it < ITK; ++it) {
    const int s = it * kThreads + tid;
    const int key = min(s >> 3, KEYS - 1);  // pad slots copy a valid row into the pad
    const int c = (s & 7) ^ kswz(key);
    const int pos = pos_of(key);
    koff[it] = (uint32_t)(pos * kD + c * 8) * 2u;
    uint4 ph;
    if (csb) {  // half-length phases (exact halving): see the input range above
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
  // float32 phases of this lane's query position (pairs 4g..4g+3 and 16+4g..),
  // the same for every level and head: loaded once and kept (16 registers; a
  // reload at each key level left its latency exposed, 0.45 ms more per step)
  const float4* csq = csb ? csb + ((int64_t)qy * W + qx) * 16 : nullptr;
  float4 cqv[4] = {};
  if (csq) {
    cqv[0] = csq[2 * g];
    cqv[1] = csq[2 * g + 1];
    cqv[2] = csq[8 + 2 * g];
    cqv[3] = csq[8 + 2 * g + 1];
  }

  auto level_base = [&](int h, int p) { return (((int64_t)b * a.heads + h) * Z + p) * HW; };
  auto issue_copy = [&](int64_t base, char* tk, char* tv) {
    const char* kp = reinterpret_cast<const char*>(a.k + base * kD);
    const char* vp = reinterpret_cast<const char*>(a.v + base * kD);
#pragma unroll
    for (int it = 0; it < ITK; ++it)
      copy16_to_lds(reinterpret_cast<const uint16_t*>(kp + koff[it]), tk + (it * kThreads + wave * 64) * 16);
#pragma unroll
    for (int it = 0; it < ITV; ++it)
      copy16_to_lds(reinterpret_cast<const uint16_t*>(vp + voff[it]), tv + (it * kThreads + wave * 64) * 16);
  };
  // Rotate this thread's K slots in place (bf16 -> scaled float16) and convert
  // its V slots to float16.  A thread's copies land in its own slots, so its own
  // wait suffices.  With QK RMSNorm the 8 slots of a key row (8 consecutive
  // lanes) add their sums of squares for the row's factor.
  auto rotate_k = [&](char* tk, char* tv) {
    uint4 y[ITV];
#pragma unroll
    for (int it = 0; it < ITV; ++it) y[it] = ld16(tv + (it * kThreads + tid) * 16);
    uint4 x[ITK];  // all reads before any write: the slots are distinct, which the compiler cannot tell
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
  // raw query rows of one level (two 16-byte pieces per lane)
  auto load_q = [&](int h, int z, uint4& x0, uint4& x1) {
    const uint4* src = reinterpret_cast<const uint4*>(a.q + (level_base(h, z) + (int64_t)qy * W + qx) * kD);
    x0 = src[g];
    x1 = src[4 + g];
  };
  auto prep_q = [&](const float4* cq, uint4 x0, uint4 x1, f16x8& q0, f16x8& q1) {
    uint4 r0, r1;
    float mul = a.qscale;
    if constexpr (NORM)  // the 4 lanes of a query row hold its 64 values
      mul *= __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(x1, sumsq8(x0, 0.f))) * (1.f / kD) + a.eps);
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

  // per query level state (only the levels whose window holds the current key
  // level are live at any time)
  f16x8 qf[Z][2];
  float m[Z];
  f32x4 lsum[Z];    // row sums (all four entries equal)
  const f16x8 ones = __builtin_bit_cast(f16x8, make_uint4(0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u));
  bool mset[Z];     // wave-uniform: m is non-zero somewhere in the wave
  f32x4 o[Z][4];
  uint4 qraw[Z][2];
  uint2 gch[GATE ? Z : 1][4];  // gate logits (bf16) of a level, loaded at the start of its last key level
  uint32_t ghd[GATE ? Z : 1];

  // K and V fragments of one key level (shared by every active query level)
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

  // one query level z at key level p
  // `hook(c)` runs beside the logits of chunk c (c = 0..NC, the last one after
  // the chunk loop): the next level's copies are spread over the first two
  // query levels this way, since a burst of them stalls the issuing wave
  // until the memory pipeline has taken them all.
  auto update = [&](auto P, auto Zi, const Frags& f, auto&& hook) {
    constexpr int p = decltype(P)::v, z = decltype(Zi)::v;
    constexpr bool first = zstart<Z>(z) == p;
    f32x4 s[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      hook(c);
      const f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.k[c][0], qf[z][0], bias[c], 0, 0, 0);
      s[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.k[c][1], qf[z][1], acc, 0, 0, 0);
    }
    hook(NC);
    {
      float mx = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
      mx = fmaxf(fmaxf(mx, s[0][3]), s[1][0]);
#pragma unroll
      for (int c = 1; c < NC; ++c) {
        if (c > 1) mx = fmaxf(fmaxf(mx, s[c][0]), s[c][1]);
        else mx = fmaxf(mx, s[c][1]);
        mx = fmaxf(fmaxf(mx, s[c][2]), s[c][3]);
      }
      mx = max_over_rows(mx);
      const bool move = mx > m[z] + kLazy || (first && mx < kLow);
      if (__any(move)) {  // rare: move the reference m
        const float mn = move ? mx : m[z];
        if constexpr (!first) {  // nothing is accumulated before a level's first key level
          const float alpha = __builtin_amdgcn_exp2f(m[z] - mn);
          lsum[z] *= alpha;
#pragma unroll
          for (int t = 0; t < 4; ++t) o[z][t] *= alpha;
        }
        m[z] = mn;
        mset[z] = true;
      }
      if (mset[z]) {
#pragma unroll
        for (int c = 0; c < NC; ++c) s[c] -= m[z];
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
        o[z][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.v[st][t], pf, o[z][t], 0, 0, 0);
      lsum[z] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones, pf, lsum[z], 0, 0, 0);
    }
    // scheduling: four VALU instructions (the exponentials and packs of the
    // later chunks) after each P.V MFMA, instead of the exponentials in one run
    // ahead of them (measured on the face step: 10.24 -> 10.05 ms)
#pragma unroll
    for (int i = 0; i < 5 * NS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // four VALU
    }
  };

  // ---- prologue: key level 0 of the first head, queries of its first levels --
  issue_copy(level_base(h_lo, 0), tK0, tV0);
  static_for<Z>([&](auto Zi) {
    constexpr int z = decltype(Zi)::v;
    if constexpr (zstart<Z>(z) == 0) load_q(h_lo, z, qraw[z][0], qraw[z][1]);
  });
  __builtin_amdgcn_s_waitcnt(0);
  rotate_k(tK0, tV0);
  __syncthreads();

  for (int h = h_lo; h < h_hi; ++h) {
    const bool more_heads = h + 1 < h_hi;
    static_for<Z>([&](auto Pi) {
      constexpr int p = decltype(Pi)::v;
      char* const tk = (p & 1) ? tK1 : tK0;
      char* const tv = (p & 1) ? tV1 : tV0;
      char* const nk = (p & 1) ? tK0 : tK1;
      char* const nv = (p & 1) ? tV0 : tV1;
      const bool has_next = p + 1 < Z || more_heads;
      // Addresses derived from these per-lane constants are recomputed at every
      // key level (a few adds) instead of being kept live across the whole
      // sweep, which would crowd out the registers of the attention itself.
#pragma unroll
      for (int c = 0; c < NC; ++c) asm volatile("" : "+v"(kaddr[c]), "+v"(vaddr[c]));
#pragma unroll
      for (int it = 0; it < ITK; ++it) asm volatile("" : "+v"(koff[it]));
#pragma unroll
      for (int it = 0; it < ITV; ++it) asm volatile("" : "+v"(voff[it]));
      // the next key level (this head's p+1, or the next head's level 0) is
      // staged by copies spread over the first two query levels below
      const int64_t nbase = p + 1 < Z ? level_base(h, p + 1) : level_base(h + 1, 0);
      const char* const nkp = reinterpret_cast<const char*>(a.k + nbase * kD);
      const char* const nvp = reinterpret_cast<const char*>(a.v + nbase * kD);

      // queries of the levels that start here: rotate the rows loaded earlier
      static_for<Z>([&](auto Zi) {
        constexpr int z = decltype(Zi)::v;
        if constexpr (zstart<Z>(z) == p) {
          prep_q(csq, qraw[z][0], qraw[z][1], qf[z][0], qf[z][1]);
          m[z] = 0.f;
          lsum[z] = f32x4{0.f, 0.f, 0.f, 0.f};
          mset[z] = false;
#pragma unroll
          for (int t = 0; t < 4; ++t) o[z][t] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      });
      // prefetch the query rows of the levels that start at the next key level
      static_for<Z>([&](auto Zi) {
        constexpr int z = decltype(Zi)::v;
        if constexpr (p + 1 < Z && zstart<Z>(z) == p + 1) load_q(h, z, qraw[z][0], qraw[z][1]);
        if constexpr (p + 1 == Z && zstart<Z>(z) == 0)
          if (more_heads) load_q(h + 1, z, qraw[z][0], qraw[z][1]);
      });

      // gate logits of the levels that end at this key level (used at their
      // store; loaded this early, their latency stays hidden)
      if constexpr (GATE) {
        static_for<Z>([&](auto Zi) {
          constexpr int z = decltype(Zi)::v;
          if constexpr (zstart<Z>(z) + KZ - 1 == p) {
            const int64_t tok = level_base(h, z) + (int64_t)qy * W + qx;
            if (a.gate_dim == 1) {
              ghd[z] = a.gate[tok];
            } else {
              const uint2* src = reinterpret_cast<const uint2*>(a.gate + tok * kD);
#pragma unroll
              for (int t = 0; t < 4; ++t) gch[z][t] = src[4 * t + g];
            }
          }
        });
      }

      // ---- the active query levels [zlo, zhi], sharing this level's fragments -
      // After the last of them, wait for the next level's copies (issued at the
      // start of this level) and rotate its K slots; the rotation can run beside
      // the tail of this level's MFMA work.
      {
        Frags f;
        load_frags(tk, tv, f);
        static_for<Z>([&](auto Zi) {
          constexpr int z = decltype(Zi)::v;
          if constexpr (zlo<Z>(p) <= z && z <= zhi<Z>(p)) {
            update(IC<p>{}, Zi, f, [&](int c) {
              if constexpr (z == zlo<Z>(p)) {  // K copies
                if (has_next && c < ITK)
                  copy16_to_lds(reinterpret_cast<const uint16_t*>(nkp + koff[c]), nk + (c * kThreads + wave * 64) * 16);
              } else if constexpr (z == zlo<Z>(p) + 1) {  // V copies
                if (has_next && c < ITV)
                  copy16_to_lds(reinterpret_cast<const uint16_t*>(nvp + voff[c]), nv + (c * kThreads + wave * 64) * 16);
              }
            });
            if constexpr (z == zhi<Z>(p)) {
              if (has_next) {
                __builtin_amdgcn_s_waitcnt(0);
                rotate_k(nk, nv);
              }
            }
          }
        });
      }

      // ---- query levels whose last key level this was: normalise and store ---
      static_for<Z>([&](auto Zi) {
        constexpr int z = decltype(Zi)::v;
        if constexpr (zstart<Z>(z) + KZ - 1 == p) {
          const float lt = lsum[z][0];
          if (in_grid) {
            float inv = 1.f / lt;
            if constexpr (GATE)
              if (a.gate_dim == 1) inv *= sigmoid_fast(__uint_as_float(ghd[z] << 16));
            const int64_t tok = level_base(h, z) + (int64_t)qy * W + qx;
            uint2* dst = reinterpret_cast<uint2*>(a.out + tok * kD);
            if constexpr (STITCH)
              if (direct)
                dst = reinterpret_cast<uint2*>(a.face + ((int64_t)(h * Z + z) * a.Hf * a.Wf + fcell) * kD);
#pragma unroll
            for (int t = 0; t < 4; ++t) {  // d = 16t + 4g + i
              f32x4 r = o[z][t] * inv;
              if constexpr (GATE)
                if (a.gate_dim != 1) r *= sigmoid4_bf16(gch[z][t]);
              uint32_t w0 = pack2(r[0], r[1]), w1 = pack2(r[2], r[3]);
              if constexpr (STITCH)
                if (direct) {
                  if (wexact) {
                    w0 = wzero ? 0u : plus_zero2(w0);
                    w1 = wzero ? 0u : plus_zero2(w1);
                  } else {
                    w0 = stitch_one2(w0, wcell);
                    w1 = stitch_one2(w1, wcell);
                  }
                }
              dst[4 * t + g] = make_uint2(w0, w1);
            }
            if (a.lse && g == 0) a.lse[tok] = (m[z] + __log2f(lt)) * kLn2;
          }
        }
      });

      __syncthreads();
    });
  }
}

}  // namespace

// Level-sweep forward for the 3x7x7 window at Z = 8, and at Z = 24 without
// options (bf16, head_dim 64); false when the problem is not that shape.  With `st` (a regular tiling of one face,
// sy <= H <= 2 sy, sx <= W <= 2 sx, checked by the caller) the cells one tile
// alone covers are stored into st->face instead of `out`.
bool launch_na3d_fwd_zs(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                        const void* v, const float* cs, void* out, float* lse, hipStream_t s,
                        const StitchArgs* st) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  if (d.kz != KZ || d.ky != KY || d.kx != KX || (d.Z != 8 && d.Z != 24)) return false;
  if (d.Z == 24 && (o.qk_norm || o.gate || st)) return false;
  if ((int64_t)d.H * d.W * kD * 2 >= (int64_t)1 << 32) return false;  // byte offsets in 32 bits
  ZArgs a = {};
  a.eps = o.eps;
  a.gate = static_cast<const uint16_t*>(o.gate);
  a.gate_dim = o.gate_dim;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.heads = d.heads;
  a.H = d.H;
  a.W = d.W;
  a.n_yb = (d.H + kBY - 1) / kBY;
  a.n_xb = (d.W + kBX - 1) / kBX;
  // a run of up to 8 heads per workgroup shares its geometry; a small problem
  // takes fewer, so that the grid still has two workgroups per CU
  a.hpw = d.heads < 8 ? d.heads : 8;
  while (a.hpw > 1 && (int64_t)d.B * ((d.heads + a.hpw - 1) / a.hpw) * a.n_yb * a.n_xb < 512)
    a.hpw = (a.hpw + 1) / 2;
  a.n_hg = (d.heads + a.hpw - 1) / a.hpw;
  a.qscale = 2.f * d.scale * kLog2e;  // K is rotated at half length
  if (st) {
    a.face = static_cast<uint16_t*>(st->face);
    a.window = st->window;
    a.nty = st->nty;
    a.ntx = st->ntx;
    a.sy = st->sy;
    a.sx = st->sx;
    a.Hf = st->Hf;
    a.Wf = st->Wf;
  }
  const int64_t blocks = (int64_t)d.B * a.n_hg * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  const dim3 grid((unsigned)blocks), block(kThreads);
  const int variant = (o.qk_norm ? 1 : 0) | (o.gate ? 2 : 0) | (st ? 4 : 0);
  if (d.Z == 24) {
    hipLaunchKernelGGL((na3d_fwd_zs_kernel<24, false, false, false>), grid, block, 0, s, a);
    return true;
  }
  switch (variant) {
    case 0: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, false, false, false>), grid, block, 0, s, a); break;
    case 1: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, true, false, false>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, false, true, false>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, true, true, false>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, false, false, true>), grid, block, 0, s, a); break;
    case 5: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, true, false, true>), grid, block, 0, s, a); break;
    case 6: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, false, true, true>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((na3d_fwd_zs_kernel<8, true, true, true>), grid, block, 0, s, a); break;
  }
  return true;
}

}  // namespace strata

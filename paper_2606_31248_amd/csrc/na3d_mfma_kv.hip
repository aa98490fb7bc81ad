// MFMA neighbourhood attention for gfx950, key-stationary kernel: the dK and dV
// part of the backward (bf16 in/out, head_dim 64).
//
// Work decomposition
//   workgroup : one (tile, head), a 4 x 4 block of (y, x) key positions and ZK key
//               levels; ZK waves, one per key level (ZK = 8 with a double buffer,
//               one workgroup per CU; ZK = 4 with a single buffer, two per CU).
//   wave      : the 16 keys of its level, stationary in registers: K~ (rotated,
//               times scale log2(e), float16) and V (bf16) as B operands, the
//               dK~^T and dV^T accumulators (64 d x 16 keys).
//   query sweep: the workgroup walks the query levels whose windows reach its key
//               levels, each once.  The queries that can see any key of the
//               block form a box per level -- the union of the per-axis inverse
//               windows [lo(j), hi(j)] (at most 4 + 3 r wide, checked on the
//               host).  Q and dO of that box are copied global -> LDS by the
//               direct-to-LDS load (one level ahead into the double buffer, or
//               into the single buffer between two barriers); each
//               thread rotates the Q pieces its own copies brought (StereoRoPE,
//               float16), stores LSE (log2 units) and -D of its queries, and one
//               barrier publishes the level.
//
// Per (key level, query level) a wave walks the box in steps of 32 queries:
//   X (16 queries x 16 keys) = Q~ . K~^T     float16 MFMA seeded with -LSE (or
//                                            -inf outside the query's window),
//                                            so P = exp2(X);
//   Y (16 queries x 16 keys) = dO . V^T - D  bf16 MFMA seeded with -D;
//   dV^T (64 d x 16 keys) += dO^T . P        bf16, P packed in place (k order of
//                                            two 16-query chunks, matched by the
//                                            transpose reads of the dO rows);
//   dK~^T (64 d x 16 keys) += Q~^T . dS      float16, dS = P Y carried with a
//                                            per-key power-of-two scale 2^(15-E),
//                                            E bounding |Y| seen so far (|dS| <=
//                                            P |Y|, P <= 1); the accumulator is
//                                            rescaled exactly when E grows.
// At the end dK = R^T (scale 2^(E-15) dK~) and dV is stored as is.
//
// Options: QK RMSNorm scales the stationary keys and the staged queries in
// float32 before their float16 rounding and applies the norm's Jacobian to dK
// before the store; a two-term dO = hi + lo (the gated upstream gradient) is
// staged as a third tile and adds one MFMA to Y and one to dV per step.
//
// Staged rows are 128 bytes (Q~ in float16, dO in bf16) with their 16-byte
// columns XOR-swizzled by sigma(u) = ((u >> 1) & 3) << 1 | ((u >> 3) & 1) of the
// box index u: the 16 rows of a chunk read at one column hit 16 distinct bank
// groups, and so do the 8 rows of a half-wave's transpose reads.  Rows past the
// box (up to the next multiple of 32) are zero and their mask bits clear, so
// every read address is a lane constant plus an immediate.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

#include <algorithm>

namespace strata {
namespace {

using namespace mfma;

constexpr int kD = 64;           // head_dim
constexpr int kRow = 128;        // LDS bytes per staged query row
constexpr int kLdsMax = 160 * 1024;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMinExp = -100;
    // lower bound of the dS exponent (keeps 2^(15-E) finite)


// ZK key levels per workgroup (one wave each); NBUF = 2: double-buffered query
// tiles, one workgroup per CU; NBUF = 1: single buffer, small enough for two
// workgroups per CU, which then hide each other's copies and barriers.
template <int KZ, int KY, int KX, int ZK, int NBUF, bool LO>
struct KvCfg {
  static constexpr int kThreads = 64 * ZK;
  static constexpr int MQY = 4 + 3 * (KY / 2), MQX = 4 + 3 * (KX / 2);  // largest query box
  static constexpr int MQ = (MQY * MQX + 31) / 32 * 32;                  // rows, whole 32-query steps
  static constexpr int TBYTES = MQ * kRow;
  static constexpr int SLOTS = MQ * (kRow / 16);
  static constexpr int IT = (SLOTS + kThreads - 1) / kThreads;           // copy slots per thread
  static constexpr int IS = (MQ + kThreads - 1) / kThreads;              // LSE / D entries per thread
  static constexpr int LDS = NBUF * ((LO ? 3 : 2) * TBYTES + 2 * MQ * 4) + MQ * 2;
  static constexpr int WG_PER_CU = NBUF == 1 && 2 * LDS <= kLdsMax ? 2 : 1;
  static_assert(LDS * WG_PER_CU <= kLdsMax, "query tiles exceed LDS");
};

struct KvArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;      // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  const uint16_t* dout;
  const float* lse;      // natural log
  const float* dvec;     // D = rowsum(dO * O)
  uint16_t* dk;
  uint16_t* dv;
  int heads, Z, H, W;
  int n_zb, n_yb, n_xb;
  float scale, kscale;   // scale, scale * log2(e)
  int qk_norm;           // QK RMSNorm of the stationary keys and the staged queries
  float eps;
  const uint16_t* dout_lo;  // low term of a two-term dO (with LO)
};

// queries whose (border-clamped) window holds position j of an axis of extent L
__host__ __device__ __forceinline__ int inv_lo(int j, int k) { return j < k ? 0 : j - (k >> 1); }
__host__ __device__ __forceinline__ int inv_hi(int j, int L, int k) { return j >= L - k ? L - 1 : j + (k >> 1); }

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

// A tile plus a lane offset, the offset passed through an empty asm: the
// compiler keeps the sum in one register per tile and lane pattern and folds
// every constant (step, chunk, column) into the read's immediate offset.  The
// pointer still derives from the tile, so the compiler can tell these reads from
// the copies into the other buffer and does not wait for those copies.
__device__ __forceinline__ const char* lds_base(const char* p, uint32_t off) {
  asm volatile("" : "+v"(off));
  return p + off;
}
__device__ __forceinline__ uint4 ldl16(const char* p) { return ld16(p); }
__device__ __forceinline__ float4 ldlf4(const char* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ uint2 trl(const char* p) { return __builtin_bit_cast(uint2, tr_read(p)); }

__device__ __forceinline__ int rswz(int u) { return (((u >> 1) & 3) << 1) | ((u >> 3) & 1); }

template <int KZ, int KY, int KX, int ZK, int NBUF, bool LO, bool NORM>
__global__ void __launch_bounds__(64 * ZK, (KvCfg<KZ, KY, KX, ZK, NBUF, LO>::WG_PER_CU)) na3d_mfma_kv_kernel(KvArgs a) {
  using C = KvCfg<KZ, KY, KX, ZK, NBUF, LO>;
  constexpr int kThreads = C::kThreads;
  constexpr int T2 = NBUF == 2 ? C::TBYTES : 16, M2 = NBUF == 2 ? C::MQ : 4;
  constexpr int TL0 = LO ? C::TBYTES : 16, TL1 = LO && NBUF == 2 ? C::TBYTES : 16;
  __shared__ __attribute__((aligned(16))) char tQ0[C::TBYTES];
  __shared__ __attribute__((aligned(16))) char tG0[C::TBYTES];
  __shared__ __attribute__((aligned(16))) char tQ1[T2];
  __shared__ __attribute__((aligned(16))) char tG1[T2];
  __shared__ __attribute__((aligned(16))) char tL0[TL0];  // low term of dO (LO)
  __shared__ __attribute__((aligned(16))) char tL1[TL1];
  __shared__ __attribute__((aligned(16))) float sL0[C::MQ];
  __shared__ __attribute__((aligned(16))) float sD0[C::MQ];
  __shared__ __attribute__((aligned(16))) float sL1[M2];
  __shared__ __attribute__((aligned(16))) float sD1[M2];
  __shared__ __attribute__((aligned(16))) unsigned short smask[C::MQ];

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
  const int y0 = 4 * yb, x0 = 4 * xb, z0 = ZK * zb;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;

  // ---- the query box of the block (the same on every level) ------------------
  const int qy0 = inv_lo(y0, KY), qy1 = inv_hi(min(y0 + 3, H - 1), H, KY);
  const int qx0 = inv_lo(x0, KX), qx1 = inv_hi(min(x0 + 3, W - 1), W, KX);
  const int nqx = qx1 - qx0 + 1;
  const int nq = (qy1 - qy0 + 1) * nqx;
  const int npairs = (nq + 31) >> 5;
  const int64_t HW = (int64_t)H * W;
  const int64_t bh_base = (int64_t)bh * Z * HW;  // token index of (b, h, 0, 0, 0)
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * 16 : nullptr;

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
      sL0[u] = 0.f;
      sD0[u] = 0.f;
      if constexpr (NBUF == 2) {
        sL1[u] = 0.f;
        sD1[u] = 0.f;
      }
    }
    smask[u] = (unsigned short)bits;
  }
  // rows past the box up to the last 32-query step: zero in all four tiles
  for (int i = nq * 8 + tid; i < npairs * 256; i += kThreads) {
    const uint4 z = make_uint4(0u, 0u, 0u, 0u);
    st16(tQ0 + i * 16, z);
    st16(tG0 + i * 16, z);
    if constexpr (LO) st16(tL0 + i * 16, z);
    if constexpr (NBUF == 2) {
      st16(tQ1 + i * 16, z);
      st16(tG1 + i * 16, z);
      if constexpr (LO) st16(tL1 + i * 16, z);
    }
  }

  __syncthreads();  // the mask table is read across lanes below
  // this lane's window bits: bit 4c + i of mb is row 16c + 4g + i of the box (the
  // rows of the X accumulator this lane holds in chunk c) seen by key qn
  static_assert(C::MQ <= 256, "window bits of a lane fit two words");
  uint32_t mb[2] = {0u, 0u};
#pragma unroll
  for (int c = 0; c < C::MQ / 16; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      mb[(4 * c + i) >> 5] |= ((smask[16 * c + 4 * (lane >> 4) + i] >> (lane & 15)) & 1u) << ((4 * c + i) & 31);

  // ---- direct-to-LDS copy map (registers): slot s = it*512 + tid ---------------
  // row u = s / 8 holds box query u; slot column s % 8 holds data column
  // (s % 8) ^ sigma(u).  Q and dO share the map; goff = -1 past the box.
  int goff[C::IT];
  uint4 ph[C::IT];
#pragma unroll
  for (int it = 0; it < C::IT; ++it) {
    const int s = it * kThreads + tid, u = s >> 3, dc = (s & 7) ^ rswz(u);
    goff[it] = -1;
    ph[it] = make_uint4(0u, 0u, 0u, 0u);
    if (s < C::SLOTS && u < nq) {
      const int qy = qy0 + u / nqx, qx = qx0 + u % nqx;
      goff[it] = (qy * W + qx) * kD + dc * 8;
      if (csb) {  // phases of pairs 4dc .. 4dc+3 as float16 (cos, sin)
        const float4* pp = csb + ((int64_t)qy * W + qx) * 16 + 2 * dc;
        const float4 p0 = pp[0], p1 = pp[1];
        ph[it] = make_uint4(pack2h(p0.x, p0.y), pack2h(p0.z, p0.w), pack2h(p1.x, p1.y), pack2h(p1.z, p1.w));
      }
    }
  }
  // LSE / D entries of this thread: token offset inside a level, or -1
  int soff[C::IS];
  float pl[C::IS], pd[C::IS];
#pragma unroll
  for (int is = 0; is < C::IS; ++is) {
    const int u = is * kThreads + tid;
    soff[is] = u < nq ? (qy0 + u / nqx) * W + qx0 + u % nqx : -1;
    pl[is] = 0.f;
    pd[is] = 0.f;
  }

  auto issue = [&](int p, char* tq, char* tg, char* tl) {
    const int64_t lev = bh_base + (int64_t)p * HW;
    const uint16_t* qp = a.q + lev * kD;
    const uint16_t* gp = a.dout + lev * kD;
    const uint16_t* lp = LO ? a.dout_lo + lev * kD : nullptr;
#pragma unroll
    for (int it = 0; it < C::IT; ++it) {
      if (goff[it] < 0) continue;
      copy16_to_lds(qp + goff[it], tq + (it * kThreads + wave * 64) * 16);
      copy16_to_lds(gp + goff[it], tg + (it * kThreads + wave * 64) * 16);
      if constexpr (LO) copy16_to_lds(lp + goff[it], tl + (it * kThreads + wave * 64) * 16);
    }
#pragma unroll
    for (int is = 0; is < C::IS; ++is) {
      if (soff[is] < 0) continue;
      pl[is] = a.lse[lev + soff[is]];
      pd[is] = a.dvec[lev + soff[is]];
    }
  };
  // wait for this thread's copies and loads, rotate its own Q slots in place
  // (bf16 -> float16; with QK RMSNorm the 8 slots of a row, 8 consecutive
  // lanes all in or all past the box, add their sums of squares for the row's
  // factor), store its LSE / D entries
  auto finish = [&](char* tq, float* sl, float* sd) {
    __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
    for (int it = 0; it < C::IT; ++it) {
      if (goff[it] < 0) continue;
      char* ad = tq + (it * kThreads + tid) * 16;
      const uint4 x = ld16(ad);
      const float mul = NORM ? __builtin_amdgcn_rsqf(sum_over_8_lanes(sumsq8(x, 0.f)) * (1.f / kD) + a.eps) : 1.f;
      st16(ad, csb ? rotate8h_pk(x, ph[it], mul) : scale8h(x, mul));
    }
#pragma unroll
    for (int is = 0; is < C::IS; ++is) {
      if (soff[is] < 0) continue;
      const int u = is * kThreads + tid;
      sl[u] = -(pl[is] * kLog2e);  // the seed of X: -LSE in log2 units
      sd[u] = -pd[is];
    }
  };

  // ---- this wave's keys: K~ and V as B operands (col = key qn, k = d) ----------
  const int ky_raw = y0 + (qn >> 2), kx_raw = x0 + (qn & 3);
  const int ky = min(ky_raw, H - 1), kx = min(kx_raw, W - 1);
  const int kz = z0 + wave;
  const bool wave_on = kz < Z;
  const int64_t ktok = bh_base + (int64_t)min(kz, Z - 1) * HW + (int64_t)ky * W + kx;
  const float4* csk = csb ? csb + ((int64_t)ky * W + kx) * 16 : nullptr;
  f16x8 kf[2];
  bf16x8 vf[2];
  float rk = 1.f;  // QK RMSNorm factor of this lane's key
  {
    const uint4* src = reinterpret_cast<const uint4*>(a.k + ktok * kD);
    const uint4 x0v = src[g], x1v = src[4 + g];
    if constexpr (NORM)  // the 4 lanes of a key row hold its 64 values
      rk = __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(x1v, sumsq8(x0v, 0.f))) * (1.f / kD) + a.eps);
    uint4 r0, r1;
    if (csk) {
      r0 = rotate8h(x0v, csk[2 * g], csk[2 * g + 1], a.kscale * rk);
      r1 = rotate8h(x1v, csk[8 + 2 * g], csk[8 + 2 * g + 1], a.kscale * rk);
    } else {
      r0 = scale8h(x0v, a.kscale * rk);
      r1 = scale8h(x1v, a.kscale * rk);
    }
    kf[0] = __builtin_bit_cast(f16x8, r0);
    kf[1] = __builtin_bit_cast(f16x8, r1);
    const uint4* vs = reinterpret_cast<const uint4*>(a.v + ktok * kD);
    vf[0] = __builtin_bit_cast(bf16x8, vs[g]);
    vf[1] = __builtin_bit_cast(bf16x8, vs[4 + g]);
  }
  f32x4 accK[4], accV[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    accK[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    accV[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  int ex = kMinExp;

  // lane-constant parts of the read addresses
  // A rows: chunk c, row 16c + qn, column g (xor 64 bytes: g + 4)
  const uint32_t aoff = qn * kRow + ((g ^ rswz(qn)) << 4);
  // transpose reads: row 32 st + 4g + qn/4 (+16 for the second chunk), the
  // 8 bytes holding elements 4 (qn % 4) .. +3 of each 16-wide d block (xor 32 t)
  const int trow = 4 * g + (qn >> 2);
  const uint32_t toff = trow * kRow + ((((qn >> 1) & 1) ^ rswz(trow)) << 4) + 8 * (qn & 1);

  auto compute = [&](const char* tq, const char* tg, const char* tl, const float* sl, const float* sd) {
    // lane bases of this level's tiles: every read below is one of them plus an
    // immediate offset (steps fully unrolled up to the largest box)
    const char* const aq0 = lds_base(tq, aoff);
    const char* const aq1 = lds_base(tq, aoff ^ 64u);
    const char* const ag0 = lds_base(tg, aoff);
    const char* const ag1 = lds_base(tg, aoff ^ 64u);
    const char* const al0 = LO ? lds_base(tl, aoff) : nullptr;
    const char* const al1 = LO ? lds_base(tl, aoff ^ 64u) : nullptr;
    const char* bq[4];
    const char* bg[4];
    const char* bl[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      bq[t] = lds_base(tq, toff ^ (32u * t));
      bg[t] = lds_base(tg, toff ^ (32u * t));
      bl[t] = LO ? lds_base(tl, toff ^ (32u * t)) : nullptr;
    }
    // the window bits pass through an empty asm at every level, so the
    // compiler derives the seeds' select masks step by step instead of hoisting
    // all 64 of them into registers
    uint32_t mw[2] = {mb[0], mb[1]};
    asm volatile("" : "+v"(mw[0]), "+v"(mw[1]));
    const char* const sl4 = lds_base(reinterpret_cast<const char*>(sl), 16 * g);
    const char* const sd4 = lds_base(reinterpret_cast<const char*>(sd), 16 * g);
    // A operands and seeds of one step (two 16-query chunks).  (Reading the next
    // step's while this one computes needs more registers than two waves per
    // SIMD leave; measured, the transpose reads issued early pay more.)
    struct StepIn {
      f16x8 q0[2], q1[2];
      bf16x8 g0[2], g1[2];
      float4 l4[2], d4[2];
    };
    auto load_in = [&](auto Si, StepIn& f) {
      constexpr int st = decltype(Si)::v;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = 2 * st + h;
        f.q0[h] = __builtin_bit_cast(f16x8, ldl16(aq0 + c * (16 * kRow)));
        f.q1[h] = __builtin_bit_cast(f16x8, ldl16(aq1 + c * (16 * kRow)));
        f.g0[h] = __builtin_bit_cast(bf16x8, ldl16(ag0 + c * (16 * kRow)));
        f.g1[h] = __builtin_bit_cast(bf16x8, ldl16(ag1 + c * (16 * kRow)));
        f.l4[h] = ldlf4(sl4 + 64 * c);
        f.d4[h] = ldlf4(sd4 + 64 * c);
      }
    };
    static_for<C::MQ / 32>([&](auto Si) {
      constexpr int st = decltype(Si)::v;
      if (st >= npairs) return;  // wave-uniform
      StepIn cur;
      load_in(Si, cur);
      constexpr int o = st * (32 * kRow);
      // transpose reads of this step, issued before its MFMAs and softmax so
      // that their latency hides there
      uint2 gtr[4][2], qtr[4][2];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        gtr[t][0] = trl(bg[t] + o);
        gtr[t][1] = trl(bg[t] + o + 16 * kRow);
        qtr[t][0] = trl(bq[t] + o);
        qtr[t][1] = trl(bq[t] + o + 16 * kRow);
      }
      f32x4 x[2], y[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = 2 * st + h;
        // seeds for rows 16c + 4g + i (the D layout of X and Y): -LSE where the
        // row's query sees this lane's key, else -inf (bit select by the
        // sign-extended window bit)
        const float lv[4] = {cur.l4[h].x, cur.l4[h].y, cur.l4[h].z, cur.l4[h].w};
        f32x4 xs;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int bit = 4 * c + i;
          const uint32_t sel = (uint32_t)__builtin_amdgcn_sbfe((int)mw[bit >> 5], bit & 31, 1);
          xs[i] = __uint_as_float((sel & __float_as_uint(lv[i])) | (~sel & 0xff800000u));
        }
        const f32x4 ys = {cur.d4[h].x, cur.d4[h].y, cur.d4[h].z, cur.d4[h].w};
        x[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(cur.q0[h], kf[0], xs, 0, 0, 0);
        x[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(cur.q1[h], kf[1], x[h], 0, 0, 0);
        y[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur.g0[h], vf[0], ys, 0, 0, 0);
        y[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur.g1[h], vf[1], y[h], 0, 0, 0);
        if constexpr (LO) {
          const bf16x8 l0 = __builtin_bit_cast(bf16x8, ldl16(al0 + c * (16 * kRow)));
          const bf16x8 l1 = __builtin_bit_cast(bf16x8, ldl16(al1 + c * (16 * kRow)));
          y[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(l0, vf[0], y[h], 0, 0, 0);
          y[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(l1, vf[1], y[h], 0, 0, 0);
        }
      }
      // exponent bound of |Y| for this lane's key (all four row groups)
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
        for (int t = 0; t < 4; ++t) accK[t] *= f;
        ex = en;
      }
      const float sc = __builtin_amdgcn_ldexpf(1.f, 15 - ex);
      // P for dV in two bf16 terms, P = hi + lo: bf16's rounding of P alone
      // would put the largest dV of a peaked softmax several percent of RMS(dV)
      // off; the second term leaves ~2^-17 P.  With the gate's two-term dA the
      // rows of dA differ in magnitude anyway and dV is held to the elementwise
      // bound of P's bf16 rounding (2^-8 sum P |dA|): one term there.
      uint32_t pb[2][2], pr[2][2], db[2][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float p0 = __builtin_amdgcn_exp2f(x[h][0]), p1 = __builtin_amdgcn_exp2f(x[h][1]);
        const float p2 = __builtin_amdgcn_exp2f(x[h][2]), p3 = __builtin_amdgcn_exp2f(x[h][3]);
        pb[h][0] = pack2(p0, p1);
        pb[h][1] = pack2(p2, p3);
        if constexpr (!LO) {
          pr[h][0] = pack2(p0 - lo_bf16(pb[h][0]), p1 - hi_bf16(pb[h][0]));
          pr[h][1] = pack2(p2 - lo_bf16(pb[h][1]), p3 - hi_bf16(pb[h][1]));
        }
        db[h][0] = pack2h_rne(p0 * sc * y[h][0], p1 * sc * y[h][1]);
        db[h][1] = pack2h_rne(p2 * sc * y[h][2], p3 * sc * y[h][3]);
      }
      const bf16x8 pf = __builtin_bit_cast(bf16x8, make_uint4(pb[0][0], pb[0][1], pb[1][0], pb[1][1]));
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(db[0][0], db[0][1], db[1][0], db[1][1]));
      bf16x8 gt[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        gt[t] = __builtin_bit_cast(bf16x8, make_uint4(gtr[t][0].x, gtr[t][0].y, gtr[t][1].x, gtr[t][1].y));
        accV[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gt[t], pf, accV[t], 0, 0, 0);
        if constexpr (LO) {
          const uint2 l_lo = trl(bl[t] + o);
          const uint2 l_hi = trl(bl[t] + o + 16 * kRow);
          const bf16x8 lt = __builtin_bit_cast(bf16x8, make_uint4(l_lo.x, l_lo.y, l_hi.x, l_hi.y));
          accV[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lt, pf, accV[t], 0, 0, 0);
        }
        const f16x8 qt = __builtin_bit_cast(f16x8, make_uint4(qtr[t][0].x, qtr[t][0].y, qtr[t][1].x, qtr[t][1].y));
        accK[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qt, df, accK[t], 0, 0, 0);
      }
      if constexpr (!LO) {
        const bf16x8 prf = __builtin_bit_cast(bf16x8, make_uint4(pr[0][0], pr[0][1], pr[1][0], pr[1][1]));
#pragma unroll
        for (int t = 0; t < 4; ++t) accV[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gt[t], prf, accV[t], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the next step's loads out of this one's registers
    });
  };
  // does query level p see this wave's key level?
  auto active = [&](int p) {
    const int zs = win_start(p, Z, KZ);
    return wave_on && kz >= zs && kz < zs + KZ;
  };

  // ---- query levels that see the block's key levels, double-buffered ---------
  // Level p+1 is copied while level p is computed; then each thread waits for
  // its own copies, finishes its own slots, and one barrier publishes the level.
  // The barrier also retires every read of the tiles the next copy overwrites.
  const int zk_last = min(z0 + ZK, Z) - 1;
  const int p_lo = inv_lo(z0, KZ), p_hi = inv_hi(zk_last, Z, KZ);
  if constexpr (NBUF == 1) {
    // one buffer: copy, publish, compute, and a barrier before the next copy
    for (int p = p_lo; p <= p_hi; ++p) {
      issue(p, tQ0, tG0, tL0);
      finish(tQ0, sL0, sD0);
      __syncthreads();
      if (active(p)) compute(tQ0, tG0, tL0, sL0, sD0);
      __syncthreads();
    }
  } else {
  issue(p_lo, tQ0, tG0, tL0);
  finish(tQ0, sL0, sD0);
  __syncthreads();
  for (int p = p_lo; p <= p_hi; p += 2) {
    const bool more1 = p + 1 <= p_hi;
    if (more1) issue(p + 1, tQ1, tG1, tL1);
    if (active(p)) compute(tQ0, tG0, tL0, sL0, sD0);
    if (more1) {
      finish(tQ1, sL1, sD1);
      __syncthreads();
      const bool more2 = p + 2 <= p_hi;
      if (more2) issue(p + 2, tQ0, tG0, tL0);
      if (active(p + 1)) compute(tQ1, tG1, tL1, sL1, sD1);
      if (more2) {
        finish(tQ0, sL0, sD0);
        __syncthreads();
      }
    }
  }
  }

  // ---- store: dV, and dK = R^T (scale 2^(E-15) dK~); lane holds d = 16t + 4g + i ----
  // With QK RMSNorm that is the gradient of k^ = r k, carried back through the
  // norm: dk = r (dk^ - k^ mean(dk^ k^)), k^ from the raw row in float32.
  const float f = a.scale * __builtin_amdgcn_ldexpf(1.f, ex - 15);
  f32x4 xk[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
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
    f32x4 kh[4];
    float c = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint2 w = kr[4 * t + g];
      kh[t] = f32x4{lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y)} * rk;
#pragma unroll
      for (int i = 0; i < 4; ++i) c = fmaf(xk[t][i], kh[t][i], c);
    }
    c = sum_over_rows(c) * (1.f / kD);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) xk[t][i] = rk * fmaf(-kh[t][i], c, xk[t][i]);
  }
  if (!wave_on || ky_raw >= H || kx_raw >= W) return;
  uint2* dkd = reinterpret_cast<uint2*>(a.dk + ktok * kD);
  uint2* dvd = reinterpret_cast<uint2*>(a.dv + ktok * kD);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
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

template <int KZ, int KY, int KX, int ZK, int NBUF, bool LO>
bool launch_kv(const strata_na3d_desc& d, const KvArgs& a0, hipStream_t s) {
  using C = KvCfg<KZ, KY, KX, ZK, NBUF, LO>;
  if (max_box(d.H, KY) > C::MQY || max_box(d.W, KX) > C::MQX) return false;
  KvArgs a = a0;
  a.n_zb = (d.Z + ZK - 1) / ZK;
  a.n_yb = (d.H + 3) / 4;
  a.n_xb = (d.W + 3) / 4;
  const int64_t blocks = (int64_t)d.B * d.heads * a.n_zb * a.n_yb * a.n_xb;
  if (blocks >= (int64_t)1 << 31) return false;
  if (a.qk_norm)
    hipLaunchKernelGGL((na3d_mfma_kv_kernel<KZ, KY, KX, ZK, NBUF, LO, true>), dim3((unsigned)blocks),
                       dim3(C::kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((na3d_mfma_kv_kernel<KZ, KY, KX, ZK, NBUF, LO, false>), dim3((unsigned)blocks),
                       dim3(C::kThreads), 0, s, a);
  return true;
}

}  // namespace

bool launch_na3d_bwd_dkdv_mfma(const strata_na3d_desc& d, const BwdOpts& o, const void* q,
                               const void* k, const void* v, const float* cs, const void* dout,
                               const float* lse, const float* dvec, void* dk, void* dv,
                               hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD) return false;
  if ((int64_t)d.H * d.W * kD >= (int64_t)1 << 31) return false;
  KvArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse = lse;
  a.dvec = dvec;
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.heads = d.heads;
  a.Z = d.Z;
  a.H = d.H;
  a.W = d.W;
  a.scale = d.scale;
  a.kscale = d.scale * kLog2e;
  a.qk_norm = o.qk_norm;
  a.eps = o.eps;
  a.dout_lo = static_cast<const uint16_t*>(o.dout_lo);
  // measured on MI355X at 16 tiles x 16 heads x 8x64x64: 3x7x7 is faster with two
  // single-buffered 4-level workgroups per CU (9.8 vs 11.6 ms for the whole
  // backward), 5x9x9 with one double-buffered 8-level workgroup (18.2 vs 18.4 ms)
  // A two-term dO adds a third staged tile: 5x9x9 then fits one single-buffered
  // workgroup per CU.
  const bool lo = o.dout_lo != nullptr;
  if (d.kz == 3 && d.ky == 7 && d.kx == 7)
    return lo ? launch_kv<3, 7, 7, 4, 1, true>(d, a, s) : launch_kv<3, 7, 7, 4, 1, false>(d, a, s);
  if (d.kz == 5 && d.ky == 9 && d.kx == 9)
    return lo ? launch_kv<5, 9, 9, 8, 1, true>(d, a, s) : launch_kv<5, 9, 9, 8, 2, false>(d, a, s);
  if (d.kz == 9 && d.ky == 9 && d.kx == 9)
    return lo ? launch_kv<9, 9, 9, 8, 1, true>(d, a, s) : launch_kv<9, 9, 9, 8, 2, false>(d, a, s);
  return false;
}

}  // namespace strata

// MFMA neighbourhood attention for gfx950, key-stationary dK/dV with every wave
// of a workgroup busy at every query level (bf16 in/out, head_dim 64; windows
// whose query boxes fit the staged grid below, e.g. the 9-wide (y, x) windows).
//
// Why: in the one-block kernel (na3d_mfma_kv.hip) a workgroup holds one 4 x 4
// block of keys on 8 levels, one wave per level; a query level sees KZ of them,
// so at 5 x 9 x 9 three of the eight waves idle at every level and one SIMD of
// four carries two busy waves while the others carry one.
//
// Work decomposition
//   workgroup : one (tile, head), two consecutive key levels and up to four
//               4 x 4 blocks of (y, x) key positions, 8 waves: wave w takes
//               level w / 4 of the pair and block w % 4 (by = (w / 2) % 2,
//               bx = w % 2).  Waves w and w + 4 share a SIMD and hold the same
//               block on the two levels, so every SIMD gets the same work.
//               (The run length is a template parameter; three levels, three
//               waves per SIMD, leave too few registers.)
//   blocks    : along each axis the 4-wide blocks are grouped in pairs: the two
//               edge blocks (0, n-1), then (1, 2), (3, 4), ... from the low
//               border and ..., (n-5, n-4), (n-3, n-2) from the high one, with
//               one interior block alone when their count is odd
//               (kvp_groups.h).  A block's queries (the union of the inverse
//               windows of its keys) span a run of "squares", 4-aligned runs of
//               4 positions; for 9-wide windows the runs of a pair cover at most
//               four squares per axis unless a single block already spans five
//               (axes of 17 to 20 positions; the host checks every group).
//   staging   : per query level the workgroup copies the 4 x 4 squares of its
//               group (16 rows each, 256 rows: Q rotated to float16 in place,
//               dO converted in place to float16 times 2^-sh, -LSE and -D 2^-sh
//               per row) with the direct-to-LDS load, double buffered.  sh comes
//               from the largest |dO| of the (batch, head), which the dQ pass
//               records, so the staged dO stays below 2^14.  Two more zero
//               squares sit past the grid for the padding chunk of an odd
//               square count.
//   wave      : the 16 keys of its block and level stay in registers (K~ times
//               scale log2(e) and V, both float16, as B operands, the dK~^T and
//               dV^T accumulators); it walks the squares of its own block's
//               query box, two squares (32 queries) per step:
//                 X = Q~ . K~^T (float16 MFMA seeded with -LSE or -inf outside the
//                 query's window), P = exp2(X); Y = dO . V^T - D (float16);
//                 dV^T += dO^T . P (float16: bf16's rounding of P alone would
//                 cost dV several percent of its RMS at peaked weights);
//                 dK~^T += Q~^T . dS (float16, dS = P Y with a per-key
//                 power-of-two scale 2^(15-E)); dK and dV are scaled back by
//                 2^sh when stored.
//   addresses : a wave's squares are fixed offsets from its first one once the
//               width of its box (in squares) is known, so the steps are
//               unrolled for width 3 (squares taken row by row, the last chunk
//               padded when the count is odd) and for widths 2 and 4 (two
//               squares of one row per step); every LDS read is a lane base
//               plus an immediate.
//   sweep     : one workgroup takes every run of key levels of its block group
//               in turn; the copies of the next (run, query level) go out while
//               the current one is computed, across the end of a run too, and
//               at a change of run the finished dK/dV are stored and the next
//               run's keys loaded in one batch.
#include "common.h"
#include "kernels.h"
#include "kvp_groups.h"
#include "mfma_util.h"

#include <algorithm>

namespace strata {
namespace {

using namespace mfma;
using namespace kvp;

constexpr int kD = 64;                   // head_dim
constexpr int kRow = 128;                // LDS bytes per staged query row
constexpr int kSq = 16 * kRow;           // one square: 16 rows
constexpr int kGrid = 16;                // staged squares (4 x 4)
constexpr int kNSq = kGrid + 2;          // plus two zero squares read by padding chunks
constexpr int kRows = kNSq * 16;
constexpr int kTB = kRows * kRow;        // bytes per staged tile
constexpr int kSlots = kGrid * 16 * 8;   // 16-byte copy slots of the grid
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMinExp = -100;            // lower bound of the dS exponent
static_assert(2 * (2 * kTB + 2 * kRows * 4) <= 160 * 1024, "staged tiles exceed LDS");

struct KvpArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float4* cs;      // [B, H, W, 16] float4 = two (cos, sin) pairs; nullptr: no rotation
  const uint16_t* dout;
  const float* lse;      // natural log
  const float* dvec;     // D = rowsum(dO * O)
  const int* emax;       // [B * heads] largest frexp exponent of |dO| (the dQ pass)
  uint16_t* dk;
  uint16_t* dv;
  int heads, Z, H, W;
  int ngy, ngx;          // block groups per axis
  float scale, kscale;   // scale, scale * log2(e)
  float eps;             // QK RMSNorm epsilon
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

// A tile plus a lane offset, the offset passed through an empty asm: the
// compiler keeps the sum in one register per tile and lane pattern and folds
// every constant (square, column) into the read's immediate offset, while the
// pointer still derives from the tile (so reads of one buffer are not made to
// wait for the copies into the other).
// bf16 x 8 -> float16 x 8 times a power of two `mul` that keeps them below 2^15
__device__ __forceinline__ uint4 f16_scaled8(uint4 x, float mul) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t r[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) r[t] = pack2h_rne(lo_bf16(w[t]) * mul, hi_bf16(w[t]) * mul);
  return make_uint4(r[0], r[1], r[2], r[3]);
}

__device__ __forceinline__ const char* lds_base(const char* p, uint32_t off) {
  asm volatile("" : "+v"(off));
  return p + off;
}
__device__ __forceinline__ uint4 ldl16(const char* p) { return ld16(p); }
__device__ __forceinline__ float4 ldlf4(const char* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ uint2 trl(const char* p) { return __builtin_bit_cast(uint2, tr_read(p)); }

// column swizzle of staged row u (bits 1..3 of u: the row inside its square)
__device__ __forceinline__ int rswz(int u) { return (((u >> 1) & 3) << 1) | ((u >> 3) & 1); }

__device__ __forceinline__ bool in_win(int q, int kpos, int L, int k) {
  const int s = win_start(q, L, k);
  return kpos >= s && kpos < s + k;
}

// chunk c of a wave's walk: the square (row a, column b) of its box
template <bool W3>
struct Walk {
  static constexpr int kChunks = W3 ? 12 : 16;
  static constexpr int row(int c) { return W3 ? c / 3 : c >> 2; }
  static constexpr int col(int c) { return W3 ? c % 3 : c & 3; }
  static constexpr int rel(int c) { return 4 * row(c) + col(c); }  // square offset from the box's first
};

// NL key levels per workgroup (4 NL waves): wave w takes level w / 4 of the
// run and block w % 4
template <int KZ, int KY, int KX, bool NORM, int NL>
__global__ void __launch_bounds__(256 * NL, 1) na3d_mfma_kvp_kernel(KvpArgs a) {
  constexpr int kThreads = 256 * NL;
  constexpr int kIT = (kSlots + kThreads - 1) / kThreads;  // copy slots per thread
  static_assert(kIT * kThreads <= kNSq * 128, "copy slots stay inside the staged tile");
  __shared__ __attribute__((aligned(16))) char tQ0[kTB];
  __shared__ __attribute__((aligned(16))) char tG0[kTB];
  __shared__ __attribute__((aligned(16))) char tQ1[kTB];
  __shared__ __attribute__((aligned(16))) char tG1[kTB];
  __shared__ __attribute__((aligned(16))) float sL0[kRows];
  __shared__ __attribute__((aligned(16))) float sD0[kRows];
  __shared__ __attribute__((aligned(16))) float sL1[kRows];
  __shared__ __attribute__((aligned(16))) float sD1[kRows];

  // ---- block coordinates (XCD-aware: neighbouring groups share an L2) -------
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int gx = bid % a.ngx;
  const int gy = (bid / a.ngx) % a.ngy;
  const int bh = bid / (a.ngx * a.ngy);
  const int b = bh / a.heads;
  const int H = a.H, W = a.W, Z = a.Z;
  const int npairs = (Z + NL - 1) / NL;  // runs of NL key levels

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, qn = lane & 15;

  const AxisGroup ay = axis_group(gy, H, KY), ax = axis_group(gx, W, KX);
  const int64_t HW = (int64_t)H * W;
  const int64_t bh_base = (int64_t)bh * Z * HW;  // token index of (b, h, 0, 0, 0)
  const float4* csb = a.cs ? a.cs + (int64_t)b * HW * 16 : nullptr;
  // dO is staged in float16 times 2^-sh, sh from the largest |dO| of this
  // (batch, head) (below 2^eb), so the staged values stay below 2^14; D is
  // scaled alike and dK, dV are scaled back when stored
  const int eb = a.emax[bh];
  const int sh = eb == kEmaxEmpty ? 0 : min(max(eb - 14, -120), 120);
  const float dsc = __builtin_amdgcn_ldexpf(1.f, -sh), dun = __builtin_amdgcn_ldexpf(1.f, sh);

  // ---- direct-to-LDS copy map: slot s = it*kThreads + tid of the 4 x 4 grid ---
  // square sq = s / 128 (entry (sq / 4, sq % 4) of the axis lists), row
  // u = s / 8 (position (u % 16) / 4, u % 4 inside the square), slot column
  // s % 8 holds data column (s % 8) ^ rswz(u); goff = -1 where no query is.
  int goff[kIT];
  uint4 ph[kIT];
#pragma unroll
  for (int it = 0; it < kIT; ++it) {
    const int s = it * kThreads + tid, u = s >> 3, sq = s >> 7, rho = u & 15;  // sq > 15: past the grid
    const int dc = (s & 7) ^ rswz(u);
    const int ey = sq >> 2, ex = sq & 3;
    goff[it] = -1;
    ph[it] = make_uint4(0u, 0u, 0u, 0u);
    const int qy = 4 * sq_abs(ay, ey) + (rho >> 2), qx = 4 * sq_abs(ax, ex) + (rho & 3);
    if (s < kSlots && ey < ay.n && ex < ax.n && qy < H && qx < W) {
      goff[it] = (qy * W + qx) * kD + dc * 8;
      if (csb) {  // phases of pairs 4dc .. 4dc+3 as float16 (cos, sin)
        const float4* pp = csb + ((int64_t)qy * W + qx) * 16 + 2 * dc;
        const float4 p0 = pp[0], p1 = pp[1];
        ph[it] = make_uint4(pack2h(p0.x, p0.y), pack2h(p0.z, p0.w), pack2h(p1.x, p1.y), pack2h(p1.z, p1.w));
      }
    } else {  // never copied: zero in both buffers, once
      const uint4 z = make_uint4(0u, 0u, 0u, 0u);
      st16(tQ0 + s * 16, z);
      st16(tG0 + s * 16, z);
      st16(tQ1 + s * 16, z);
      st16(tG1 + s * 16, z);
    }
  }
  // the two padding squares
  for (int s = kSlots + tid; s < kNSq * 128; s += kThreads) {
    const uint4 z = make_uint4(0u, 0u, 0u, 0u);
    st16(tQ0 + s * 16, z);
    st16(tG0 + s * 16, z);
    st16(tQ1 + s * 16, z);
    st16(tG1 + s * 16, z);
  }
  // LSE / D entry of this thread (rows < 256): token offset inside a level, or -1
  int soff = -1;
  float pl = 0.f, pd = 0.f;
  {
    const int u = tid, sq = u >> 4, rho = u & 15, ey = sq >> 2, ex = sq & 3;
    const int qy = 4 * sq_abs(ay, ey) + (rho >> 2), qx = 4 * sq_abs(ax, ex) + (rho & 3);
    if (u < kGrid * 16 && ey < ay.n && ex < ax.n && qy < H && qx < W) soff = qy * W + qx;
  }
  for (int u = tid; u < kRows; u += kThreads)
    if (u >= kGrid * 16 || soff < 0) {
      sL0[u] = 0.f;
      sD0[u] = 0.f;
      sL1[u] = 0.f;
      sD1[u] = 0.f;
    }

  auto issue = [&](int p, char* tq, char* tg) __attribute__((always_inline)) {
    const int64_t lev = bh_base + (int64_t)p * HW;
    const uint16_t* qp = a.q + lev * kD;
    const uint16_t* gp = a.dout + lev * kD;
#pragma unroll
    for (int it = 0; it < kIT; ++it) {
      if (goff[it] < 0) continue;
      copy16_to_lds(qp + goff[it], tq + (it * kThreads + wave * 64) * 16);
      copy16_to_lds(gp + goff[it], tg + (it * kThreads + wave * 64) * 16);
    }
    if (soff >= 0) {
      pl = a.lse[lev + soff];
      pd = a.dvec[lev + soff];
    }
  };
  // wait for this thread's copies and loads, rotate its own Q slots in place
  // (bf16 -> float16; with QK RMSNorm the 8 slots of a row, 8 consecutive lanes
  // all valid or all not, add their sums of squares for the row's factor),
  // convert its own dO slots to scaled float16 in place, store its LSE / D entry
  auto finish = [&](char* tq, char* tg, float* sl, float* sd) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
    for (int it = 0; it < kIT; ++it) {
      if (goff[it] < 0) continue;
      char* ad = tq + (it * kThreads + tid) * 16;
      const uint4 x = ld16(ad);
      const float mul = NORM ? __builtin_amdgcn_rsqf(sum_over_8_lanes(sumsq8(x, 0.f)) * (1.f / kD) + a.eps) : 1.f;
      st16(ad, csb ? rotate8h_pk(x, ph[it], mul) : scale8h(x, mul));
      char* ag = tg + (it * kThreads + tid) * 16;
      st16(ag, f16_scaled8(ld16(ag), dsc));
    }
    if (soff >= 0) {
      sl[tid] = -(pl * kLog2e);  // the seed of X: -LSE in log2 units
      sd[tid] = -pd * dsc;
    }
  };

  // ---- this wave's block, level and box ---------------------------------------
  const int lev_w = wave >> 2, by = (wave >> 1) & 1, bx = wave & 1;
  const bool blk_on = by < ay.nblk && bx < ax.nblk;
  const int jy = by ? ay.blk1 : ay.blk0, jx = bx ? ax.blk1 : ax.blk0;
  const int sy0 = by ? ay.run1 : ay.run0, nsy = by ? ay.len1 : ay.len0;
  const int sx0 = bx ? ax.run1 : ax.run0, nsx = bx ? ax.len1 : ax.len0;
  const bool w3 = nsx == 3;
  const int ky_raw = 4 * jy + (qn >> 2), kx_raw = 4 * jx + (qn & 3);
  const int ky = max(0, min(ky_raw, H - 1)), kx = max(0, min(kx_raw, W - 1));

  // window bits: bit 4c + i of mb is row 4g + i of chunk c of the walk (the
  // rows of the X accumulator this lane holds) seen by key qn; rows outside the
  // box (and the padding chunk) stay clear
  uint32_t mb[2] = {0u, 0u};
  {
    bool yok[4];
    uint32_t xok[4];  // bit i: column i of the square seen by the key
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int qy = 4 * sq_abs(ay, sy0 + r) + g;
      yok[r] = r < nsy && qy < H && in_win(qy, ky, H, KY);
      uint32_t m = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int qx = 4 * sq_abs(ax, sx0 + r) + i;
        if (r < nsx && qx < W && in_win(qx, kx, W, KX)) m |= 1u << i;
      }
      xok[r] = m;
    }
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const uint32_t b4 = w3 ? (c < 12 && yok[c / 3] ? xok[c % 3] : 0u) : (yok[c >> 2] ? xok[c & 3] : 0u);
      mb[c >> 3] |= b4 << (4 * (c & 7));
    }
  }

  // ---- this wave's keys (of the current pair): K~ and V as B operands (col = key
  // qn, k = d), the dK~^T and dV^T accumulators and the exponent of dS ----------
  const float4* csk = csb ? csb + ((int64_t)ky * W + kx) * 16 : nullptr;
  const int64_t kpos = bh_base + (int64_t)ky * W + kx;  // token of the key on level 0
  f16x8 kf[2];
  f16x8 vf[2];  // V in float16 (round toward zero: saturates at 65504)
  float rk = 1.f;  // QK RMSNorm factor of this lane's key
  f32x4 accK[4], accV[4];
  int ex = kMinExp;
  // What a change of pair reads from global memory, loaded in one batch (one
  // wait): this lane's phases for rotating dK back and for rotating the next
  // pair's K, the stored key's raw row (the norm's Jacobian), the next K and V.
  struct PairIo {
    float4 ps[4];        // phases of pairs 8t+2g, 8t+2g+1 (the store)
    float4 pk[4];        // phases of pairs 4g..4g+3 and 16+4g..16+4g+3 (the load)
    uint2 kr[4];         // raw row of the stored key
    uint4 xk[2], xv[2];  // the next pair's K and V rows
  };
  auto key_tok = [&](int j) { return kpos + (int64_t)min(NL * j + lev_w, Z - 1) * HW; };
  auto load_io = [&](PairIo& io, int j, int jn, bool more) __attribute__((always_inline)) {
    if (csk) {
#pragma unroll
      for (int t = 0; t < 4; ++t) io.ps[t] = csk[4 * t + g];
      io.pk[0] = csk[2 * g];
      io.pk[1] = csk[2 * g + 1];
      io.pk[2] = csk[8 + 2 * g];
      io.pk[3] = csk[8 + 2 * g + 1];
    }
    if (NORM && j >= 0) {
      const uint2* kr = reinterpret_cast<const uint2*>(a.k + key_tok(j) * kD);
#pragma unroll
      for (int t = 0; t < 4; ++t) io.kr[t] = kr[4 * t + g];
    }
    if (more) {
      const uint4* src = reinterpret_cast<const uint4*>(a.k + key_tok(jn) * kD);
      const uint4* vs = reinterpret_cast<const uint4*>(a.v + key_tok(jn) * kD);
      io.xk[0] = src[g];
      io.xk[1] = src[4 + g];
      io.xv[0] = vs[g];
      io.xv[1] = vs[4 + g];
    }
  };
  auto begin_pair = [&](const PairIo& io) __attribute__((always_inline)) {
    if constexpr (NORM)  // the 4 lanes of a key row hold its 64 values
      rk = __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(io.xk[1], sumsq8(io.xk[0], 0.f))) * (1.f / kD) + a.eps);
    uint4 r0, r1;
    if (csk) {
      r0 = rotate8h(io.xk[0], io.pk[0], io.pk[1], a.kscale * rk);
      r1 = rotate8h(io.xk[1], io.pk[2], io.pk[3], a.kscale * rk);
    } else {
      r0 = scale8h(io.xk[0], a.kscale * rk);
      r1 = scale8h(io.xk[1], a.kscale * rk);
    }
    kf[0] = __builtin_bit_cast(f16x8, r0);
    kf[1] = __builtin_bit_cast(f16x8, r1);
    vf[0] = __builtin_bit_cast(f16x8, bf16x8_to_f16x8(io.xv[0]));
    vf[1] = __builtin_bit_cast(f16x8, bf16x8_to_f16x8(io.xv[1]));
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      accK[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      accV[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    ex = kMinExp;
  };

  // lane-constant parts of the read addresses, from the box's first square
  const uint32_t wb = (uint32_t)(4 * sy0 + sx0);
  // A rows: row qn of a square, column g (xor 64 bytes: g + 4)
  const uint32_t aoff = wb * kSq + qn * kRow + ((g ^ rswz(qn)) << 4);
  // transpose reads: row 4g + qn/4 of a square, the 8 bytes holding elements
  // 4 (qn % 4) .. +3 of each 16-wide d block (xor 32 t)
  const int trow = 4 * g + (qn >> 2);
  const uint32_t toff = wb * kSq + trow * kRow + ((((qn >> 1) & 1) ^ rswz(trow)) << 4) + 8 * (qn & 1);

  auto compute = [&](auto W3c, const char* tq, const char* tg, const float* sl, const float* sd)
                     __attribute__((always_inline)) {
    constexpr bool W3 = decltype(W3c)::v != 0;
    using Wk = Walk<W3>;
    const char* const aq0 = lds_base(tq, aoff);
    const char* const aq1 = lds_base(tq, aoff ^ 64u);
    const char* const ag0 = lds_base(tg, aoff);
    const char* const ag1 = lds_base(tg, aoff ^ 64u);
    const char* bq[4];
    const char* bg[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      bq[t] = lds_base(tq, toff ^ (32u * t));
      bg[t] = lds_base(tg, toff ^ (32u * t));
    }
    // the window bits pass through an empty asm at every level, so the
    // compiler derives the seeds' select masks step by step instead of hoisting
    // all of them into registers
    uint32_t mw[2] = {mb[0], mb[1]};
    asm volatile("" : "+v"(mw[0]), "+v"(mw[1]));
    const char* const sl4 = lds_base(reinterpret_cast<const char*>(sl), wb * 64 + 16 * g);
    const char* const sd4 = lds_base(reinterpret_cast<const char*>(sd), wb * 64 + 16 * g);
    static_for<Wk::kChunks / 2>([&](auto Si) {
      constexpr int st = decltype(Si)::v;
      constexpr int c0 = 2 * st, c1 = 2 * st + 1;  // the step's two chunks
      // wave-uniform: width 3 walks 3 nsy chunks (the last padded when odd);
      // widths 2 and 4 take two squares of one row per step
      if constexpr (W3) {
        if (c0 >= 3 * nsy) return;
      } else {
        if (Wk::row(c0) >= nsy || Wk::col(c0) >= nsx) return;
      }
      constexpr uint32_t o[2] = {Wk::rel(c0) * kSq, Wk::rel(c1) * kSq};
      constexpr uint32_t ol[2] = {Wk::rel(c0) * 64u, Wk::rel(c1) * 64u};
      f16x8 q0[2], q1[2];
      f16x8 g0[2], g1[2];
      float4 l4[2], d4[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        q0[h] = __builtin_bit_cast(f16x8, ldl16(aq0 + o[h]));
        q1[h] = __builtin_bit_cast(f16x8, ldl16(aq1 + o[h]));
        g0[h] = __builtin_bit_cast(f16x8, ldl16(ag0 + o[h]));
        g1[h] = __builtin_bit_cast(f16x8, ldl16(ag1 + o[h]));
        l4[h] = ldlf4(sl4 + ol[h]);
        d4[h] = ldlf4(sd4 + ol[h]);
      }
      // transpose reads of this step, issued before its MFMAs and softmax so
      // that their latency hides there
      uint2 gtr[4][2], qtr[4][2];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        gtr[t][0] = trl(bg[t] + o[0]);
        gtr[t][1] = trl(bg[t] + o[1]);
        qtr[t][0] = trl(bq[t] + o[0]);
        qtr[t][1] = trl(bq[t] + o[1]);
      }
      f32x4 x[2], y[2];
      // the two waves of a SIMD alternate between MFMA blocks and softmax work:
      // raised priority while a wave issues its MFMAs keeps the matrix unit
      // fed (measured: training-tile backward 13.41 -> 13.29 ms; the same in the
      // dQ pass, three waves per SIMD, gained nothing)
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = 2 * st + h;
        // seeds for rows 4g + i of the chunk: -LSE where the row's query sees
        // this lane's key, else -inf (bit select by the sign-extended window bit)
        const float lv[4] = {l4[h].x, l4[h].y, l4[h].z, l4[h].w};
        f32x4 xs;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int bit = 4 * c + i;
          const uint32_t sel = (uint32_t)__builtin_amdgcn_sbfe((int)mw[bit >> 5], bit & 31, 1);
          xs[i] = __uint_as_float((sel & __float_as_uint(lv[i])) | (~sel & 0xff800000u));
        }
        const f32x4 ys = {d4[h].x, d4[h].y, d4[h].z, d4[h].w};
        x[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(q0[h], kf[0], xs, 0, 0, 0);
        x[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(q1[h], kf[1], x[h], 0, 0, 0);
        y[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(g0[h], vf[0], ys, 0, 0, 0);
        y[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(g1[h], vf[1], y[h], 0, 0, 0);
      }
      __builtin_amdgcn_s_setprio(0);
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
      // P for dV in float16 (bf16's rounding of P alone would put the largest
      // dV of a peaked softmax several percent of RMS(dV) off)
      uint32_t pb[2][2], db[2][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float p0 = __builtin_amdgcn_exp2f(x[h][0]), p1 = __builtin_amdgcn_exp2f(x[h][1]);
        const float p2 = __builtin_amdgcn_exp2f(x[h][2]), p3 = __builtin_amdgcn_exp2f(x[h][3]);
        pb[h][0] = pack2h_rne(p0, p1);
        pb[h][1] = pack2h_rne(p2, p3);
        db[h][0] = pack2h_rne(p0 * sc * y[h][0], p1 * sc * y[h][1]);
        db[h][1] = pack2h_rne(p2 * sc * y[h][2], p3 * sc * y[h][3]);
      }
      const f16x8 pf = __builtin_bit_cast(f16x8, make_uint4(pb[0][0], pb[0][1], pb[1][0], pb[1][1]));
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(db[0][0], db[0][1], db[1][0], db[1][1]));
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const f16x8 gt = __builtin_bit_cast(f16x8, make_uint4(gtr[t][0].x, gtr[t][0].y, gtr[t][1].x, gtr[t][1].y));
        accV[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(gt, pf, accV[t], 0, 0, 0);
        const f16x8 qt = __builtin_bit_cast(f16x8, make_uint4(qtr[t][0].x, qtr[t][0].y, qtr[t][1].x, qtr[t][1].y));
        accK[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qt, df, accK[t], 0, 0, 0);
      }
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);  // keep the next step's loads out of this one's registers
    });
  };
  auto compute_level = [&](const char* tq, const char* tg, const float* sl, const float* sd)
                           __attribute__((always_inline)) {
    if (w3)
      compute(IC<1>{}, tq, tg, sl, sd);
    else
      compute(IC<0>{}, tq, tg, sl, sd);
  };
  // does query level p see this wave's key level in pair j?
  auto active = [&](int j, int p) {
    const int kz = NL * j + lev_w, zs = win_start(p, Z, KZ);
    return blk_on && kz < Z && kz >= zs && kz < zs + KZ;
  };
  // store the pair's dV, and dK = R^T (scale 2^(E-15) dK~); lane holds d = 16t + 4g + i.
  // With QK RMSNorm that is the gradient of k^ = r k, carried back through the
  // norm: dk = r (dk^ - k^ mean(dk^ k^)), k^ from the raw row in float32.
  auto store_pair = [&](int j, const PairIo& io) __attribute__((always_inline)) {
    const int kz = NL * j + lev_w;
    const int64_t ktok = key_tok(j);
    const float f = a.scale * __builtin_amdgcn_ldexpf(1.f, ex - 15 + sh);
    f32x4 xk[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      xk[t] = accK[t] * f;
      if (csk) {
        const float4 p = io.ps[t];  // pairs 8t+2g and 8t+2g+1
        const float r0 = fmaf(xk[t][0], p.x, xk[t][1] * p.y), r1 = fmaf(xk[t][1], p.x, -xk[t][0] * p.y);
        const float r2 = fmaf(xk[t][2], p.z, xk[t][3] * p.w), r3 = fmaf(xk[t][3], p.z, -xk[t][2] * p.w);
        xk[t] = f32x4{r0, r1, r2, r3};
      }
    }
    if constexpr (NORM) {
      f32x4 kh[4];
      float c = 0.f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const uint2 w = io.kr[t];
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
    if (!blk_on || kz >= Z || ky_raw >= H || kx_raw >= W) return;
    uint2* dkd = reinterpret_cast<uint2*>(a.dk + ktok * kD);
    uint2* dvd = reinterpret_cast<uint2*>(a.dv + ktok * kD);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const f32x4 xv = accV[t] * dun;
      dvd[4 * t + g] = make_uint2(pack2(xv[0], xv[1]), pack2(xv[2], xv[3]));
      dkd[4 * t + g] = make_uint2(pack2(xk[t][0], xk[t][1]), pack2(xk[t][2], xk[t][3]));
    }
  };

  // ---- one sweep over the key-level pairs, double-buffered --------------------
  // Pair j (key levels 2j, 2j+1) is seen by the query levels [p_lo(j), p_hi(j)];
  // the workgroup walks them pair after pair, copying the next (pair, level)
  // while the current one is computed, so the copies keep running across the
  // end of a pair.  Each thread waits for its own copies, finishes its own
  // slots, and one barrier publishes the level; the barrier also retires every
  // read of the tiles the next copy overwrites.
  auto p_lo = [&](int j) { return inv_lo(NL * j, KZ); };
  auto p_hi = [&](int j) { return inv_hi(min(NL * j + NL - 1, Z - 1), Z, KZ); };
  // the (pair, level) after (j, p)
  auto next_of = [&](int j, int p, int& nj, int& np) {
    nj = j;
    np = p + 1;
    if (np > p_hi(j)) {
      nj = j + 1;
      np = nj < npairs ? p_lo(nj) : 0;
    }
  };
  auto change_pair = [&](int j, int nj, bool more) __attribute__((always_inline)) {
    PairIo io;
    load_io(io, j, nj, more);
    store_pair(j, io);
    if (more) begin_pair(io);
  };
  int cj = 0, cp = p_lo(0);
  {
    PairIo io;
    load_io(io, -1, 0, true);
    begin_pair(io);
  }
  issue(cp, tQ0, tG0);
  finish(tQ0, tG0, sL0, sD0);
  __syncthreads();
  for (;;) {
    int nj, np;
    next_of(cj, cp, nj, np);
    bool more = nj < npairs;
    if (more) issue(np, tQ1, tG1);
    if (active(cj, cp)) compute_level(tQ0, tG0, sL0, sD0);
    if (nj != cj) change_pair(cj, nj, more);
    if (!more) break;
    finish(tQ1, tG1, sL1, sD1);
    __syncthreads();
    cj = nj;
    cp = np;
    next_of(cj, cp, nj, np);
    more = nj < npairs;
    if (more) issue(np, tQ0, tG0);
    if (active(cj, cp)) compute_level(tQ1, tG1, sL1, sD1);
    if (nj != cj) change_pair(cj, nj, more);
    if (!more) break;
    finish(tQ0, tG0, sL0, sD0);
    __syncthreads();
    cj = nj;
    cp = np;
  }
}

template <int KZ, int KY, int KX, int NL>
bool launch_kvp(const strata_na3d_desc& d, const KvpArgs& a0, bool norm, hipStream_t s) {
  KvpArgs a = a0;
  a.ngy = n_groups(d.H);
  a.ngx = n_groups(d.W);
  const int64_t blocks = (int64_t)d.B * d.heads * a.ngy * a.ngx;
  if (norm)
    hipLaunchKernelGGL((na3d_mfma_kvp_kernel<KZ, KY, KX, true, NL>), dim3((unsigned)blocks), dim3(256 * NL), 0, s, a);
  else
    hipLaunchKernelGGL((na3d_mfma_kvp_kernel<KZ, KY, KX, false, NL>), dim3((unsigned)blocks), dim3(256 * NL), 0, s, a);
  return true;
}

}  // namespace

bool na3d_bwd_dkdv_kvp_takes(const strata_na3d_desc& d, const BwdOpts& o) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD || o.dout_lo != nullptr) return false;
  if ((int64_t)d.H * d.W * kD >= (int64_t)1 << 31) return false;
  if (!(d.ky == 9 && d.kx == 9 && (d.kz == 5 || d.kz == 9))) return false;
  if (!groups_fit(d.H, d.ky, false) || !groups_fit(d.W, d.kx, true)) return false;
  return (int64_t)d.B * d.heads * n_groups(d.H) * n_groups(d.W) < (int64_t)1 << 31;
}

bool launch_na3d_bwd_dkdv_kvp(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                              const void* v, const float* cs, const void* dout, const float* lse,
                              const float* dvec, const int* emax, void* dk, void* dv, hipStream_t s) {
  if (!emax || !na3d_bwd_dkdv_kvp_takes(d, o)) return false;
  KvpArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cs = reinterpret_cast<const float4*>(cs);
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse = lse;
  a.dvec = dvec;
  a.emax = emax;
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.heads = d.heads;
  a.Z = d.Z;
  a.H = d.H;
  a.W = d.W;
  a.scale = d.scale;
  a.kscale = d.scale * kLog2e;
  a.eps = o.eps;
  // two key levels per workgroup (two waves per SIMD, ~240 registers); three
  // levels (three waves per SIMD) leave 168 registers and spill 52 of them:
  // 8.94 against 7.67 ms for the training-tile dK/dV
  if (d.kz == 5 && d.ky == 9 && d.kx == 9) return launch_kvp<5, 9, 9, 2>(d, a, o.qk_norm, s);
  if (d.kz == 9 && d.ky == 9 && d.kx == 9) return launch_kvp<9, 9, 9, 2>(d, a, o.qk_norm, s);
  return false;
}

}  // namespace strata

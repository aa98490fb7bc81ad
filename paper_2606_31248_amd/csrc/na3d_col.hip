// Column-wise attention for gfx950 (Sec. 3.2: attention along the vertical
// within each column, alternating with the NA3D blocks), as neighbourhood
// attention with window (kz, 1, 1): a query at level i of column (y, x) sees the
// kz levels [s, s + kz) of its own column, s = clamp(i - (kz-1)/2, 0, Z - kz);
// kz = Z is the full column.  bf16 in/out, head_dim 64, Z <= 32.
//
// StereoRoPE: every token of a column has the same (y, x) and so the same
// rotation R; <R q, R k> = <q, k>, so the rotation cancels exactly and is not
// applied (the phase table is not read).
//
// Work decomposition: one wave per (tile, head, y, x) column, grid-strided.
// The column's levels are padded to 16 NB (NB = 1 or 2 blocks of 16):
//   S^T (keys x queries) = K . Q^T   float16 MFMA 16x16x32, two per (key block,
//                                    query block); Q is scaled by scale log2(e)
//                                    (times its QK RMSNorm factor) and K by its
//                                    norm factor in float32 before the float16
//                                    rounding, both straight from global memory;
//                                    the accumulator is seeded with the window
//                                    mask (0 or -inf; padded levels -inf);
//   P = exp2(S^T - max) in one pass (all keys of a query are present), bf16;
//   O^T (64 d x 16 queries) += V^T . P^T  bf16 MFMA with the V^T fragments read
//                                    by the LDS transpose read from the column's
//                                    V rows, staged by the direct-to-LDS copy
//                                    (160-byte rows, pad columns copy column 0);
//   L = 1 . P^T                      the row sums (every lane gets its query's).
// The lane layouts are those of the neighbourhood kernels: a lane (qn, g) holds
// keys 16c + 4g + i of query qn in S^T, and P^T packed in place is the B operand
// of the P.V product with the keys in the same (permuted) order as the
// transpose reads deliver V.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"

namespace strata {
namespace {

using namespace mfma;

constexpr int kD = 64;
constexpr int kVRow = 160;           // LDS bytes per staged V row (8 data + 2 pad 16-byte columns)
constexpr int kWaves = 4;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct ColArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* out;
  float* lse;
  const uint16_t* gate;  // with GATE: logits per (token, head) (gate_dim 1) or per channel
  int gate_dim;
  float eps;
  int Z, kz;
  int64_t HW;            // tokens per level
  int64_t ncol;          // B * heads * H * W
  float qscale;          // scale * log2(e)
};

template <int NB, bool NORM, bool GATE>
__global__ void __launch_bounds__(64 * kWaves) na3d_col_kernel(ColArgs a) {
  constexpr int ZP = 16 * NB;                       // padded levels
  constexpr int SLOTS = ZP * (kVRow / 16);          // 16-byte slots of the V tile
  constexpr int ITV = (SLOTS + 63) / 64;            // copy instructions per wave
  __shared__ __attribute__((aligned(16))) char sV[kWaves][ITV * 64 * 16];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, qn = lane & 15;
  const int Z = a.Z, kz = a.kz;
  const int64_t HW = a.HW;
  char* tv = sV[wave];

  // lane-constant parts: V copy offsets (rows clamped into the column, pad
  // columns copy column 0) and transpose-read addresses
  int vrow[ITV], vcol[ITV];  // level and element offset in the row of this lane's V slots
#pragma unroll
  for (int it = 0; it < ITV; ++it) {
    const int s = it * 64 + lane;
    vrow[it] = min(min(s / 10, ZP - 1), Z - 1);
    vcol[it] = (s % 10 < 8 ? s % 10 : 0) * 8;
  }
  uint32_t vaddr[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) vaddr[c] = (16 * c + 4 * g + (qn >> 2)) * kVRow + (qn & 3) * 8;
  // window mask, per (query block, key block): key 16c + 4g + i of query 16b + qn
  f32x4 bias[NB][NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int qi = min(16 * b + qn, Z - 1);
    const int ws = win_start(qi, Z, kz);
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * c + 4 * g + i;
        bias[b][c][i] = (j < Z && j >= ws && j < ws + kz) ? 0.f : -INFINITY;
      }
  }
  const bf16x8 ones = __builtin_bit_cast(bf16x8, make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));

  const int64_t nwaves = (int64_t)gridDim.x * kWaves;
  for (int64_t col = (int64_t)blockIdx.x * kWaves + wave; col < a.ncol; col += nwaves) {
    // column (t, h, y, x) = col: token of level z is ((t*heads + h) * Z + z) * HW + yx
    const int64_t th = col / HW, yx = col - th * HW;
    const int64_t base = th * Z * HW + yx;  // token index of level 0
    auto tok = [&](int z) { return base + (int64_t)z * HW; };

    // V rows -> LDS (direct copy); its wait comes before the transpose reads
#pragma unroll
    for (int it = 0; it < ITV; ++it) copy16_to_lds(a.v + tok(vrow[it]) * kD + vcol[it], tv + it * 64 * 16);
    // Q (B operand) and K (A operand) fragments: level 16b + qn, d = 8g.. and 32 + 8g..
    uint4 qraw[NB][2], kraw[NB][2];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int z = min(16 * b + qn, Z - 1);
      const uint4* qs = reinterpret_cast<const uint4*>(a.q + tok(z) * kD);
      const uint4* ks = reinterpret_cast<const uint4*>(a.k + tok(z) * kD);
      qraw[b][0] = qs[g];
      qraw[b][1] = qs[4 + g];
      kraw[b][0] = ks[g];
      kraw[b][1] = ks[4 + g];
    }
    f16x8 qf[NB][2], kf[NB][2];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float mq = a.qscale, mk = 1.f;
      if constexpr (NORM) {  // the 4 lanes of a row hold its 64 values
        mq *= __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(qraw[b][1], sumsq8(qraw[b][0], 0.f))) * (1.f / kD) + a.eps);
        mk = __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(kraw[b][1], sumsq8(kraw[b][0], 0.f))) * (1.f / kD) + a.eps);
      }
      qf[b][0] = __builtin_bit_cast(f16x8, scale8h(qraw[b][0], mq));
      qf[b][1] = __builtin_bit_cast(f16x8, scale8h(qraw[b][1], mq));
      kf[b][0] = __builtin_bit_cast(f16x8, scale8h(kraw[b][0], mk));
      kf[b][1] = __builtin_bit_cast(f16x8, scale8h(kraw[b][1], mk));
    }
    __builtin_amdgcn_s_waitcnt(0);  // this lane's V copies have landed (each lane reads its own wave's tile)
    __builtin_amdgcn_wave_barrier();
    // V^T fragments: d block t, keys of chunks (0, 1)
    bf16x8 vf[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const i16x4 lo = tr_read(tv + vaddr[0] + 32 * t);
      const i16x4 hi = NB > 1 ? tr_read(tv + vaddr[NB > 1 ? 1 : 0] + 32 * t) : i16x4{0, 0, 0, 0};
      const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
      vf[t] = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
    }

#pragma unroll
    for (int b = 0; b < NB; ++b) {  // query block
      f32x4 s[NB];
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[c][0], qf[b][0], bias[b][c], 0, 0, 0);
        s[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[c][1], qf[b][1], acc, 0, 0, 0);
      }
      float mx = fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3]));
      if constexpr (NB > 1) mx = fmaxf(mx, fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
      mx = max_over_rows(mx);
      uint32_t pk[2][2] = {{0u, 0u}, {0u, 0u}};
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        pk[c][0] = pack2(__builtin_amdgcn_exp2f(s[c][0] - mx), __builtin_amdgcn_exp2f(s[c][1] - mx));
        pk[c][1] = pack2(__builtin_amdgcn_exp2f(s[c][2] - mx), __builtin_amdgcn_exp2f(s[c][3] - mx));
      }
      const bf16x8 pf = __builtin_bit_cast(bf16x8, make_uint4(pk[0][0], pk[0][1], pk[1][0], pk[1][1]));
      f32x4 o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[t], pf, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
      const f32x4 lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
      const int z = 16 * b + qn;
      if (z < Z) {
        const float lt = lsum[0];
        float inv = 1.f / lt;
        const int64_t tk = tok(z);
        if constexpr (GATE)
          if (a.gate_dim == 1) inv *= sigmoid_fast(bf16_to_f32(a.gate[tk]));
        uint2* dst = reinterpret_cast<uint2*>(a.out + tk * kD);
#pragma unroll
        for (int t = 0; t < 4; ++t) {  // d = 16t + 4g + i
          f32x4 r = o[t] * inv;
          if constexpr (GATE)
            if (a.gate_dim != 1) r *= sigmoid4_bf16(reinterpret_cast<const uint2*>(a.gate + tk * kD)[4 * t + g]);
          dst[4 * t + g] = make_uint2(pack2(r[0], r[1]), pack2(r[2], r[3]));
        }
        if (a.lse && g == 0) a.lse[tk] = (mx + __log2f(lt)) * kLn2;
      }
    }
    __builtin_amdgcn_wave_barrier();  // the next column's copies overwrite this wave's V tile
  }
}

}  // namespace

// Column-wise forward for windows (kz, 1, 1) with Z <= 32 (bf16, head_dim 64);
// false for any other problem.
bool launch_na3d_fwd_col(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                         const void* v, void* out, float* lse, hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD || d.ky != 1 || d.kx != 1 || d.Z > 32) return false;
  ColArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.gate = static_cast<const uint16_t*>(o.gate);
  a.gate_dim = o.gate_dim;
  a.eps = o.eps;
  a.Z = d.Z;
  a.kz = d.kz;
  a.HW = (int64_t)d.H * d.W;
  a.ncol = (int64_t)d.B * d.heads * a.HW;
  a.qscale = d.scale * kLog2e;
  const int64_t want = (a.ncol + kWaves - 1) / kWaves;
  const unsigned blocks = (unsigned)(want < 65536 ? want : 65536);
  const dim3 grid(blocks), block(64 * kWaves);
  const bool nb2 = d.Z > 16;
#define L(NB, N, G) hipLaunchKernelGGL((na3d_col_kernel<NB, N, G>), grid, block, 0, s, a)
  if (nb2) {
    if (o.qk_norm) { if (o.gate) L(2, true, true); else L(2, true, false); }
    else { if (o.gate) L(2, false, true); else L(2, false, false); }
  } else {
    if (o.qk_norm) { if (o.gate) L(1, true, true); else L(1, true, false); }
    else { if (o.gate) L(1, false, true); else L(1, false, false); }
  }
#undef L
  return true;
}

// ---------------------------------------------------------------------------
// Column-wise attention backward: dq, dk, dv of one column per wave.
//
// A lane's fragments of a row (level 16b + qn, d = 8g.. and 32 + 8g..) serve as
// the A operand and as the B operand of a 16x16x32 MFMA alike, so both
// orientations come from the same registers:
//   queries as columns (dq):  S^T = K^ Q^T seeded with the mask, P^T = exp2(S^T
//     - lse2), Y^T = V dO^T - D, dS^T = P^T Y^T, dQ^T = K^T dS^T with the K^T
//     fragments read transposed from the float16 K^ rows staged in LDS;
//   keys as columns (dk, dv):  S = Q K^T, P, Y = dO V^T - D, dS = P Y,
//     dV^T = dO^T P (dO rows staged in LDS by the direct copy, read
//     transposed), dK^T = Q^T dS (float16 Q^ rows staged in LDS).
// dS enters its float16 MFMA scaled by 2^(15 - E), E the exponent of the
// largest |dS| of the column's query (resp. key): all keys of a query are
// present at once, so one exact power-of-two scale suffices.  lse2 = lse log2 e
// and D of padded levels are +inf and 0, so their P and dS vanish.
// Options: QK RMSNorm (q^ = r q, k^ = r k in float32 before the float16
// rounding; dq = r (dq^ - q^ mean(dq^ q^)) and likewise dk, q^ and k^ re-read
// from the raw rows), and dO given as two bf16 terms hi + lo.
struct ColBwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* dout;
  const uint16_t* dout_lo;
  const float* lse;   // natural log
  const float* dvec;  // D = rowsum(dO * O)
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  float eps;
  int Z, kz;
  int64_t HW, ncol;
  float scale, qscale;
};

namespace {

constexpr int kMinExp = -100;

template <int NB, bool NORM, bool LO>
__global__ void __launch_bounds__(64 * kWaves) na3d_col_bwd_kernel(ColBwdArgs a) {
  constexpr int ZP = 16 * NB;
  constexpr int RB = 160;                            // LDS bytes per staged row
  constexpr int ITG = (ZP * (RB / 16) + 63) / 64;    // direct-copy instructions per staged dO tile
  constexpr int GT = ITG * 64 * 16;
  __shared__ __attribute__((aligned(16))) char sQ[kWaves][ZP * RB];
  __shared__ __attribute__((aligned(16))) char sK[kWaves][ZP * RB];
  __shared__ __attribute__((aligned(16))) char sG[kWaves][GT];
  __shared__ __attribute__((aligned(16))) char sGl[kWaves][LO ? GT : 16];
  __shared__ __attribute__((aligned(16))) float sL[kWaves][ZP];
  __shared__ __attribute__((aligned(16))) float sD[kWaves][ZP];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, qn = lane & 15;
  const int Z = a.Z, kz = a.kz;
  const int64_t HW = a.HW;
  char* tq = sQ[wave];
  char* tk = sK[wave];
  char* tg = sG[wave];
  char* tgl = sGl[wave];

  int grow[ITG], gcol[ITG];  // dO copy slots: level and element offset (pad columns copy column 0)
#pragma unroll
  for (int it = 0; it < ITG; ++it) {
    const int s = it * 64 + lane;
    grow[it] = min(min(s / 10, ZP - 1), Z - 1);
    gcol[it] = (s % 10 < 8 ? s % 10 : 0) * 8;
  }
  // transpose-read rows of chunk c: 16c + 4g + qn/4, 8 bytes at (qn % 4) of a 16-element block
  uint32_t taddr[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) taddr[c] = (16 * c + 4 * g + (qn >> 2)) * RB + (qn & 3) * 8;
  // masks: queries as columns (key 16c + 4g + i, query 16b + qn) and keys as
  // columns (query 16b + 4g + i, key 16c + qn)
  f32x4 biasT[NB][NB], biasN[NB][NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        {
          const int qi = min(16 * b + qn, Z - 1), j = 16 * c + 4 * g + i, ws = win_start(qi, Z, kz);
          biasT[b][c][i] = (j < Z && j >= ws && j < ws + kz) ? 0.f : -INFINITY;
        }
        {
          const int qi = min(16 * b + 4 * g + i, Z - 1), j = 16 * c + qn, ws = win_start(qi, Z, kz);
          biasN[b][c][i] = (j < Z && j >= ws && j < ws + kz) ? 0.f : -INFINITY;
        }
      }

  auto tr8 = [&](const char* tile, int t) {  // 16 d x 32 rows (chunks 0 and 1), transposed
    const i16x4 lo = tr_read(tile + taddr[0] + 32 * t);
    const i16x4 hi = NB > 1 ? tr_read(tile + taddr[NB > 1 ? 1 : 0] + 32 * t) : i16x4{0, 0, 0, 0};
    const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
    return make_uint4(l2.x, l2.y, h2.x, h2.y);
  };
  auto dmax = [](const f32x4& x, float m) {
    return fmaxf(m, fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3]))));
  };

  const int64_t nwaves = (int64_t)gridDim.x * kWaves;
  for (int64_t col = (int64_t)blockIdx.x * kWaves + wave; col < a.ncol; col += nwaves) {
    const int64_t th = col / HW, yx = col - th * HW;
    const int64_t base = th * Z * HW + yx;
    auto tok = [&](int z) { return base + (int64_t)z * HW; };

    // dO rows -> LDS (direct copy), row fragments -> registers
#pragma unroll
    for (int it = 0; it < ITG; ++it) {
      copy16_to_lds(a.dout + tok(grow[it]) * kD + gcol[it], tg + it * 64 * 16);
      if constexpr (LO) copy16_to_lds(a.dout_lo + tok(grow[it]) * kD + gcol[it], tgl + it * 64 * 16);
    }
    uint4 qr[NB][2], kr[NB][2], vr[NB][2], gr[NB][2], glr[LO ? NB : 1][2];
    float lseA[NB], dA[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int z = min(16 * b + qn, Z - 1);
      const int64_t tz = tok(z);
      const uint4* qs = reinterpret_cast<const uint4*>(a.q + tz * kD);
      const uint4* ks = reinterpret_cast<const uint4*>(a.k + tz * kD);
      const uint4* vs = reinterpret_cast<const uint4*>(a.v + tz * kD);
      const uint4* gs = reinterpret_cast<const uint4*>(a.dout + tz * kD);
      qr[b][0] = qs[g]; qr[b][1] = qs[4 + g];
      kr[b][0] = ks[g]; kr[b][1] = ks[4 + g];
      vr[b][0] = vs[g]; vr[b][1] = vs[4 + g];
      gr[b][0] = gs[g]; gr[b][1] = gs[4 + g];
      if constexpr (LO) {
        const uint4* ls = reinterpret_cast<const uint4*>(a.dout_lo + tz * kD);
        glr[b][0] = ls[g]; glr[b][1] = ls[4 + g];
      }
      const bool live = 16 * b + qn < Z;
      lseA[b] = live ? a.lse[tz] * kLog2e : INFINITY;
      dA[b] = live ? a.dvec[tz] : 0.f;
    }
    // norms, float16 operands, staged rows of q^ and k^
    f16x8 qf[NB][2], kf[NB][2];
    float rq[NB], rk[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      rq[b] = 1.f;
      rk[b] = 1.f;
      if constexpr (NORM) {
        rq[b] = __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(qr[b][1], sumsq8(qr[b][0], 0.f))) * (1.f / kD) + a.eps);
        rk[b] = __builtin_amdgcn_rsqf(sum_over_rows(sumsq8(kr[b][1], sumsq8(kr[b][0], 0.f))) * (1.f / kD) + a.eps);
      }
      qf[b][0] = __builtin_bit_cast(f16x8, scale8h(qr[b][0], a.qscale * rq[b]));
      qf[b][1] = __builtin_bit_cast(f16x8, scale8h(qr[b][1], a.qscale * rq[b]));
      const uint4 k0 = scale8h(kr[b][0], rk[b]), k1 = scale8h(kr[b][1], rk[b]);
      kf[b][0] = __builtin_bit_cast(f16x8, k0);
      kf[b][1] = __builtin_bit_cast(f16x8, k1);
      char* rowq = tq + (16 * b + qn) * RB;
      char* rowk = tk + (16 * b + qn) * RB;
      st16(rowq + 16 * g, scale8h(qr[b][0], rq[b]));
      st16(rowq + 64 + 16 * g, scale8h(qr[b][1], rq[b]));
      st16(rowk + 16 * g, k0);
      st16(rowk + 64 + 16 * g, k1);
      if (g == 0) {
        sL[wave][16 * b + qn] = lseA[b];
        sD[wave][16 * b + qn] = dA[b];
      }
    }
    __builtin_amdgcn_s_waitcnt(0);  // the wave's dO copies and LDS writes are complete
    __builtin_amdgcn_wave_barrier();

    // ---- queries as columns: dq ----------------------------------------------
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      f32x4 ds[NB];
      float mx = 0.f;
      const f32x4 nd = {-dA[b], -dA[b], -dA[b], -dA[b]};
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        f32x4 s = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[c][0], qf[b][0], biasT[b][c], 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[c][1], qf[b][1], s, 0, 0, 0);
        f32x4 y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[c][0]),
                                                          __builtin_bit_cast(bf16x8, gr[b][0]), nd, 0, 0, 0);
        y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[c][1]),
                                                    __builtin_bit_cast(bf16x8, gr[b][1]), y, 0, 0, 0);
        if constexpr (LO) {
          y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[c][0]),
                                                      __builtin_bit_cast(bf16x8, glr[b][0]), y, 0, 0, 0);
          y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[c][1]),
                                                      __builtin_bit_cast(bf16x8, glr[b][1]), y, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) ds[c][i] = __builtin_amdgcn_exp2f(s[i] - lseA[b]) * y[i];
        mx = dmax(ds[c], mx);
      }
      const int e = max(__builtin_amdgcn_frexp_expf(max_over_rows(mx)), kMinExp);
      const float up = __builtin_amdgcn_ldexpf(1.f, 15 - e);
      uint32_t dk2[2][2] = {{0u, 0u}, {0u, 0u}};
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        dk2[c][0] = pack2h_rne(ds[c][0] * up, ds[c][1] * up);
        dk2[c][1] = pack2h_rne(ds[c][2] * up, ds[c][3] * up);
      }
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(dk2[0][0], dk2[0][1], dk2[1][0], dk2[1][1]));
      const float down = a.scale * __builtin_amdgcn_ldexpf(1.f, e - 15);
      f32x4 x[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        x[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, tr8(tk, t)), df,
                                                      f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0) * down;
      const int z = 16 * b + qn;
      const int64_t tz = tok(min(z, Z - 1));
      if constexpr (NORM) {  // through the norm's Jacobian; lane holds d = 16t + 4g + i
        const uint2* src = reinterpret_cast<const uint2*>(a.q + tz * kD);
        f32x4 xh[4];
        float cdot = 0.f;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint2 w = src[4 * t + g];
          xh[t] = f32x4{lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y)} * rq[b];
#pragma unroll
          for (int i = 0; i < 4; ++i) cdot = fmaf(x[t][i], xh[t][i], cdot);
        }
        cdot = sum_over_rows(cdot) * (1.f / kD);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) x[t][i] = rq[b] * fmaf(-xh[t][i], cdot, x[t][i]);
      }
      if (z < Z) {
        uint2* dst = reinterpret_cast<uint2*>(a.dq + tz * kD);
#pragma unroll
        for (int t = 0; t < 4; ++t) dst[4 * t + g] = make_uint2(pack2(x[t][0], x[t][1]), pack2(x[t][2], x[t][3]));
      }
    }

    // ---- keys as columns: dk, dv ----------------------------------------------
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      f32x4 ds[NB];
      uint32_t pb[2][2] = {{0u, 0u}, {0u, 0u}};
      float mx = 0.f;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float4 l4 = *reinterpret_cast<const float4*>(&sL[wave][16 * b + 4 * g]);
        const float4 d4 = *reinterpret_cast<const float4*>(&sD[wave][16 * b + 4 * g]);
        f32x4 s = __builtin_amdgcn_mfma_f32_16x16x32_f16(qf[b][0], kf[c][0], biasN[b][c], 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_16x16x32_f16(qf[b][1], kf[c][1], s, 0, 0, 0);
        f32x4 y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, gr[b][0]),
                                                          __builtin_bit_cast(bf16x8, vr[c][0]),
                                                          f32x4{-d4.x, -d4.y, -d4.z, -d4.w}, 0, 0, 0);
        y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, gr[b][1]),
                                                    __builtin_bit_cast(bf16x8, vr[c][1]), y, 0, 0, 0);
        if constexpr (LO) {
          y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, glr[b][0]),
                                                      __builtin_bit_cast(bf16x8, vr[c][0]), y, 0, 0, 0);
          y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, glr[b][1]),
                                                      __builtin_bit_cast(bf16x8, vr[c][1]), y, 0, 0, 0);
        }
        const float p0 = __builtin_amdgcn_exp2f(s[0] - l4.x), p1 = __builtin_amdgcn_exp2f(s[1] - l4.y);
        const float p2 = __builtin_amdgcn_exp2f(s[2] - l4.z), p3 = __builtin_amdgcn_exp2f(s[3] - l4.w);
        pb[b][0] = pack2(p0, p1);
        pb[b][1] = pack2(p2, p3);
        ds[b] = f32x4{p0 * y[0], p1 * y[1], p2 * y[2], p3 * y[3]};
        mx = dmax(ds[b], mx);
      }
      const int e = max(__builtin_amdgcn_frexp_expf(max_over_rows(mx)), kMinExp);
      const float up = __builtin_amdgcn_ldexpf(1.f, 15 - e);
      uint32_t db[2][2] = {{0u, 0u}, {0u, 0u}};
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        db[b][0] = pack2h_rne(ds[b][0] * up, ds[b][1] * up);
        db[b][1] = pack2h_rne(ds[b][2] * up, ds[b][3] * up);
      }
      const bf16x8 pf = __builtin_bit_cast(bf16x8, make_uint4(pb[0][0], pb[0][1], pb[1][0], pb[1][1]));
      const f16x8 df = __builtin_bit_cast(f16x8, make_uint4(db[0][0], db[0][1], db[1][0], db[1][1]));
      const float down = a.scale * __builtin_amdgcn_ldexpf(1.f, e - 15);
      f32x4 xv[4], xk[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        xv[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, tr8(tg, t)), pf,
                                                       f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
        if constexpr (LO)
          xv[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, tr8(tgl, t)), pf, xv[t], 0, 0, 0);
        xk[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, tr8(tq, t)), df,
                                                       f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0) * down;
      }
      const int z = 16 * c + qn;
      const int64_t tz = tok(min(z, Z - 1));
      if constexpr (NORM) {
        const uint2* src = reinterpret_cast<const uint2*>(a.k + tz * kD);
        f32x4 xh[4];
        float cdot = 0.f;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint2 w = src[4 * t + g];
          xh[t] = f32x4{lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y)} * rk[c];
#pragma unroll
          for (int i = 0; i < 4; ++i) cdot = fmaf(xk[t][i], xh[t][i], cdot);
        }
        cdot = sum_over_rows(cdot) * (1.f / kD);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) xk[t][i] = rk[c] * fmaf(-xh[t][i], cdot, xk[t][i]);
      }
      if (z < Z) {
        uint2* dkd = reinterpret_cast<uint2*>(a.dk + tz * kD);
        uint2* dvd = reinterpret_cast<uint2*>(a.dv + tz * kD);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          dkd[4 * t + g] = make_uint2(pack2(xk[t][0], xk[t][1]), pack2(xk[t][2], xk[t][3]));
          dvd[4 * t + g] = make_uint2(pack2(xv[t][0], xv[t][1]), pack2(xv[t][2], xv[t][3]));
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);  // LDS reads of this column retire before the next column's writes
    __builtin_amdgcn_wave_barrier();
  }
}

}  // namespace

// Column-wise backward (dq, dk, dv in one pass) for windows (kz, 1, 1) with
// Z <= 32 (bf16, head_dim 64); reads D from dvec.  False for any other problem.
bool launch_na3d_bwd_col(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                         const void* v, const void* dout, const float* lse, const float* dvec, void* dq,
                         void* dk, void* dv, hipStream_t s) {
  if (d.dtype != STRATA_BF16 || d.head_dim != kD || d.ky != 1 || d.kx != 1 || d.Z > 32) return false;
  ColBwdArgs a = {};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.dout = static_cast<const uint16_t*>(dout);
  a.dout_lo = static_cast<const uint16_t*>(o.dout_lo);
  a.lse = lse;
  a.dvec = dvec;
  a.dq = static_cast<uint16_t*>(dq);
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.eps = o.eps;
  a.Z = d.Z;
  a.kz = d.kz;
  a.HW = (int64_t)d.H * d.W;
  a.ncol = (int64_t)d.B * d.heads * a.HW;
  a.scale = d.scale;
  a.qscale = d.scale * kLog2e;
  const int64_t want = (a.ncol + kWaves - 1) / kWaves;
  const dim3 grid((unsigned)(want < 65536 ? want : 65536)), block(64 * kWaves);
  const bool nb2 = d.Z > 16, norm = o.qk_norm != 0, lo = o.dout_lo != nullptr;
#define L(NB, N, LO_) hipLaunchKernelGGL((na3d_col_bwd_kernel<NB, N, LO_>), grid, block, 0, s, a)
  if (nb2) {
    if (norm) { if (lo) L(2, true, true); else L(2, true, false); }
    else { if (lo) L(2, false, true); else L(2, false, false); }
  } else {
    if (norm) { if (lo) L(1, true, true); else L(1, true, false); }
    else { if (lo) L(1, false, true); else L(1, false, false); }
  }
#undef L
  return true;
}

}  // namespace strata

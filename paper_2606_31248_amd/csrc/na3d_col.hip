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

}  // namespace strata

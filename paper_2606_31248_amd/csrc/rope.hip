// StereoRoPE: phase table from stereographic coordinates, and the pairwise rotation.
// Both are streaming kernels bound by HBM bandwidth.
#include "common.h"
#include "kernels.h"

namespace strata {

// One thread per (b, y, x, pair t).  Phases in float64, stored as float32 (cos, sin).
// The frequencies base^(-t'/q) depend on the pair alone: a block computes them
// once into LDS (the same pow call, so the same values) when they fit.
constexpr int kPhaseThreads = 256;

__global__ void __launch_bounds__(kPhaseThreads) rope_phases_kernel(const float* __restrict__ coords,
                                                                    int64_t n_pos, int n_pairs, double base,
                                                                    float2* __restrict__ cs) {
  __shared__ double omega[kPhaseThreads];
  const int q = n_pairs >> 1;  // head_dim / 4 pairs per axis
  auto freq = [&](int t) {
    const int tt = t - (t >= q) * q;
    return pow(base, -(double)tt / (double)q);
  };
  const bool table = n_pairs <= kPhaseThreads;
  if (table) {
    if ((int)threadIdx.x < n_pairs) omega[threadIdx.x] = freq(threadIdx.x);
    __syncthreads();
  }
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_pos * n_pairs) return;
  int t = (int)(idx % n_pairs);
  int64_t pos = idx / n_pairs;
  int axis = t >= q;
  double c = (double)coords[2 * pos + axis];
  double th = c * (table ? omega[t] : freq(t));
  double sn, cn;
  sincos(th, &sn, &cn);
  cs[idx] = make_float2((float)cn, (float)sn);
}

void launch_rope_phases(const float* coords, int B, int H, int W, int head_dim, double base,
                        float* cs, hipStream_t s) {
  int64_t n_pos = (int64_t)B * H * W;
  int n_pairs = head_dim / 2;
  int64_t n = n_pos * n_pairs;
  int threads = kPhaseThreads;
  int blocks = (int)((n + threads - 1) / threads);
  hipLaunchKernelGGL(rope_phases_kernel, dim3(blocks), dim3(threads), 0, s, coords, n_pos, n_pairs,
                     base, reinterpret_cast<float2*>(cs));
}

// One thread per 4 pairs (8 elements) of one token: a 16-byte bf16 or 32-byte
// f32 load and store plus 32 bytes of phases.  Consecutive threads walk the
// head_dim of one token, then the next token, so every access is contiguous.
// tok_per_b = heads*Z*H*W tokens per tile; HW = H*W positions per tile.
template <bool BF16>
__global__ void rope_apply_kernel(const void* __restrict__ xin, void* __restrict__ yout,
                                  const float4* __restrict__ cs, int64_t n_groups,
                                  int groups_per_tok, int64_t tok_per_b, int HW, float sign) {
  int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  int gi = (int)(g % groups_per_tok);
  int64_t tok = g / groups_per_tok;
  int64_t b = tok / tok_per_b;
  int64_t pos = b * HW + (int)(tok % HW);
  // the phase row of a position holds head_dim/2 (cos, sin) pairs = 2*groups_per_tok float4
  const float4* ph = cs + pos * (2 * groups_per_tok) + 2 * gi;
  float4 p0 = ph[0], p1 = ph[1];
  float c[4] = {p0.x, p0.z, p1.x, p1.z};
  float s[4] = {sign * p0.y, sign * p0.w, sign * p1.y, sign * p1.w};
  float v[8];
  if (BF16) {
    uint4 raw = reinterpret_cast<const uint4*>(xin)[g];
    uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_to_f32((uint16_t)(w[i] & 0xFFFFu));
      v[2 * i + 1] = bf16_to_f32((uint16_t)(w[i] >> 16));
    }
  } else {
    float4 a = reinterpret_cast<const float4*>(xin)[2 * g];
    float4 bq = reinterpret_cast<const float4*>(xin)[2 * g + 1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = bq.x; v[5] = bq.y; v[6] = bq.z; v[7] = bq.w;
  }
  float o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float a = v[2 * i], bb = v[2 * i + 1];
    o[2 * i] = fmaf(a, c[i], -bb * s[i]);
    o[2 * i + 1] = fmaf(a, s[i], bb * c[i]);
  }
  if (BF16) {
    uint4 r;
    r.x = pack_bf16x2(o[0], o[1]);
    r.y = pack_bf16x2(o[2], o[3]);
    r.z = pack_bf16x2(o[4], o[5]);
    r.w = pack_bf16x2(o[6], o[7]);
    reinterpret_cast<uint4*>(yout)[g] = r;
  } else {
    reinterpret_cast<float4*>(yout)[2 * g] = make_float4(o[0], o[1], o[2], o[3]);
    reinterpret_cast<float4*>(yout)[2 * g + 1] = make_float4(o[4], o[5], o[6], o[7]);
  }
}

void launch_rope_apply(const void* x, void* y, const float* cs, int B, int heads, int Z, int H,
                       int W, int head_dim, strata_dtype dt, int transpose, hipStream_t s) {
  int groups_per_tok = head_dim / 8;
  int64_t n_tok = (int64_t)B * heads * Z * H * W;
  int64_t n_groups = n_tok * groups_per_tok;
  int64_t tok_per_b = (int64_t)heads * Z * H * W;
  float sign = transpose ? -1.0f : 1.0f;
  int threads = 256;
  int blocks = (int)((n_groups + threads - 1) / threads);
  const float4* c4 = reinterpret_cast<const float4*>(cs);
  if (dt == STRATA_BF16)
    hipLaunchKernelGGL(rope_apply_kernel<true>, dim3(blocks), dim3(threads), 0, s, x, y, c4, n_groups,
                       groups_per_tok, tok_per_b, H * W, sign);
  else
    hipLaunchKernelGGL(rope_apply_kernel<false>, dim3(blocks), dim3(threads), 0, s, x, y, c4,
                       n_groups, groups_per_tok, tok_per_b, H * W, sign);
}

}  // namespace strata

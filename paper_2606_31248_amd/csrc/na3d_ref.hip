// Plain neighbourhood-attention kernels: one thread per query (forward, dq) or
// per key (dk/dv), float32 arithmetic, StereoRoPE applied while loading.  The
// options: QK RMSNorm after the rotation (the rotation keeps the mean square;
// in the backward its Jacobian is applied to dq and dk before the transposed
// rotation), the sigmoid gate on the forward output, and the backward's
// upstream gradient given as two terms.
// They serve the float32 path and every shape the MFMA kernels do not cover.
#include "common.h"
#include "kernels.h"

namespace strata {

template <typename T>
__device__ __forceinline__ float ld(const T* p);
template <>
__device__ __forceinline__ float ld<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

template <typename T>
__device__ __forceinline__ void st(T* p, float v);
template <>
__device__ __forceinline__ void st<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void st<uint16_t>(uint16_t* p, float v) { *p = f32_to_bf16(v); }

// Load a head_dim vector and rotate it by the phases of its (b, y, x) (sign -1: R^T).
template <typename T, int D>
__device__ __forceinline__ void load_rot(const T* src, const float2* ph, float sign, float* dst) {
#pragma unroll
  for (int t = 0; t < D / 2; ++t) {
    float a = ld(src + 2 * t), b = ld(src + 2 * t + 1);
    if (ph) {
      float2 p = ph[t];
      float s = sign * p.y;
      dst[2 * t] = fmaf(a, p.x, -b * s);
      dst[2 * t + 1] = fmaf(a, s, b * p.x);
    } else {
      dst[2 * t] = a;
      dst[2 * t + 1] = b;
    }
  }
}

// Divide a head_dim vector by its root mean square (QK RMSNorm, no scale);
// returns the factor r = (mean(x^2) + eps)^(-1/2).
template <int D>
__device__ __forceinline__ float rms_normalise(float* x, float eps) {
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < D; ++e) ss = fmaf(x[e], x[e], ss);
  const float r = 1.f / sqrtf(ss / D + eps);
#pragma unroll
  for (int e = 0; e < D; ++e) x[e] *= r;
  return r;
}

// Jacobian of the norm applied to a gradient g of x^ = r x (in place):
// g <- r (g - x^ mean(g x^)).  Rotation-invariant, so g and x^ may both be
// given in the rotated frame.
template <int D>
__device__ __forceinline__ void rms_norm_vjp(float* g, const float* xh, float r) {
  float c = 0.f;
#pragma unroll
  for (int e = 0; e < D; ++e) c = fmaf(g[e], xh[e], c);
  c /= D;
#pragma unroll
  for (int e = 0; e < D; ++e) g[e] = r * fmaf(-xh[e], c, g[e]);
}

// upstream gradient element: dout (+ its low part when given as two terms)
template <typename T>
__device__ __forceinline__ float ld_g(const T* hi, const T* lo, int64_t i) {
  return lo ? ld(hi + i) + ld(lo + i) : ld(hi + i);
}

__device__ __forceinline__ float sigmoid(float g) { return 1.f / (1.f + expf(-g)); }

struct Dims {
  int B, heads, Z, H, W, kz, ky, kx;
  float scale;
};

__device__ __forceinline__ void split_tok(int64_t i, const Dims& d, int& b, int& h, int& z, int& y,
                                          int& x) {
  x = (int)(i % d.W); i /= d.W;
  y = (int)(i % d.H); i /= d.H;
  z = (int)(i % d.Z); i /= d.Z;
  h = (int)(i % d.heads); i /= d.heads;
  b = (int)i;
}

template <typename T, int D>
__global__ void __launch_bounds__(128) na3d_fwd_ref_kernel(const T* __restrict__ q, const T* __restrict__ k,
                                                           const T* __restrict__ v, const float2* __restrict__ cs,
                                                           T* __restrict__ out, float* __restrict__ lse, Dims dm,
                                                           NaOpts opt) {
  int64_t nq = (int64_t)dm.B * dm.heads * dm.Z * dm.H * dm.W;
  int64_t qi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (qi >= nq) return;
  int b, h, z, y, x;
  split_tok(qi, dm, b, h, z, y, x);
  const int64_t bh = (int64_t)b * dm.heads + h;
  float qv[D], kv[D], acc[D];
  load_rot<T, D>(q + qi * D, cs ? cs + (((int64_t)b * dm.H + y) * dm.W + x) * (D / 2) : nullptr, 1.f, qv);
  if (opt.qk_norm) rms_normalise<D>(qv, opt.eps);  // the rotation keeps the mean square
#pragma unroll
  for (int e = 0; e < D; ++e) acc[e] = 0.f;
  float m = -INFINITY, l = 0.f;
  int zs = win_start(z, dm.Z, dm.kz), ys = win_start(y, dm.H, dm.ky), xs = win_start(x, dm.W, dm.kx);
  for (int jz = zs; jz < zs + dm.kz; ++jz)
    for (int jy = ys; jy < ys + dm.ky; ++jy)
      for (int jx = xs; jx < xs + dm.kx; ++jx) {
        int64_t kj = ((bh * dm.Z + jz) * dm.H + jy) * dm.W + jx;
        load_rot<T, D>(k + kj * D, cs ? cs + (((int64_t)b * dm.H + jy) * dm.W + jx) * (D / 2) : nullptr, 1.f, kv);
        if (opt.qk_norm) rms_normalise<D>(kv, opt.eps);
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < D; ++e) s = fmaf(qv[e], kv[e], s);
        s *= dm.scale;
        float mn = fmaxf(m, s);
        float alpha = expf(m - mn);
        float p = expf(s - mn);
        l = fmaf(l, alpha, p);
        const T* vr = v + kj * D;
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = fmaf(acc[e], alpha, p * ld(vr + e));
        m = mn;
      }
  float inv = 1.f / l;
  const T* gate = static_cast<const T*>(opt.gate);
  if (gate && opt.gate_dim == 1) inv *= sigmoid(ld(gate + qi));
#pragma unroll
  for (int e = 0; e < D; ++e) {
    float val = acc[e] * inv;
    if (gate && opt.gate_dim != 1) val *= sigmoid(ld(gate + qi * D + e));
    st(out + qi * D + e, val);
  }
  if (lse) lse[qi] = m + logf(l);
}

// Small problems: one wave per query, so that a problem of a few thousand
// queries still spreads over the chip.  Lane l takes the keys l, l + 64, ... of
// the query's window (in (z, y, x) order) with its own running maximum, sum and
// accumulator; the 64 partial states are then merged by butterfly exchanges
// (each rescaled to the common maximum before it is added).  The options as in
// the kernel above.
template <typename T, int D>
__global__ void __launch_bounds__(256) na3d_fwd_wave_kernel(const T* __restrict__ q, const T* __restrict__ k,
                                                            const T* __restrict__ v, const float2* __restrict__ cs,
                                                            T* __restrict__ out, float* __restrict__ lse, Dims dm,
                                                            NaOpts opt) {
  const int64_t nq = (int64_t)dm.B * dm.heads * dm.Z * dm.H * dm.W;
  const int64_t qi = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (qi >= nq) return;  // whole waves
  int b, h, z, y, x;
  split_tok(qi, dm, b, h, z, y, x);
  const int64_t bh = (int64_t)b * dm.heads + h;
  float qv[D], kv[D], acc[D];
  load_rot<T, D>(q + qi * D, cs ? cs + (((int64_t)b * dm.H + y) * dm.W + x) * (D / 2) : nullptr, 1.f, qv);
  if (opt.qk_norm) rms_normalise<D>(qv, opt.eps);  // the rotation keeps the mean square
#pragma unroll
  for (int e = 0; e < D; ++e) acc[e] = 0.f;
  float m = -INFINITY, l = 0.f;
  const int zs = win_start(z, dm.Z, dm.kz), ys = win_start(y, dm.H, dm.ky), xs = win_start(x, dm.W, dm.kx);
  const int nyx = dm.ky * dm.kx, nk = dm.kz * nyx;
  for (int t = lane; t < nk; t += 64) {
    const int jz = zs + t / nyx, jy = ys + (t % nyx) / dm.kx, jx = xs + t % dm.kx;
    const int64_t kj = ((bh * dm.Z + jz) * dm.H + jy) * dm.W + jx;
    load_rot<T, D>(k + kj * D, cs ? cs + (((int64_t)b * dm.H + jy) * dm.W + jx) * (D / 2) : nullptr, 1.f, kv);
    if (opt.qk_norm) rms_normalise<D>(kv, opt.eps);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) s = fmaf(qv[e], kv[e], s);
    s *= dm.scale;
    const float mn = fmaxf(m, s);
    const float alpha = expf(m - mn);
    const float p = expf(s - mn);
    l = fmaf(l, alpha, p);
    const T* vr = v + kj * D;
#pragma unroll
    for (int e = 0; e < D; ++e) acc[e] = fmaf(acc[e], alpha, p * ld(vr + e));
    m = mn;
  }
  // merge the lanes: common maximum, then sums of the rescaled partial states
  float mx = m;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  const float f = m == -INFINITY ? 0.f : expf(m - mx);  // a lane without keys adds nothing
  l *= f;
#pragma unroll
  for (int e = 0; e < D; ++e) acc[e] *= f;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    l += __shfl_xor(l, off);
#pragma unroll
    for (int e = 0; e < D; ++e) acc[e] += __shfl_xor(acc[e], off);
  }
  // lane e < D stores element e (times the gate's sigmoid)
  float val = 0.f;
#pragma unroll
  for (int e = 0; e < D; ++e) val = lane == e ? acc[e] : val;
  if (lane < D) {
    float r = val / l;
    const T* gate = static_cast<const T*>(opt.gate);
    if (gate) r *= sigmoid(ld(gate + (opt.gate_dim == 1 ? qi : qi * D + lane)));
    st(out + qi * D + lane, r);
  }
  if (lse && lane == 0) lse[qi] = mx + logf(l);
}

template <typename T, int D>
static void fwd_ref(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                    const void* v, const float* cs, void* out, float* lse, hipStream_t s) {
  Dims dm{d.B, d.heads, d.Z, d.H, d.W, d.kz, d.ky, d.kx, d.scale};
  int64_t nq = (int64_t)d.B * d.heads * d.Z * d.H * d.W;
  // a problem too small to fill the chip with one query per thread (fewer than
  // 2^18 queries) takes one wave per query
  if constexpr (D <= 64) {
    if (nq < ((int64_t)1 << 18)) {
      hipLaunchKernelGGL((na3d_fwd_wave_kernel<T, D>), dim3((unsigned)((nq + 3) / 4)), dim3(256), 0, s,
                         static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                         reinterpret_cast<const float2*>(cs), static_cast<T*>(out), lse, dm, o);
      return;
    }
  }
  // one query per thread; a small problem takes one wave per workgroup so that
  // its workgroups spread over more CUs
  int threads = nq < (int64_t)512 * 128 ? 64 : 128;
  int blocks = (int)((nq + threads - 1) / threads);
  hipLaunchKernelGGL((na3d_fwd_ref_kernel<T, D>), dim3(blocks), dim3(threads), 0, s,
                     static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                     reinterpret_cast<const float2*>(cs), static_cast<T*>(out), lse, dm, o);
}

void launch_na3d_fwd_ref(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                         const void* v, const float* cs, void* out, float* lse, hipStream_t s) {
  if (d.dtype == STRATA_BF16) {
    if (d.head_dim == 32) fwd_ref<uint16_t, 32>(d, o, q, k, v, cs, out, lse, s);
    else if (d.head_dim == 64) fwd_ref<uint16_t, 64>(d, o, q, k, v, cs, out, lse, s);
    else fwd_ref<uint16_t, 128>(d, o, q, k, v, cs, out, lse, s);
  } else {
    if (d.head_dim == 32) fwd_ref<float, 32>(d, o, q, k, v, cs, out, lse, s);
    else if (d.head_dim == 64) fwd_ref<float, 64>(d, o, q, k, v, cs, out, lse, s);
    else fwd_ref<float, 128>(d, o, q, k, v, cs, out, lse, s);
  }
}

// ---- backward ----------------------------------------------------------------
// D_i = <dout_i, out_i> in float32.  A lane reads one 16-byte piece of a row of
// both tensors; the CPR lanes of a row (aligned within the wave) add their
// partial sums by butterfly exchanges.
template <typename T, int D>
__global__ void __launch_bounds__(256) na3d_bwd_pre_kernel(const T* __restrict__ out, const T* __restrict__ dout,
                                                           float* __restrict__ dvec, int64_t nq) {
  constexpr int E = 16 / (int)sizeof(T);  // elements per 16-byte piece
  constexpr int CPR = D / E;              // pieces per row: 4, 8 or 16
  static_assert(64 % CPR == 0, "a row's lanes must not straddle a wave");
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid / CPR;
  const int c = (int)(gid % CPR);
  float acc = 0.f;
  if (row < nq) {
    const uint4 a = *reinterpret_cast<const uint4*>(out + row * D + c * E);
    const uint4 g = *reinterpret_cast<const uint4*>(dout + row * D + c * E);
    const T* pa = reinterpret_cast<const T*>(&a);
    const T* pg = reinterpret_cast<const T*>(&g);
#pragma unroll
    for (int e = 0; e < E; ++e) acc = fmaf(ld(pg + e), ld(pa + e), acc);
  }
#pragma unroll
  for (int off = CPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (row < nq && c == 0) dvec[row] = acc;
}

template <typename T, int D>
__global__ void __launch_bounds__(128) na3d_bwd_dq_ref_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, const float2* __restrict__ cs,
    const T* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ dvec,
    T* __restrict__ dq, Dims dm, BwdOpts opt) {
  int64_t nq = (int64_t)dm.B * dm.heads * dm.Z * dm.H * dm.W;
  int64_t qi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (qi >= nq) return;
  int b, h, z, y, x;
  split_tok(qi, dm, b, h, z, y, x);
  const int64_t bh = (int64_t)b * dm.heads + h;
  const T* dlo = static_cast<const T*>(opt.dout_lo);
  float qv[D], kv[D], g[D], acc[D];
  const float2* phq = cs ? cs + (((int64_t)b * dm.H + y) * dm.W + x) * (D / 2) : nullptr;
  load_rot<T, D>(q + qi * D, phq, 1.f, qv);
  const float rq = opt.qk_norm ? rms_normalise<D>(qv, opt.eps) : 1.f;
#pragma unroll
  for (int e = 0; e < D; ++e) {
    g[e] = ld_g(dout, dlo, qi * D + e);
    acc[e] = 0.f;
  }
  const float L = lse[qi], Di = dvec[qi];
  int zs = win_start(z, dm.Z, dm.kz), ys = win_start(y, dm.H, dm.ky), xs = win_start(x, dm.W, dm.kx);
  for (int jz = zs; jz < zs + dm.kz; ++jz)
    for (int jy = ys; jy < ys + dm.ky; ++jy)
      for (int jx = xs; jx < xs + dm.kx; ++jx) {
        int64_t kj = ((bh * dm.Z + jz) * dm.H + jy) * dm.W + jx;
        load_rot<T, D>(k + kj * D, cs ? cs + (((int64_t)b * dm.H + jy) * dm.W + jx) * (D / 2) : nullptr, 1.f, kv);
        if (opt.qk_norm) rms_normalise<D>(kv, opt.eps);
        float s = 0.f, dp = 0.f;
        const T* vr = v + kj * D;
#pragma unroll
        for (int e = 0; e < D; ++e) {
          s = fmaf(qv[e], kv[e], s);
          dp = fmaf(g[e], ld(vr + e), dp);
        }
        float p = expf(s * dm.scale - L);
        float ds = p * (dp - Di);
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = fmaf(ds, kv[e], acc[e]);
      }
  // dq = R^T (scale * acc), through the norm's Jacobian first when normalising
#pragma unroll
  for (int e = 0; e < D; ++e) acc[e] *= dm.scale;
  if (opt.qk_norm) rms_norm_vjp<D>(acc, qv, rq);
#pragma unroll
  for (int t = 0; t < D / 2; ++t) {
    float a = acc[2 * t], bb = acc[2 * t + 1];
    float c = 1.f, sn = 0.f;
    if (phq) { c = phq[t].x; sn = -phq[t].y; }
    st(dq + qi * D + 2 * t, fmaf(a, c, -bb * sn));
    st(dq + qi * D + 2 * t + 1, fmaf(a, sn, bb * c));
  }
}

// dk_j, dv_j: loop over the queries whose window holds key j (a box of
// contiguous ranges per axis, closed form).
__device__ __forceinline__ void inv_range(int j, int L, int k, int& lo, int& hi) {
  int r = k >> 1;
  hi = (j >= L - k) ? L - 1 : j + r;
  lo = (j < k) ? 0 : j - r;
}

template <typename T, int D>
__global__ void __launch_bounds__(128) na3d_bwd_dkdv_ref_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, const float2* __restrict__ cs,
    const T* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ dvec,
    T* __restrict__ dk, T* __restrict__ dv, Dims dm, BwdOpts opt) {
  int64_t nk = (int64_t)dm.B * dm.heads * dm.Z * dm.H * dm.W;
  int64_t kj = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (kj >= nk) return;
  int b, h, z, y, x;
  split_tok(kj, dm, b, h, z, y, x);
  const int64_t bh = (int64_t)b * dm.heads + h;
  const T* dlo = static_cast<const T*>(opt.dout_lo);
  float kv[D], vv[D], qv[D], ak[D], av[D];
  const float2* phk = cs ? cs + (((int64_t)b * dm.H + y) * dm.W + x) * (D / 2) : nullptr;
  load_rot<T, D>(k + kj * D, phk, 1.f, kv);
  const float rk = opt.qk_norm ? rms_normalise<D>(kv, opt.eps) : 1.f;
#pragma unroll
  for (int e = 0; e < D; ++e) {
    vv[e] = ld(v + kj * D + e);
    ak[e] = 0.f;
    av[e] = 0.f;
  }
  int zlo, zhi, ylo, yhi, xlo, xhi;
  inv_range(z, dm.Z, dm.kz, zlo, zhi);
  inv_range(y, dm.H, dm.ky, ylo, yhi);
  inv_range(x, dm.W, dm.kx, xlo, xhi);
  for (int iz = zlo; iz <= zhi; ++iz)
    for (int iy = ylo; iy <= yhi; ++iy)
      for (int ix = xlo; ix <= xhi; ++ix) {
        int64_t qi = ((bh * dm.Z + iz) * dm.H + iy) * dm.W + ix;
        load_rot<T, D>(q + qi * D, cs ? cs + (((int64_t)b * dm.H + iy) * dm.W + ix) * (D / 2) : nullptr, 1.f, qv);
        if (opt.qk_norm) rms_normalise<D>(qv, opt.eps);
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int e = 0; e < D; ++e) {
          s = fmaf(qv[e], kv[e], s);
          dp = fmaf(ld_g(dout, dlo, qi * D + e), vv[e], dp);
        }
        float p = expf(s * dm.scale - lse[qi]);
        float ds = p * (dp - dvec[qi]);
#pragma unroll
        for (int e = 0; e < D; ++e) {
          av[e] = fmaf(p, ld_g(dout, dlo, qi * D + e), av[e]);
          ak[e] = fmaf(ds, qv[e], ak[e]);
        }
      }
  // dk = R^T (scale * ak), through the norm's Jacobian first when normalising
#pragma unroll
  for (int e = 0; e < D; ++e) ak[e] *= dm.scale;
  if (opt.qk_norm) rms_norm_vjp<D>(ak, kv, rk);
#pragma unroll
  for (int t = 0; t < D / 2; ++t) {
    float a = ak[2 * t], bb = ak[2 * t + 1];
    float c = 1.f, sn = 0.f;
    if (phk) { c = phk[t].x; sn = -phk[t].y; }
    st(dk + kj * D + 2 * t, fmaf(a, c, -bb * sn));
    st(dk + kj * D + 2 * t + 1, fmaf(a, sn, bb * c));
    st(dv + kj * D + 2 * t, av[2 * t]);
    st(dv + kj * D + 2 * t + 1, av[2 * t + 1]);
  }
}

// part: 0 = D = rowsum(dO * O), 1 = dq, 2 = dk and dv
template <typename T, int D>
static void bwd_ref(int part, const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                    const void* v, const float* cs, const void* out, const void* dout, const float* lse,
                    void* dq, void* dk, void* dv, float* dvec, hipStream_t s) {
  Dims dm{d.B, d.heads, d.Z, d.H, d.W, d.kz, d.ky, d.kx, d.scale};
  int64_t n = (int64_t)d.B * d.heads * d.Z * d.H * d.W;
  int threads = 128;
  int blocks = (int)((n + threads - 1) / threads);
  const float2* c2 = reinterpret_cast<const float2*>(cs);
  if (part == 0)
    hipLaunchKernelGGL((na3d_bwd_pre_kernel<T, D>), dim3((int)((n * (D * sizeof(T) / 16) + 255) / 256)),
                       dim3(256), 0, s, static_cast<const T*>(out), static_cast<const T*>(dout), dvec, n);
  else if (part == 1)
    hipLaunchKernelGGL((na3d_bwd_dq_ref_kernel<T, D>), dim3(blocks), dim3(threads), 0, s,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), c2,
                       static_cast<const T*>(dout), lse, dvec, static_cast<T*>(dq), dm, o);
  else
    hipLaunchKernelGGL((na3d_bwd_dkdv_ref_kernel<T, D>), dim3(blocks), dim3(threads), 0, s,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), c2,
                       static_cast<const T*>(dout), lse, dvec, static_cast<T*>(dk), static_cast<T*>(dv),
                       dm, o);
}

void launch_na3d_bwd_ref(int part, const strata_na3d_desc& d, const BwdOpts& o, const void* q,
                         const void* k, const void* v, const float* cs, const void* out,
                         const void* dout, const float* lse, void* dq, void* dk, void* dv,
                         float* dvec, hipStream_t s) {
  if (d.dtype == STRATA_BF16) {
    if (d.head_dim == 32) bwd_ref<uint16_t, 32>(part, d, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
    else if (d.head_dim == 64) bwd_ref<uint16_t, 64>(part, d, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
    else bwd_ref<uint16_t, 128>(part, d, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
  } else {
    if (d.head_dim == 32) bwd_ref<float, 32>(part, d, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
    else if (d.head_dim == 64) bwd_ref<float, 64>(part, d, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
    else bwd_ref<float, 128>(part, d, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
  }
}

}  // namespace strata

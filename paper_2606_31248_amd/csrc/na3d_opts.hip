// Row pass of the attention backward with the sigmoid output gate (App. B.5):
//   D = <dO, out>, and with a = sigmoid(g):  dA = a dO,
//   dgate = (1 - a) dO out per channel, or (1 - a) D for one logit per (token,
//   head); 1 - a is evaluated as sigmoid(-g).
// dA feeds the attention backward in place of dO.  For bf16 it is written as
// two terms, hi = bf16(dA) and lo = bf16(dA - hi), whose sum carries dA to
// ~2^-16 relative: rounding dA to bf16 alone would cost more than a percent of
// the gradients' RMS.  A lane handles one 16-byte piece of a row (8 bf16 or 4
// float32 values); the CPR lanes of a row are consecutive and aligned inside
// the wave and add their partial sums by butterfly exchanges.  Arithmetic in
// float32.
#include "common.h"
#include "kernels.h"

namespace strata {
namespace {

template <typename T>
struct Piece;
template <>
struct Piece<uint16_t> {  // 8 bf16
  static constexpr int E = 8;
  static __device__ __forceinline__ void unpack(const uint4& u, float* f) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  static __device__ __forceinline__ uint4 pack(const float* f) {
    return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                      pack_bf16x2(f[6], f[7]));
  }
  static __device__ __forceinline__ float load1(const uint16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ void store1(uint16_t* p, float v) { *p = f32_to_bf16(v); }
  // remainders f - bf16(f), rounded to bf16
  static __device__ __forceinline__ uint4 pack_lo(const float* f) {
    float r[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = f[i] - bf16_to_f32(f32_to_bf16(f[i]));
    return pack(r);
  }
};
template <>
struct Piece<float> {  // 4 float32
  static constexpr int E = 4;
  static __device__ __forceinline__ void unpack(const uint4& u, float* f) {
    f[0] = __uint_as_float(u.x);
    f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z);
    f[3] = __uint_as_float(u.w);
  }
  static __device__ __forceinline__ uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
  static __device__ __forceinline__ float load1(const float* p) { return *p; }
  static __device__ __forceinline__ void store1(float* p, float v) { *p = v; }
  static __device__ __forceinline__ uint4 pack_lo(const float*) { return make_uint4(0u, 0u, 0u, 0u); }
};

__device__ __forceinline__ float sigm(float g) { return 1.f / (1.f + expf(-g)); }

template <int CPR>
__device__ __forceinline__ float row_sum(float x) {
#pragma unroll
  for (int off = CPR / 2; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

template <typename T, int D>
__global__ void __launch_bounds__(256) gate_prep_kernel(const T* __restrict__ out, const T* __restrict__ dout,
                                                        const T* __restrict__ gate, int gate_dim,
                                                        float* __restrict__ dvec, T* __restrict__ da,
                                                        T* __restrict__ da_lo, T* __restrict__ dgate, int64_t n) {
  using PC = Piece<T>;
  constexpr int E = PC::E, CPR = D / E;
  static_assert(64 % CPR == 0, "a row's lanes must not straddle a wave");
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid / CPR;
  const int c = (int)(gid % CPR);
  const bool live = row < n;
  float o[E], g[E];
  float acc = 0.f;
  if (live) {
    PC::unpack(*reinterpret_cast<const uint4*>(out + row * D + c * E), o);
    PC::unpack(*reinterpret_cast<const uint4*>(dout + row * D + c * E), g);
#pragma unroll
    for (int e = 0; e < E; ++e) acc = fmaf(g[e], o[e], acc);
  }
  const float Dr = row_sum<CPR>(acc);
  if (!live) return;
  if (c == 0) dvec[row] = Dr;
  if (!gate) return;
  float a[E], ra[E];  // sigmoid(g), sigmoid(-g) = 1 - sigmoid(g)
  if (gate_dim == 1) {
    const float gl = PC::load1(gate + row);
    const float s = sigm(gl), rs = sigm(-gl);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      a[e] = s;
      ra[e] = rs;
    }
    if (c == 0) PC::store1(dgate + row, rs * Dr);
  } else {
    float gl[E];
    PC::unpack(*reinterpret_cast<const uint4*>(gate + row * D + c * E), gl);
    float dg[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      a[e] = sigm(gl[e]);
      ra[e] = sigm(-gl[e]);
      dg[e] = ra[e] * g[e] * o[e];
    }
    *reinterpret_cast<uint4*>(dgate + row * D + c * E) = PC::pack(dg);
  }
  float d[E];
#pragma unroll
  for (int e = 0; e < E; ++e) d[e] = a[e] * g[e];
  *reinterpret_cast<uint4*>(da + row * D + c * E) = PC::pack(d);
  if (da_lo) *reinterpret_cast<uint4*>(da_lo + row * D + c * E) = PC::pack_lo(d);
}

int64_t rows(const strata_na3d_desc& d) { return (int64_t)d.B * d.heads * d.Z * d.H * d.W; }

template <typename T, int D>
unsigned blocks_for(int64_t n) {
  constexpr int CPR = D / Piece<T>::E;
  return (unsigned)((n * CPR + 255) / 256);
}

}  // namespace

#define STRATA_DISPATCH_TD(d, F)                       \
  do {                                                 \
    if ((d).dtype == STRATA_BF16) {                    \
      if ((d).head_dim == 32) F(uint16_t, 32);         \
      else if ((d).head_dim == 64) F(uint16_t, 64);    \
      else F(uint16_t, 128);                           \
    } else {                                           \
      if ((d).head_dim == 32) F(float, 32);            \
      else if ((d).head_dim == 64) F(float, 64);       \
      else F(float, 128);                              \
    }                                                  \
  } while (0)

void launch_na3d_bwd_gate_prep(const strata_na3d_desc& d, const NaOpts& o, const void* out,
                               const void* dout, float* dvec, void* da_hi, void* da_lo, void* dgate,
                               hipStream_t s) {
  const int64_t n = rows(d);
#define F(T, D)                                                                                   \
  hipLaunchKernelGGL((gate_prep_kernel<T, D>), dim3(blocks_for<T, D>(n)), dim3(256), 0, s,        \
                     static_cast<const T*>(out), static_cast<const T*>(dout),                    \
                     static_cast<const T*>(o.gate), o.gate_dim, dvec, static_cast<T*>(da_hi),     \
                     static_cast<T*>(da_lo), static_cast<T*>(dgate), n)
  STRATA_DISPATCH_TD(d, F);
#undef F
}

}  // namespace strata

// Tile stitch S = D^-1 P^T W on a regular tiling, and tile extraction P.
//
// The stitch is a deterministic gather: each thread owns VEC consecutive
// channels of one face cell, finds the covering tiles in closed form and
// accumulates them in a fixed order (ascending tile row a, then column b) with
// fused multiply-adds, then divides once.  That order and the precision
// (float32 accumulation for bf16 data, float64 for float32 data) make the
// result reproducible bit for bit.  Streaming, HBM-bound.
#include "common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace strata {

template <typename T>
struct BlendTraits;

template <>
struct BlendTraits<uint16_t> {  // bf16 data, float32 accumulation
  using Acc = float;
  static __device__ __forceinline__ Acc load(const uint16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ uint16_t store(Acc v) { return f32_to_bf16(v); }
  static __device__ __forceinline__ Acc fma_(Acc a, Acc b, Acc c) { return __builtin_fmaf(a, b, c); }
};

template <>
struct BlendTraits<float> {  // float32 data, float64 accumulation
  using Acc = double;
  static __device__ __forceinline__ Acc load(const float* p) { return (double)*p; }
  static __device__ __forceinline__ float store(Acc v) { return (float)v; }
  static __device__ __forceinline__ Acc fma_(Acc a, Acc b, Acc c) { return __builtin_fma(a, b, c); }
};

// Closed-form range of tiles along one axis covering face position y:
// a in [ceil((y - Ht + 1) / s), floor(y / s)] clipped to [0, n).
__device__ __forceinline__ void cover_range(int y, int Ht, int s, int n, int* lo, int* hi) {
  int num = y - Ht + 1;
  int a0 = num <= 0 ? 0 : (num + s - 1) / s;
  int a1 = y / s;
  *lo = a0;
  *hi = a1 < n - 1 ? a1 : n - 1;
}

// One block covers BLK consecutive (x, channel-vector) items of one face row
// (p, y); the covering tile rows follow from y once per block.  CV > 0: the
// number of channel vectors per cell is known at compile time.
template <typename T, int VEC, int CV>
__global__ void __launch_bounds__(256) tile_blend_kernel(const T* __restrict__ tiles, int nty, int ntx, int P,
                                                         int Ht, int Wt, int C, int sy, int sx,
                                                         const float* __restrict__ window,
                                                         T* __restrict__ out, int Hf, int Wf, int bpr) {
  using Tr = BlendTraits<T>;
  using Acc = typename Tr::Acc;
  const int cv = CV > 0 ? CV : C / VEC;
  const int row = blockIdx.x / bpr;                 // p * Hf + y
  const int j = (blockIdx.x - row * bpr) * blockDim.x + threadIdx.x;
  if (j >= Wf * cv) return;
  const int y = row % Hf, p = row / Hf;
  const int x = j / cv, c0 = (j - x * cv) * VEC;
  int alo, ahi, blo, bhi;
  cover_range(y, Ht, sy, nty, &alo, &ahi);
  cover_range(x, Wt, sx, ntx, &blo, &bhi);
  Acc acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = (Acc)0;
  Acc dsum = (Acc)0;
  const int64_t tile_elems = (int64_t)P * Ht * Wt * C;
  for (int a = alo; a <= ahi; ++a) {
    const int ly = y - a * sy;
    const T* trow = tiles + (int64_t)a * ntx * tile_elems + ((int64_t)p * Ht + ly) * Wt * C + c0;
    for (int b = blo; b <= bhi; ++b) {
      const int lx = x - b * sx;
      const Acc w = (Acc)window[ly * Wt + lx];
      const T* src = trow + b * tile_elems + lx * C;
      T vals[VEC];
      if constexpr (VEC * sizeof(T) == 16) {
        *reinterpret_cast<uint4*>(vals) = *reinterpret_cast<const uint4*>(src);
      } else {
#pragma unroll
        for (int v = 0; v < VEC; ++v) vals[v] = src[v];
      }
#pragma unroll
      for (int v = 0; v < VEC; ++v) acc[v] = Tr::fma_(w, Tr::load(&vals[v]), acc[v]);
      dsum = dsum + w;
    }
  }
  T res[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) res[v] = Tr::store(dsum == (Acc)0 ? (Acc)0 : acc[v] / dsum);
  T* dst = out + ((int64_t)row * Wf + x) * C + c0;
  if constexpr (VEC * sizeof(T) == 16) {
    *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(res);
  } else {
#pragma unroll
    for (int v = 0; v < VEC; ++v) dst[v] = res[v];
  }
}

template <typename T, int VEC, int CV>
static void blend_launch(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                         int sx, const float* window, void* out, int Hf, int Wf, hipStream_t s) {
  const int threads = 256;
  const int64_t per_row = (int64_t)Wf * (C / VEC);
  const int bpr = (int)((per_row + threads - 1) / threads);
  const int64_t blocks = (int64_t)P * Hf * bpr;
  hipLaunchKernelGGL((tile_blend_kernel<T, VEC, CV>), dim3((unsigned)blocks), dim3(threads), 0, s,
                     static_cast<const T*>(tiles), nty, ntx, P, Ht, Wt, C, sy, sx, window,
                     static_cast<T*>(out), Hf, Wf, bpr);
}

void launch_tile_blend(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                       int sx, const float* window, void* out, int Hf, int Wf, strata_dtype dt,
                       hipStream_t s) {
  if (dt == STRATA_BF16) {
    if (C == 64)
      blend_launch<uint16_t, 8, 8>(tiles, nty, ntx, P, Ht, Wt, C, sy, sx, window, out, Hf, Wf, s);
    else if (C % 8 == 0)
      blend_launch<uint16_t, 8, 0>(tiles, nty, ntx, P, Ht, Wt, C, sy, sx, window, out, Hf, Wf, s);
    else
      blend_launch<uint16_t, 1, 0>(tiles, nty, ntx, P, Ht, Wt, C, sy, sx, window, out, Hf, Wf, s);
  } else {
    if (C % 4 == 0)
      blend_launch<float, 4, 0>(tiles, nty, ntx, P, Ht, Wt, C, sy, sx, window, out, Hf, Wf, s);
    else
      blend_launch<float, 1, 0>(tiles, nty, ntx, P, Ht, Wt, C, sy, sx, window, out, Hf, Wf, s);
  }
}

// ---- extraction: one thread per 16 bytes (or one element) of a tile row -----
template <typename T, int VEC>
__global__ void tile_extract_kernel(const T* __restrict__ face, int ntx, int P, int Ht, int Wt,
                                    int C, int sy, int sx, int Hf, int Wf, T* __restrict__ tiles,
                                    int64_t total) {
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int cv = C / VEC;
  int c0 = (int)(idx % cv) * VEC;
  int64_t r = idx / cv;
  int j = (int)(r % Wt); r /= Wt;
  int i = (int)(r % Ht); r /= Ht;
  int p = (int)(r % P); r /= P;
  int64_t t = r;
  int a = (int)(t / ntx), b = (int)(t % ntx);
  const T* src = face + ((((int64_t)p * Hf + (a * sy + i)) * Wf + (b * sx + j)) * C + c0);
  T* dst = tiles + (idx * VEC);
  if constexpr (VEC * sizeof(T) == 16) {
    *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
  } else {
#pragma unroll
    for (int v = 0; v < VEC; ++v) dst[v] = src[v];
  }
}

template <typename T, int VEC>
static void extract_launch(const void* face, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                           int sx, int Hf, int Wf, void* tiles, hipStream_t s) {
  int64_t total = (int64_t)nty * ntx * P * Ht * Wt * (C / VEC);
  int threads = 256;
  int blocks = (int)((total + threads - 1) / threads);
  hipLaunchKernelGGL((tile_extract_kernel<T, VEC>), dim3(blocks), dim3(threads), 0, s,
                     static_cast<const T*>(face), ntx, P, Ht, Wt, C, sy, sx, Hf, Wf,
                     static_cast<T*>(tiles), total);
}

void launch_tile_extract(const void* face, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                         int sx, int Hf, int Wf, void* tiles, strata_dtype dt, hipStream_t s) {
  if (dt == STRATA_BF16) {
    if (C % 8 == 0)
      extract_launch<uint16_t, 8>(face, nty, ntx, P, Ht, Wt, C, sy, sx, Hf, Wf, tiles, s);
    else
      extract_launch<uint16_t, 1>(face, nty, ntx, P, Ht, Wt, C, sy, sx, Hf, Wf, tiles, s);
  } else {
    if (C % 4 == 0)
      extract_launch<float, 4>(face, nty, ntx, P, Ht, Wt, C, sy, sx, Hf, Wf, tiles, s);
    else
      extract_launch<float, 1>(face, nty, ntx, P, Ht, Wt, C, sy, sx, Hf, Wf, tiles, s);
  }
}

}  // namespace strata

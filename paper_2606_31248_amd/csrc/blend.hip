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

// bf16 stitch for channel counts C % 8 == 0 when no face position is covered
// by more than two tiles along an axis (Ht <= 2 stride_y, Wt <= 2 stride_x).
// Each thread handles ITEMS cells x 8 channels of one face row and issues all
// its loads (up to 2 x 2 covering tiles per cell, predicated) before any
// arithmetic, which keeps enough bytes in flight per CU to stream at HBM rate.
// Every tile element is read once and every face element written once, so
// both go through non-temporal (streaming) accesses.
// Same operation order as the plain kernel: tiles in ascending (a, b), fmaf,
// the weight sum from 0, one correctly rounded division (skipped when the sum
// is exactly 1, where it is the identity), round to nearest even.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// ITEMS cells x 8 channels of face row (p, y), whose covering tile rows are
// [alo, ahi]; item(k, x, c0) names the k-th cell of this thread (false: none).
template <int ITEMS, typename Item>
__device__ __forceinline__ void stitch_cells_bf16(const uint16_t* __restrict__ tiles, int ntx, int P, int Ht,
                                                  int Wt, int C, int sy, int sx, const float* __restrict__ window,
                                                  uint16_t* __restrict__ out_row, int y, int p, int alo, int ahi,
                                                  Item item) {
  const int64_t tile_elems = (int64_t)P * Ht * Wt * C;
  uint4 val[ITEMS][2][2];
  float wt[ITEMS][2][2];
  bool ok[ITEMS][2][2];
  bool live[ITEMS];
  int xs[ITEMS], cs[ITEMS];
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    int x = 0, c0 = 0;
    live[k] = item(k, x, c0);
    xs[k] = x;
    cs[k] = c0;
    int blo, bhi;
    cover_range(x, Wt, sx, ntx, &blo, &bhi);
#pragma unroll
    for (int ia = 0; ia < 2; ++ia) {
#pragma unroll
      for (int ib = 0; ib < 2; ++ib) {
        const int a = alo + ia, b = blo + ib;
        ok[k][ia][ib] = live[k] && a <= ahi && b <= bhi;
        val[k][ia][ib] = make_uint4(0u, 0u, 0u, 0u);
        wt[k][ia][ib] = 0.f;
        if (ok[k][ia][ib]) {
          const int ly = y - a * sy, lx = x - b * sx;
          const uint16_t* src =
              tiles + ((int64_t)a * ntx + b) * tile_elems + (((int64_t)p * Ht + ly) * Wt + lx) * C + c0;
          const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
          val[k][ia][ib] = make_uint4(t.x, t.y, t.z, t.w);
          wt[k][ia][ib] = window[ly * Wt + lx];
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    if (!live[k]) continue;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float dsum = 0.f;
#pragma unroll
    for (int ia = 0; ia < 2; ++ia) {
#pragma unroll
      for (int ib = 0; ib < 2; ++ib) {
        if (!ok[k][ia][ib]) continue;
        const float w = wt[k][ia][ib];
        const uint32_t wv[4] = {val[k][ia][ib].x, val[k][ia][ib].y, val[k][ia][ib].z, val[k][ia][ib].w};
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          acc[2 * v] = __builtin_fmaf(w, __uint_as_float(wv[v] << 16), acc[2 * v]);
          acc[2 * v + 1] = __builtin_fmaf(w, __uint_as_float(wv[v] & 0xFFFF0000u), acc[2 * v + 1]);
        }
        dsum = dsum + w;
      }
    }
    if (dsum != 1.f) {
#pragma unroll
      for (int v = 0; v < 8; ++v) acc[v] = dsum == 0.f ? 0.f : acc[v] / dsum;
    }
    uint32_t r[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) r[v] = pack_bf16x2(acc[2 * v], acc[2 * v + 1]);
    __builtin_nontemporal_store(u32x4{r[0], r[1], r[2], r[3]},
                                reinterpret_cast<u32x4*>(out_row + (int64_t)xs[k] * C + cs[k]));
  }
}

template <int ITEMS>
__global__ void __launch_bounds__(256) tile_blend_bf16_kernel(const uint16_t* __restrict__ tiles, int nty, int ntx,
                                                              int P, int Ht, int Wt, int C, int sy, int sx,
                                                              const float* __restrict__ window,
                                                              uint16_t* __restrict__ out, int Hf, int Wf, int bpr) {
  const int cv = C >> 3;
  const int row = blockIdx.x / bpr;  // p * Hf + y
  const int jb = (blockIdx.x - row * bpr) * (256 * ITEMS) + threadIdx.x;
  const int y = row % Hf, p = row / Hf;
  int alo, ahi;
  cover_range(y, Ht, sy, nty, &alo, &ahi);
  const int per_row = Wf * cv;
  stitch_cells_bf16<ITEMS>(tiles, ntx, P, Ht, Wt, C, sy, sx, window, out + (int64_t)row * Wf * C, y, p, alo, ahi,
                           [&](int k, int& x, int& c0) {
                             const int j = jb + k * 256;
                             if (j >= per_row) return false;
                             x = j / cv;
                             c0 = (j - x * cv) * 8;
                             return true;
                           });
}

// The same stitch restricted to the cells that two or more tiles cover, for a
// tiling whose tiles cover the face with sy <= Ht <= 2 sy, sx <= Wt <= 2 sx:
// one block per face row (p, y); a row inside a y overlap [a sy, (a-1) sy + Ht)
// is stitched whole, any other row only at the x overlaps [b sx, (b-1) sx + Wt).
// The cells one tile covers alone are left as they are.
template <int ITEMS>
__global__ void __launch_bounds__(256) tile_blend_overlap_bf16_kernel(const uint16_t* __restrict__ tiles, int nty,
                                                                      int ntx, int P, int Ht, int Wt, int C, int sy,
                                                                      int sx, const float* __restrict__ window,
                                                                      uint16_t* __restrict__ out, int Hf, int Wf) {
  const int cv = C >> 3;
  const int row = blockIdx.x;  // p * Hf + y
  const int y = row % Hf, p = row / Hf;
  int alo, ahi;
  cover_range(y, Ht, sy, nty, &alo, &ahi);
  const bool whole = alo < ahi;
  const int ovx = Wt - sx;
  const int nitems = (whole ? Wf : (ntx - 1) * ovx) * cv;
  uint16_t* const out_row = out + (int64_t)row * Wf * C;
  for (int j0 = 0; j0 < nitems; j0 += 256 * ITEMS) {
    stitch_cells_bf16<ITEMS>(tiles, ntx, P, Ht, Wt, C, sy, sx, window, out_row, y, p, alo, ahi,
                             [&](int k, int& x, int& c0) {
                               const int j = j0 + k * 256 + (int)threadIdx.x;
                               if (j >= nitems) return false;
                               const int cell = j / cv;
                               c0 = (j - cell * cv) * 8;
                               x = whole ? cell : (cell / ovx + 1) * sx + cell % ovx;
                               return true;
                             });
  }
}

void launch_tile_blend_overlap(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                               int sx, const float* window, void* out, int Hf, int Wf, hipStream_t s) {
  const int64_t blocks = (int64_t)P * Hf;
  hipLaunchKernelGGL((tile_blend_overlap_bf16_kernel<2>), dim3((unsigned)blocks), dim3(256), 0, s,
                     static_cast<const uint16_t*>(tiles), nty, ntx, P, Ht, Wt, C, sy, sx, window,
                     static_cast<uint16_t*>(out), Hf, Wf);
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
    if (C % 8 == 0 && Ht <= 2 * sy && Wt <= 2 * sx) {
      constexpr int kItems = 2;
      const int64_t per_row = (int64_t)Wf * (C / 8);
      const int bpr = (int)((per_row + 256 * kItems - 1) / (256 * kItems));
      const int64_t blocks = (int64_t)P * Hf * bpr;
      hipLaunchKernelGGL((tile_blend_bf16_kernel<kItems>), dim3((unsigned)blocks), dim3(256), 0, s,
                         static_cast<const uint16_t*>(tiles), nty, ntx, P, Ht, Wt, C, sy, sx, window,
                         static_cast<uint16_t*>(out), Hf, Wf, bpr);
    } else if (C == 64)
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

// Vectorised extraction: one block per tile row (t, p, i), its threads over
// the row's Wt C / VEC 16-byte pieces, which sit contiguously in the face row
// (a sy + i) from column b sx on.  The row indices are block-uniform.
template <typename T, int VEC>
__global__ void __launch_bounds__(256) tile_extract_rows_kernel(const T* __restrict__ face, int ntx, int P, int Ht,
                                                                int Wt, int C, int sy, int sx, int Hf, int Wf,
                                                                T* __restrict__ tiles) {
  const int row = blockIdx.x;  // (t * P + p) * Ht + i
  const int i = row % Ht;
  const int tp = row / Ht;
  const int p = tp % P, t = tp / P;
  const int a = t / ntx, b = t - a * ntx;
  const int n = Wt * C / VEC;
  const uint4* src =
      reinterpret_cast<const uint4*>(face + (((int64_t)p * Hf + (a * sy + i)) * Wf + (int64_t)b * sx) * C);
  uint4* dst = reinterpret_cast<uint4*>(tiles + (int64_t)row * Wt * C);
  for (int j = threadIdx.x; j < n; j += blockDim.x) dst[j] = src[j];
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
  const int64_t rows = (int64_t)nty * ntx * P * Ht;
  const int vec = dt == STRATA_BF16 ? 8 : 4;
  if (C % vec == 0 && rows < ((int64_t)1 << 31) && (int64_t)Wt * C < ((int64_t)1 << 31)) {
    if (dt == STRATA_BF16)
      hipLaunchKernelGGL((tile_extract_rows_kernel<uint16_t, 8>), dim3((unsigned)rows), dim3(256), 0, s,
                         static_cast<const uint16_t*>(face), ntx, P, Ht, Wt, C, sy, sx, Hf, Wf,
                         static_cast<uint16_t*>(tiles));
    else
      hipLaunchKernelGGL((tile_extract_rows_kernel<float, 4>), dim3((unsigned)rows), dim3(256), 0, s,
                         static_cast<const float*>(face), ntx, P, Ht, Wt, C, sy, sx, Hf, Wf,
                         static_cast<float*>(tiles));
    return;
  }
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

// ---- Kaiser-Bessel-derived blend window (App. F) -----------------------------
// Per axis: 1 in the interior, over `overlap` cells at each end the rising half
// of the KBD window of length 2*overlap, w[n] = sqrt(sum_{j<=n} k_j / sum_j k_j)
// with the Kaiser weights k_j = I0(beta sqrt(1 - (2j/overlap - 1)^2)),
// j = 0..overlap; the 2D window is the product of the axes.  I0 by its power
// series sum_m ((x/2)^(2m) / (m!)^2), summed until the terms stop changing the
// float64 sum; everything in float64, rounded to float32 once.
__device__ double bessel_i0(double x) {
  const double q = 0.25 * x * x;
  double term = 1.0, sum = 1.0;
  for (int m = 1; m < 500; ++m) {
    term *= q / ((double)m * (double)m);
    const double next = sum + term;
    if (next == sum) break;
    sum = next;
  }
  return sum;
}

__device__ double kbd_rise(int n, int overlap, double beta) {
  double part = 0.0, total = 0.0;
  for (int j = 0; j <= overlap; ++j) {
    const double r = 2.0 * (double)j / (double)overlap - 1.0;
    const double k = bessel_i0(beta * sqrt(fmax(0.0, 1.0 - r * r)));
    total += k;
    if (j <= n) part += k;
  }
  return sqrt(part / total);
}

__device__ double kbd_axis(int i, int L, int overlap, double beta) {
  double w = 1.0;
  if (i < overlap) w = fmin(w, kbd_rise(i, overlap, beta));
  if (i >= L - overlap) w = fmin(w, kbd_rise(L - 1 - i, overlap, beta));
  return w;
}

__global__ void kbd_window_kernel(int Ht, int Wt, int overlap, double beta, float* __restrict__ window) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= Ht * Wt) return;
  const int y = idx / Wt, x = idx % Wt;
  window[idx] = (float)(kbd_axis(y, Ht, overlap, beta) * kbd_axis(x, Wt, overlap, beta));
}

void launch_kbd_window(int Ht, int Wt, int overlap, double beta, float* window, hipStream_t s) {
  const int n = Ht * Wt;
  hipLaunchKernelGGL(kbd_window_kernel, dim3((n + 255) / 256), dim3(256), 0, s, Ht, Wt, overlap, beta, window);
}

}  // namespace strata

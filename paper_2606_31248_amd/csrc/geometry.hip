// Window indexing (integer) and stereographic tile coordinates (float64).
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace strata {

// ---- one axis of the border-clamped window ----------------------------------
// starts[i] = clamp(i - r, 0, L - k); the queries whose window holds j form the
// contiguous range [qlo, qhi] (start() is non-decreasing):
//   qhi = L - 1 if j >= L - k else j + r;   qlo = 0 if j < k else j - r.
__global__ void axis_index_kernel(int L, int k, int32_t* starts, int32_t* qlo, int32_t* qhi) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= L) return;
  int r = k >> 1;
  starts[i] = win_start(i, L, k);
  qhi[i] = (i >= L - k) ? L - 1 : i + r;
  qlo[i] = (i < k) ? 0 : i - r;
}

void launch_axis_index(int L, int k, int32_t* starts, int32_t* qlo, int32_t* qhi, hipStream_t s) {
  int threads = 256;
  int blocks = (L + threads - 1) / threads;
  hipLaunchKernelGGL(axis_index_kernel, dim3(blocks), dim3(threads), 0, s, L, k, starts, qlo, qhi);
}

// ---- stereographic coordinates (Eq. 1) ---------------------------------------
// Equiangular angle of the centre of patch t along one face axis.
__device__ __forceinline__ double patch_angle(int t, int patch, double step) {
  return -0.25 * M_PI + ((double)patch * (double)t + 0.5 * (double)patch) * step;
}

// (lat, lon) of the cube point of face f at angles (alpha: columns, beta: rows).
__device__ void face_latlon(int f, double alpha, double beta, double* lat, double* lon) {
  double a = tan(alpha), c = tan(beta);
  double X, Y, Zc;
  switch (f) {
    case 0: X = 1.0; Y = a; Zc = c; break;
    case 1: X = -a; Y = 1.0; Zc = c; break;
    case 2: X = -1.0; Y = -a; Zc = c; break;
    case 3: X = a; Y = -1.0; Zc = c; break;
    case 4: X = -c; Y = a; Zc = 1.0; break;
    default: X = c; Y = a; Zc = -1.0; break;
  }
  *lat = atan2(Zc, hypot(X, Y));
  *lon = atan2(Y, X);
}

__global__ void stereo_coords_kernel(const int32_t* __restrict__ face, const int32_t* __restrict__ oy,
                                     const int32_t* __restrict__ ox, int B, int H, int W,
                                     int face_cells, int patch, double l_scale,
                                     float* __restrict__ coords) {
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * H * W) return;
  int x = (int)(idx % W);
  int y = (int)((idx / W) % H);
  int b = (int)(idx / ((int64_t)W * H));
  const double step = 0.5 * M_PI / (double)face_cells;
  int f = face[b], y0 = oy[b], x0 = ox[b];
  double beta = patch_angle(y0 + y, patch, step);
  double alpha = patch_angle(x0 + x, patch, step);
  double beta_c = 0.5 * (patch_angle(y0, patch, step) + patch_angle(y0 + H - 1, patch, step));
  double alpha_c = 0.5 * (patch_angle(x0, patch, step) + patch_angle(x0 + W - 1, patch, step));
  double lat, lon, lat0, lon0;
  face_latlon(f, alpha, beta, &lat, &lon);
  face_latlon(f, alpha_c, beta_c, &lat0, &lon0);
  double dl = lon - lon0;
  double sl, cl, sp, cp, sp0, cp0;
  sincos(dl, &sl, &cl);
  sincos(lat, &sp, &cp);
  sincos(lat0, &sp0, &cp0);
  double cos_c = sp0 * sp + cp0 * cp * cl;
  double kk = 2.0 / (1.0 + cos_c);
  double xe = (kk / l_scale) * cp * sl;
  double yn = (kk / l_scale) * (cp0 * sp - sp0 * cp * cl);
  coords[2 * idx + 0] = (float)xe;
  coords[2 * idx + 1] = (float)yn;
}

void launch_stereo_coords(const int32_t* face, const int32_t* oy, const int32_t* ox, int B, int H,
                          int W, int face_cells, int patch, double l_scale, float* coords,
                          hipStream_t s) {
  int64_t n = (int64_t)B * H * W;
  int threads = 256;
  int blocks = (int)((n + threads - 1) / threads);
  hipLaunchKernelGGL(stereo_coords_kernel, dim3(blocks), dim3(threads), 0, s, face, oy, ox, B, H, W,
                     face_cells, patch, l_scale, coords);
}

// ---- wind vectors into the tile-centre frame (Sec. 3.3, Eq. 2) ----------------
// With v = U e + V n at (lat, lon) and the centre frame (e0, n0, r0), the
// tangential projection leaves the components unchanged (e0 and n0 are
// orthogonal to r0), so per cell (U_loc, V_loc) = M (U, V) with, for
// dl = lon - lon0,
//   M = [ e.e0  n.e0 ] = [ cos dl                 -sin lat sin dl                         ]
//       [ e.n0  n.n0 ]   [ sin lat0 sin dl          sin lat sin lat0 cos dl + cos lat cos lat0 ]
// computed once per cell and applied to every plane: float32 geometry and
// arithmetic for bf16 data (errors ~1e-7 against bf16's 2^-9), float64 for
// float32 data.
// cube point of face f at angles (alpha, beta) (columns, rows), not normalised
template <typename F>
__device__ __forceinline__ void cube_point_of(int f, F a, F c, F* X, F* Y, F* Zc) {
  switch (f) {
    case 0: *X = F(1); *Y = a; *Zc = c; break;
    case 1: *X = -a; *Y = F(1); *Zc = c; break;
    case 2: *X = F(-1); *Y = -a; *Zc = c; break;
    case 3: *X = a; *Y = F(-1); *Zc = c; break;
    case 4: *X = -c; *Y = a; *Zc = F(1); break;
    default: *X = c; *Y = a; *Zc = F(-1); break;
  }
}
__device__ __forceinline__ void face_point_f(int f, float alpha, float beta, float* X, float* Y, float* Zc) {
  cube_point_of<float>(f, tanf(alpha), tanf(beta), X, Y, Zc);
}
__device__ __forceinline__ void face_point(int f, double alpha, double beta, double* X, double* Y, double* Zc) {
  cube_point_of<double>(f, tan(alpha), tan(beta), X, Y, Zc);
}

// one (U, V) pair of one plane: two bf16 in a word, or two float32
template <typename T>
struct WindPair {
  using type = typename std::conditional<sizeof(T) == 2, uint32_t, float2>::type;
};

template <typename T>
__global__ void wind_tile_frame_kernel(const T* __restrict__ field, int face, int n_cells, int ntx, int P,
                                       int Ht, int Wt, int sy, int sx, int64_t ncells_out,
                                       T* __restrict__ tiles) {
  using Pair = typename WindPair<T>::type;
  constexpr int kBatch = 8;  // planes whose loads are in flight while the frame is computed
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= ncells_out) return;
  const int j = (int)(idx % Wt);
  const int i = (int)((idx / Wt) % Ht);
  const int64_t t = idx / ((int64_t)Wt * Ht);
  const int a = (int)(t / ntx), b = (int)(t % ntx);
  const int fy = a * sy + i, fx = b * sx + j;
  const int64_t plane_in = (int64_t)n_cells * n_cells, plane_out = (int64_t)Ht * Wt;
  const Pair* src = reinterpret_cast<const Pair*>(field) + (int64_t)fy * n_cells + fx;
  Pair* dst = reinterpret_cast<Pair*>(tiles) + (t * P) * plane_out + (int64_t)i * Wt + j;
  // the first planes' loads go out before the geometry
  Pair w[kBatch];
#pragma unroll
  for (int u = 0; u < kBatch; ++u)
    if (u < P) w[u] = src[u * plane_in];
  // the frame products straight from the two cube points (no angles): with
  // rho = |(X, Y)| and r = |(X, Y, Z)|, sin lat = Z / r, cos lat = rho / r,
  // cos dl = (X X0 + Y Y0) / (rho rho0), sin dl = (Y X0 - X Y0) / (rho rho0);
  // on the polar axis (rho = 0) the longitude is atan2's of the signed zeros:
  // 0 for X = +0, pi for X = -0 (face 4's pole has X = -0)
  double m00, m01, m10, m11;
  if constexpr (sizeof(T) == 2) {  // geometry in float32
    const float step = 0.5f * (float)M_PI / (float)n_cells;
    auto ang = [&](int c) { return -0.25f * (float)M_PI + ((float)c + 0.5f) * step; };
    float X, Y, Zc, X0, Y0, Z0;
    face_point_f(face, ang(fx), ang(fy), &X, &Y, &Zc);
    face_point_f(face, 0.5f * (ang(b * sx) + ang(b * sx + Wt - 1)), 0.5f * (ang(a * sy) + ang(a * sy + Ht - 1)),
                 &X0, &Y0, &Z0);
    const float rho2 = fmaf(X, X, Y * Y), rho02 = fmaf(X0, X0, Y0 * Y0);
    const float irho = rho2 > 0.f ? __frsqrt_rn(rho2) : 0.f, irho0 = rho02 > 0.f ? __frsqrt_rn(rho02) : 0.f;
    const float ir = __frsqrt_rn(fmaf(Zc, Zc, rho2)), ir0 = __frsqrt_rn(fmaf(Z0, Z0, rho02));
    const float ex = rho2 > 0.f ? X * irho : copysignf(1.f, X), ey = rho2 > 0.f ? Y * irho : 0.f;  // (cos, sin) lon
    const float ex0 = rho02 > 0.f ? X0 * irho0 : copysignf(1.f, X0), ey0 = rho02 > 0.f ? Y0 * irho0 : 0.f;
    const float cd = fmaf(ex, ex0, ey * ey0), sd = fmaf(ey, ex0, -ex * ey0);
    const float sp = Zc * ir, cp = rho2 * irho * ir, sp0 = Z0 * ir0, cp0 = rho02 * irho0 * ir0;
    m00 = cd;
    m01 = -sp * sd;
    m10 = sp0 * sd;
    m11 = fmaf(sp * sp0, cd, cp * cp0);
  } else {
    const double step = 0.5 * M_PI / (double)n_cells;
    auto ang = [&](int c) { return -0.25 * M_PI + ((double)c + 0.5) * step; };
    double X, Y, Zc, X0, Y0, Z0;
    face_point(face, ang(fx), ang(fy), &X, &Y, &Zc);
    face_point(face, 0.5 * (ang(b * sx) + ang(b * sx + Wt - 1)), 0.5 * (ang(a * sy) + ang(a * sy + Ht - 1)), &X0,
               &Y0, &Z0);
    const double rho = sqrt(X * X + Y * Y), rho0 = sqrt(X0 * X0 + Y0 * Y0);
    const double r = sqrt(rho * rho + Zc * Zc), r0 = sqrt(rho0 * rho0 + Z0 * Z0);
    const double ex = rho > 0.0 ? X / rho : copysign(1.0, X), ey = rho > 0.0 ? Y / rho : 0.0;
    const double ex0 = rho0 > 0.0 ? X0 / rho0 : copysign(1.0, X0), ey0 = rho0 > 0.0 ? Y0 / rho0 : 0.0;
    const double cd = ex * ex0 + ey * ey0, sd = ey * ex0 - ex * ey0;
    const double sp = Zc / r, cp = rho / r, sp0 = Z0 / r0, cp0 = rho0 / r0;
    m00 = cd;
    m01 = -sp * sd;
    m10 = sp0 * sd;
    m11 = sp * sp0 * cd + cp * cp0;
  }
  auto rotate = [&](Pair x) {
    if constexpr (sizeof(T) == 2) {
      const float u = bf16_to_f32((uint16_t)(x & 0xFFFFu)), v = bf16_to_f32((uint16_t)(x >> 16));
      return pack_bf16x2(fmaf((float)m00, u, (float)m01 * v), fmaf((float)m10, u, (float)m11 * v));
    } else {
      const double u = x.x, v = x.y;
      return make_float2((float)fma(m00, u, m01 * v), (float)fma(m10, u, m11 * v));
    }
  };
#pragma unroll
  for (int u = 0; u < kBatch; ++u)
    if (u < P) dst[u * plane_out] = rotate(w[u]);
  for (int p = kBatch; p < P; ++p) dst[p * plane_out] = rotate(src[p * plane_in]);
}

void launch_wind_tile_frame(const void* field, int face, int n_cells, int nty, int ntx, int P, int Ht, int Wt,
                            int sy, int sx, void* tiles, strata_dtype dt, hipStream_t s) {
  const int64_t n = (int64_t)nty * ntx * Ht * Wt;
  const int threads = 256;
  const unsigned blocks = (unsigned)((n + threads - 1) / threads);
  if (dt == STRATA_BF16)
    hipLaunchKernelGGL((wind_tile_frame_kernel<uint16_t>), dim3(blocks), dim3(threads), 0, s,
                       static_cast<const uint16_t*>(field), face, n_cells, ntx, P, Ht, Wt, sy, sx, n,
                       static_cast<uint16_t*>(tiles));
  else
    hipLaunchKernelGGL((wind_tile_frame_kernel<float>), dim3(blocks), dim3(threads), 0, s,
                       static_cast<const float*>(field), face, n_cells, ntx, P, Ht, Wt, sy, sx, n,
                       static_cast<float*>(tiles));
}

}  // namespace strata

// Window indexing (integer) and stereographic tile coordinates (float64).
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

}  // namespace strata

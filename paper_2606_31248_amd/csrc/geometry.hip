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
// (lat, lon) of the cube point in float32 (the bf16 path: errors ~1e-7, far
// below bf16's 2^-9).
__device__ void face_latlon_f(int f, float alpha, float beta, float* lat, float* lon) {
  const float a = tanf(alpha), c = tanf(beta);
  float X, Y, Zc;
  switch (f) {
    case 0: X = 1.f; Y = a; Zc = c; break;
    case 1: X = -a; Y = 1.f; Zc = c; break;
    case 2: X = -1.f; Y = -a; Zc = c; break;
    case 3: X = a; Y = -1.f; Zc = c; break;
    case 4: X = -c; Y = a; Zc = 1.f; break;
    default: X = c; Y = a; Zc = -1.f; break;
  }
  *lat = atan2f(Zc, hypotf(X, Y));
  *lon = atan2f(Y, X);
}

template <typename T>
__global__ void wind_tile_frame_kernel(const T* __restrict__ field, int face, int n_cells, int ntx, int P,
                                       int Ht, int Wt, int sy, int sx, int64_t ncells_out,
                                       T* __restrict__ tiles) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= ncells_out) return;
  const int j = (int)(idx % Wt);
  const int i = (int)((idx / Wt) % Ht);
  const int64_t t = idx / ((int64_t)Wt * Ht);
  const int a = (int)(t / ntx), b = (int)(t % ntx);
  const int fy = a * sy + i, fx = b * sx + j;
  double m00, m01, m10, m11;
  if constexpr (sizeof(T) == 2) {  // geometry in float32
    const float step = 0.5f * (float)M_PI / (float)n_cells;
    auto ang = [&](int c) { return -0.25f * (float)M_PI + ((float)c + 0.5f) * step; };
    float lat, lon, lat0, lon0, sd, cd, sp, cp, sp0, cp0;
    face_latlon_f(face, ang(fx), ang(fy), &lat, &lon);
    face_latlon_f(face, 0.5f * (ang(b * sx) + ang(b * sx + Wt - 1)), 0.5f * (ang(a * sy) + ang(a * sy + Ht - 1)),
                  &lat0, &lon0);
    sincosf(lon - lon0, &sd, &cd);
    sincosf(lat, &sp, &cp);
    sincosf(lat0, &sp0, &cp0);
    m00 = cd;
    m01 = -sp * sd;
    m10 = sp0 * sd;
    m11 = fmaf(sp * sp0, cd, cp * cp0);
  } else {
    const double step = 0.5 * M_PI / (double)n_cells;
    auto ang = [&](int c) { return -0.25 * M_PI + ((double)c + 0.5) * step; };
    double lat, lon, lat0, lon0;
    face_latlon(face, ang(fx), ang(fy), &lat, &lon);
    face_latlon(face, 0.5 * (ang(b * sx) + ang(b * sx + Wt - 1)), 0.5 * (ang(a * sy) + ang(a * sy + Ht - 1)),
                &lat0, &lon0);
    double sd, cd, sp, cp, sp0, cp0;
    sincos(lon - lon0, &sd, &cd);
    sincos(lat, &sp, &cp);
    sincos(lat0, &sp0, &cp0);
    m00 = cd;
    m01 = -sp * sd;
    m10 = sp0 * sd;
    m11 = sp * sp0 * cd + cp * cp0;
  }
  const int64_t plane_in = (int64_t)n_cells * n_cells, plane_out = (int64_t)Ht * Wt;
  const T* src = field + 2 * ((int64_t)fy * n_cells + fx);
  T* dst = tiles + 2 * ((t * P) * plane_out + (int64_t)i * Wt + j);
  for (int p = 0; p < P; ++p) {
    const T* s2 = src + 2 * p * plane_in;
    T* d2 = dst + 2 * p * plane_out;
    if constexpr (sizeof(T) == 2) {
      const uint32_t w = *reinterpret_cast<const uint32_t*>(s2);
      const float u = bf16_to_f32((uint16_t)(w & 0xFFFFu)), v = bf16_to_f32((uint16_t)(w >> 16));
      const float ul = fmaf((float)m00, u, (float)m01 * v), vl = fmaf((float)m10, u, (float)m11 * v);
      *reinterpret_cast<uint32_t*>(d2) = pack_bf16x2(ul, vl);
    } else {
      const float2 w = *reinterpret_cast<const float2*>(s2);
      const double u = w.x, v = w.y;
      *reinterpret_cast<float2*>(d2) = make_float2((float)fma(m00, u, m01 * v), (float)fma(m10, u, m11 * v));
    }
  }
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

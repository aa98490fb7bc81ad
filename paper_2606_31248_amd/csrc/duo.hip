// Duo-grid halo padding of the six cube faces (App. F, "Tile extraction and
// DUO-style boundary padding"): face f is extended by `halo` cells on each
// side.  Interior cells are copied.  A halo cell extends f's equiangular mesh
// on f's own plane (alpha = -pi/4 + (j + 1/2) step with j past the face), its
// cube point is projected to the sphere, and its value is the inverse
// great-circle-distance weighted average of the 4 nearest cells of the face
// that contains that point -- the padding operator P, 4 non-zeros per row.
//
// Neighbour search: the 4 nearest cells lie within the 6 x 6 block of the
// containing face's cell lattice around the point's (clamped) floor index, so
// only those 36 candidates are measured.  Face scores and distances are
// compared on a 1e-12 grid, equal ones by index (face number; row, then
// column): exact ties -- a point on an edge, cells mirrored about it -- resolve
// the same way everywhere.  Geometry in float64 per halo cell; the weighted
// sums (nearest first, fused multiply-adds from 0) in float32 for bf16 data, in
// float64 for float32 data.
#include <climits>

#include "common.h"
#include "kernels.h"

namespace strata {
namespace {

constexpr double kTie = 1e-12;

// face axes: point = normal + a right + b up, a = tan(alpha), b = tan(beta)
__device__ __forceinline__ void face_axes(int f, double* n, double* r, double* u) {
  n[0] = n[1] = n[2] = r[0] = r[1] = r[2] = u[0] = u[1] = u[2] = 0.0;
  switch (f) {
    case 0: n[0] = 1; r[1] = 1; u[2] = 1; break;
    case 1: n[1] = 1; r[0] = -1; u[2] = 1; break;
    case 2: n[0] = -1; r[1] = -1; u[2] = 1; break;
    case 3: n[1] = -1; r[0] = 1; u[2] = 1; break;
    case 4: n[2] = 1; r[1] = 1; u[0] = -1; break;
    default: n[2] = -1; r[1] = 1; u[0] = 1; break;
  }
}

// unit sphere point of (possibly extended) cell (i, j) of face f
__device__ __forceinline__ void cell_point(int f, int i, int j, double step, double* p) {
  double n[3], r[3], u[3];
  face_axes(f, n, r, u);
  const double a = tan(-0.25 * M_PI + ((double)j + 0.5) * step);
  const double b = tan(-0.25 * M_PI + ((double)i + 0.5) * step);
  double s = 0.0;
  for (int k = 0; k < 3; ++k) {
    p[k] = n[k] + a * r[k] + b * u[k];
    s += p[k] * p[k];
  }
  const double inv = 1.0 / sqrt(s);
  for (int k = 0; k < 3; ++k) p[k] *= inv;
}

// the 4 nearest cells of the face containing halo cell (i, j) of face f
__device__ void halo_neighbours(int f, int i, int j, int n, int* fp_out, int* rows, int* cols, double* w) {
  const double step = 0.5 * M_PI / (double)n;
  double p[3];
  cell_point(f, i, j, step, p);
  // containing face: largest normal . p on the 1e-12 grid; a point on an edge
  // or corner belongs to the lowest-numbered of its faces
  int fp = 0;
  long long best = LLONG_MIN;
  for (int g = 0; g < 6; ++g) {
    double nn[3], rr[3], uu[3];
    face_axes(g, nn, rr, uu);
    const long long s = llrint((nn[0] * p[0] + nn[1] * p[1] + nn[2] * p[2]) / kTie);
    if (s > best) {
      best = s;
      fp = g;
    }
  }
  double nn[3], rr[3], uu[3];
  face_axes(fp, nn, rr, uu);
  const double pn = nn[0] * p[0] + nn[1] * p[1] + nn[2] * p[2];
  const double a = (rr[0] * p[0] + rr[1] * p[1] + rr[2] * p[2]) / pn;
  const double b = (uu[0] * p[0] + uu[1] * p[1] + uu[2] * p[2]) / pn;
  const int j0 = min(max((int)floor((atan(a) + 0.25 * M_PI) / step - 0.5), 0), n - 2);
  const int i0 = min(max((int)floor((atan(b) + 0.25 * M_PI) / step - 0.5), 0), n - 2);
  const int r0 = min(max(i0 - 2, 0), n - 6), c0 = min(max(j0 - 2, 0), n - 6);
  long long key[4];
  double dist[4];
  for (int k = 0; k < 4; ++k) {
    key[k] = LLONG_MAX;
    rows[k] = n;
    cols[k] = n;
    dist[k] = 0.0;
  }
  for (int r = r0; r < r0 + 6; ++r)
    for (int c = c0; c < c0 + 6; ++c) {
      double q[3];
      cell_point(fp, r, c, step, q);
      const double cx = q[1] * p[2] - q[2] * p[1], cy = q[2] * p[0] - q[0] * p[2], cz = q[0] * p[1] - q[1] * p[0];
      const double d = atan2(sqrt(cx * cx + cy * cy + cz * cz), q[0] * p[0] + q[1] * p[1] + q[2] * p[2]);
      const long long kd = llrint(d / kTie);
      // insert (kd, r, c) into the sorted top 4 (candidates come in (row, column) order)
      int pos = 4;
      while (pos > 0 && kd < key[pos - 1]) --pos;
      if (pos == 4) continue;
      for (int s = 3; s > pos; --s) {
        key[s] = key[s - 1];
        rows[s] = rows[s - 1];
        cols[s] = cols[s - 1];
        dist[s] = dist[s - 1];
      }
      key[pos] = kd;
      rows[pos] = r;
      cols[pos] = c;
      dist[pos] = d;
    }
  if (dist[0] == 0.0) {
    w[0] = 1.0;
    w[1] = w[2] = w[3] = 0.0;
  } else {
    double s = 0.0;
    for (int k = 0; k < 4; ++k) {
      w[k] = 1.0 / dist[k];
      s += w[k];
    }
    for (int k = 0; k < 4; ++k) w[k] /= s;
  }
  *fp_out = fp;
}

template <typename T>
__global__ void duo_halo_kernel(const T* __restrict__ in, int P, int n, int C, int halo, T* __restrict__ out) {
  const int m = n + 2 * halo;
  const int64_t per_face = (int64_t)m * m - (int64_t)n * n;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= 6 * per_face) return;
  const int f = (int)(idx / per_face);
  const int64_t hc = idx % per_face;
  int ip, jp;  // padded cell of the halo: top band, bottom band, then left/right strips
  const int64_t band = (int64_t)halo * m;
  if (hc < band) {
    ip = (int)(hc / m);
    jp = (int)(hc % m);
  } else if (hc < 2 * band) {
    const int64_t r = hc - band;
    ip = n + halo + (int)(r / m);
    jp = (int)(r % m);
  } else {
    const int64_t r = hc - 2 * band;
    ip = halo + (int)(r / (2 * halo));
    const int k = (int)(r % (2 * halo));
    jp = k < halo ? k : n + k;
  }
  int fp, rows[4], cols[4];
  double w[4];
  halo_neighbours(f, ip - halo, jp - halo, n, &fp, rows, cols, w);
  const int64_t plane_in = (int64_t)n * n * C, plane_out = (int64_t)m * m * C;
  const T* src = in + (int64_t)fp * P * plane_in;
  T* dst = out + (int64_t)f * P * plane_out + ((int64_t)ip * m + jp) * C;
  int64_t off[4];
  for (int k = 0; k < 4; ++k) off[k] = ((int64_t)rows[k] * n + cols[k]) * C;
  for (int p = 0; p < P; ++p) {
    const T* s = src + p * plane_in;
    T* d = dst + p * plane_out;
    for (int c = 0; c < C; ++c) {
      if constexpr (sizeof(T) == 2) {
        float acc = 0.f;
        for (int k = 0; k < 4; ++k) acc = fmaf((float)w[k], bf16_to_f32(s[off[k] + c]), acc);
        d[c] = f32_to_bf16(acc);
      } else {
        double acc = 0.0;
        for (int k = 0; k < 4; ++k) acc = fma(w[k], (double)s[off[k] + c], acc);
        d[c] = (float)acc;
      }
    }
  }
}

// interior: out[f, p, halo + i, halo + j, :] = in[f, p, i, j, :], one row of n*C
// elements per (f, p, i), copied in 4-byte words when the layout allows, else
// element by element
template <typename W>
__global__ void duo_interior_kernel(const char* __restrict__ in, int64_t rows, int64_t row_bytes, int n, int halo,
                                    int64_t cell_bytes, char* __restrict__ out) {
  const int64_t words = row_bytes / (int64_t)sizeof(W);
  const int m = n + 2 * halo;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const int64_t fp_ = row / n;  // (f, p) plane
    const int i = (int)(row % n);
    const W* s = reinterpret_cast<const W*>(in + row * row_bytes);
    W* d = reinterpret_cast<W*>(out + ((fp_ * m + halo + i) * m + halo) * cell_bytes);
    for (int64_t x = threadIdx.x; x < words; x += blockDim.x) d[x] = s[x];
  }
}

}  // namespace

void launch_duo_pad(const void* in, int P, int n, int C, int halo, void* out, strata_dtype dt, hipStream_t s) {
  const int64_t es = dt == STRATA_BF16 ? 2 : 4;
  const int64_t cell = C * es, row_bytes = (int64_t)n * cell, rows = 6LL * P * n;
  const unsigned blocks = (unsigned)(rows < 65536 ? rows : 65536);
  if (row_bytes % 4 == 0 && (halo * cell) % 4 == 0 && (halo * 2 * cell) % 4 == 0)
    hipLaunchKernelGGL((duo_interior_kernel<uint32_t>), dim3(blocks), dim3(256), 0, s,
                       static_cast<const char*>(in), rows, row_bytes, n, halo, cell, static_cast<char*>(out));
  else
    hipLaunchKernelGGL((duo_interior_kernel<uint16_t>), dim3(blocks), dim3(256), 0, s,
                       static_cast<const char*>(in), rows, row_bytes, n, halo, cell, static_cast<char*>(out));
  const int64_t m = n + 2 * halo, nh = 6 * (m * m - (int64_t)n * n);
  const unsigned hb = (unsigned)((nh + 127) / 128);
  if (dt == STRATA_BF16)
    hipLaunchKernelGGL((duo_halo_kernel<uint16_t>), dim3(hb), dim3(128), 0, s, static_cast<const uint16_t*>(in), P,
                       n, C, halo, static_cast<uint16_t*>(out));
  else
    hipLaunchKernelGGL((duo_halo_kernel<float>), dim3(hb), dim3(128), 0, s, static_cast<const float*>(in), P, n, C,
                       halo, static_cast<float*>(out));
}

}  // namespace strata

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
// only those 36 candidates are ranked, first by the cosine of their angle to the
// point; the exact great-circle distance is taken for the few within 1e-9 of the
// fourth-largest cosine.  Face scores and distances are compared on a 1e-12 grid, equal ones by index (face number; row, then
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
  const double pr = rr[0] * p[0] + rr[1] * p[1] + rr[2] * p[2];
  const double pu = uu[0] * p[0] + uu[1] * p[1] + uu[2] * p[2];
  const double a = pr / pn, b = pu / pn;
  const int j0 = min(max((int)floor((atan(a) + 0.25 * M_PI) / step - 0.5), 0), n - 2);
  const int i0 = min(max((int)floor((atan(b) + 0.25 * M_PI) / step - 0.5), 0), n - 2);
  const int r0 = min(max(i0 - 2, 0), n - 6), c0 = min(max(j0 - 2, 0), n - 6);
  // the block's mesh is separable: one tangent per row and per column
  double ta[6], tb[6];
  for (int t = 0; t < 6; ++t) {
    ta[t] = tan(-0.25 * M_PI + ((double)(c0 + t) + 0.5) * step);
    tb[t] = tan(-0.25 * M_PI + ((double)(r0 + t) + 0.5) * step);
  }
  // cosine of the angle from p to candidate (r, c) of the block: decreasing in
  // the great-circle distance
  // (the face axes are orthonormal: |n + x r + y u|^2 = 1 + x^2 + y^2)
  auto cosine = [&](int r, int c) {
    const double x = ta[c], y = tb[r];
    return (pn + x * pr + y * pu) * rsqrt(1.0 + x * x + y * y);
  };
  // pass 1: the fourth-largest cosine (fixed-index bubble steps keep the list
  // in registers)
  double top[4] = {-2.0, -2.0, -2.0, -2.0};
  for (int r = 0; r < 6; ++r)
    for (int c = 0; c < 6; ++c) {
      const double cs = cosine(r, c);
      if (cs > top[3]) {
        top[3] = cs;
#pragma unroll
        for (int t = 3; t > 0; --t)
          if (top[t] > top[t - 1]) {
            const double x = top[t];
            top[t] = top[t - 1];
            top[t - 1] = x;
          }
      }
    }
  // pass 2: exact distances on the tie grid for the shortlist only.  A
  // candidate whose cosine is 1e-9 below the fourth-largest lies more than
  // 1e-9 rad farther than four others (|d cos / d angle| <= 1), far beyond the
  // grid, so dropping it cannot change the selected four.
  const double floor_cos = top[3] - 1e-9;
  long long key[4];
  double dist[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    key[k] = LLONG_MAX;
    rows[k] = n;
    cols[k] = n;
    dist[k] = 0.0;
  }
  for (int r = 0; r < 6; ++r)
    for (int c = 0; c < 6; ++c) {
      if (cosine(r, c) < floor_cos) continue;
      double q[3], qs = 0.0;
      for (int k = 0; k < 3; ++k) {
        q[k] = nn[k] + ta[c] * rr[k] + tb[r] * uu[k];
        qs += q[k] * q[k];
      }
      const double qi = 1.0 / sqrt(qs);
      for (int k = 0; k < 3; ++k) q[k] *= qi;
      const double cx = q[1] * p[2] - q[2] * p[1], cy = q[2] * p[0] - q[0] * p[2], cz = q[0] * p[1] - q[1] * p[0];
      const double d = atan2(sqrt(cx * cx + cy * cy + cz * cz), q[0] * p[0] + q[1] * p[1] + q[2] * p[2]);
      const long long kd = llrint(d / kTie);
      // place (kd, row, column) last and move it up past strictly larger keys:
      // candidates come in (row, column) order, so equal keys keep that order
      if (kd < key[3]) {
        key[3] = kd;
        rows[3] = r0 + r;
        cols[3] = c0 + c;
        dist[3] = d;
#pragma unroll
        for (int t = 3; t > 0; --t)
          if (key[t] < key[t - 1]) {
            const long long k1 = key[t];
            key[t] = key[t - 1];
            key[t - 1] = k1;
            const int r1 = rows[t];
            rows[t] = rows[t - 1];
            rows[t - 1] = r1;
            const int c1 = cols[t];
            cols[t] = cols[t - 1];
            cols[t - 1] = c1;
            const double d1 = dist[t];
            dist[t] = dist[t - 1];
            dist[t - 1] = d1;
          }
      }
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

// padded cell (ip, jp) of halo cell number hc of a face: the top band (halo
// rows of m cells), the bottom band, then the left/right strips (2 halo cells
// per interior row)
__device__ __forceinline__ void halo_cell_position(int64_t hc, int n, int halo, int* ip, int* jp) {
  const int m = n + 2 * halo;
  const int64_t band = (int64_t)halo * m;
  if (hc < band) {
    *ip = (int)(hc / m);
    *jp = (int)(hc % m);
  } else if (hc < 2 * band) {
    const int64_t r = hc - band;
    *ip = n + halo + (int)(r / m);
    *jp = (int)(r % m);
  } else {
    const int64_t r = hc - 2 * band;
    *ip = halo + (int)(r / (2 * halo));
    const int k = (int)(r % (2 * halo));
    *jp = k < halo ? k : n + k;
  }
}

// G channels of one cell moved as one access
template <typename T, int G>
struct alignas(sizeof(T) * G) Group {
  T v[G];
};

// accumulation type: float for bf16 data, double for float32 data
__device__ __forceinline__ float widen(uint16_t x) { return bf16_to_f32(x); }
__device__ __forceinline__ double widen(float x) { return x; }

// one channel group of one halo cell, all P levels: weighted sum of the 4
// source cells, nearest first.  src and dst point at the group's first channel
// of level 0; off holds the source cells' element offsets.
template <typename T, int G>
__device__ __forceinline__ void gather_group(const T* src, const int64_t* off, const double* w, int P,
                                             int64_t plane_in, int64_t plane_out, T* dst) {
  using Acc = decltype(widen(T{}));
  Acc wk[4];
  for (int k = 0; k < 4; ++k) wk[k] = (Acc)w[k];
  for (int p = 0; p < P; ++p) {
    Group<T, G> g[4], o;
    for (int k = 0; k < 4; ++k) g[k] = *reinterpret_cast<const Group<T, G>*>(src + p * plane_in + off[k]);
    for (int e = 0; e < G; ++e) {
      Acc acc = 0;
      for (int k = 0; k < 4; ++k) acc = fma(wk[k], widen(g[k].v[e]), acc);
      if constexpr (sizeof(T) == 2)
        o.v[e] = f32_to_bf16(acc);
      else
        o.v[e] = (float)acc;
    }
    *reinterpret_cast<Group<T, G>*>(dst + p * plane_out) = o;
  }
}

// one halo cell, all P levels and C channels, G channels per access
template <typename T, int G>
__device__ __forceinline__ void gather_cell(const T* src, const int64_t* off, const double* w, int P, int C,
                                            int64_t plane_in, int64_t plane_out, T* dst) {
  for (int c = 0; c < C; c += G) gather_group<T, G>(src + c, off, w, P, plane_in, plane_out, dst + c);
}

// interior row i of plane pl: out[pl, halo + i, halo : halo + n, :] = in[pl, i, :, :]
template <typename W>
__device__ __forceinline__ void copy_row(const char* in, int64_t row, int64_t row_bytes, int n, int halo,
                                         int64_t cell_bytes, char* out) {
  const int m = n + 2 * halo;
  const int64_t pl = row / n;
  const int i = (int)(row % n);
  const W* s = reinterpret_cast<const W*>(in + row * row_bytes);
  W* d = reinterpret_cast<W*>(out + ((pl * m + halo + i) * m + halo) * cell_bytes);
  const int64_t words = row_bytes / (int64_t)sizeof(W);
  for (int64_t x = threadIdx.x; x < words; x += blockDim.x) d[x] = s[x];
}

// One launch for the whole padding.  Blocks [0, halo_blocks) take one halo
// cell per thread (geometry-bound); the following blocks copy one interior
// row each (bandwidth-bound), so the two kinds of work overlap on the chip.
// `group` is the channel access width of the halo gathers (4, 2 or 1
// elements) and `word` the byte width of the interior copy (16, 8, 4 or 2),
// both chosen by the host from the layout and the base addresses.
template <typename T>
__global__ __launch_bounds__(256) void duo_pad_kernel(const T* __restrict__ in, int P, int n, int C, int halo,
                                                      int group, int word, int64_t halo_blocks,
                                                      T* __restrict__ out) {
  const int m = n + 2 * halo;
  if ((int64_t)blockIdx.x >= halo_blocks) {
    const int64_t row = (int64_t)blockIdx.x - halo_blocks;
    const int64_t cell = (int64_t)C * sizeof(T), row_bytes = (int64_t)n * cell;
    const char* src = reinterpret_cast<const char*>(in);
    char* dst = reinterpret_cast<char*>(out);
    if (word == 16)
      copy_row<uint4>(src, row, row_bytes, n, halo, cell, dst);
    else if (word == 8)
      copy_row<uint2>(src, row, row_bytes, n, halo, cell, dst);
    else if (word == 4)
      copy_row<uint32_t>(src, row, row_bytes, n, halo, cell, dst);
    else
      copy_row<uint16_t>(src, row, row_bytes, n, halo, cell, dst);
    return;
  }
  const int64_t per_face = (int64_t)m * m - (int64_t)n * n;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= 6 * per_face) return;
  const int f = (int)(idx / per_face);
  int ip, jp;
  halo_cell_position(idx % per_face, n, halo, &ip, &jp);
  int fp, rows[4], cols[4];
  double w[4];
  halo_neighbours(f, ip - halo, jp - halo, n, &fp, rows, cols, w);
  const int64_t plane_in = (int64_t)n * n * C, plane_out = (int64_t)m * m * C;
  const T* src = in + (int64_t)fp * P * plane_in;
  T* dst = out + (int64_t)f * P * plane_out + ((int64_t)ip * m + jp) * C;
  int64_t off[4];
  for (int k = 0; k < 4; ++k) off[k] = ((int64_t)rows[k] * n + cols[k]) * C;
  if (group == 4)
    gather_cell<T, 4>(src, off, w, P, C, plane_in, plane_out, dst);
  else if (group == 2)
    gather_cell<T, 2>(src, off, w, P, C, plane_in, plane_out, dst);
  else
    gather_cell<T, 1>(src, off, w, P, C, plane_in, plane_out, dst);
}

// ---- the padding operator as a plan --------------------------------------
// The neighbours and weights depend only on (n, halo): built once, the
// operator is then applied as a bandwidth-bound gather.  One 64-byte entry per
// halo cell, faces in order, cells of a face in the order top band, bottom
// band, left/right strips (the halo enumeration above).
struct alignas(16) DuoEntry {
  double w[4];       // inverse-distance weights, nearest first, sum 1
  int32_t cell[4];   // source cells r * n + c on `face`
  int32_t face;
  int32_t unused[3];
};
static_assert(sizeof(DuoEntry) == 64, "plan entry layout");

// halo cell number of padded cell (ip, jp), inverse of the enumeration
__device__ __forceinline__ int64_t halo_cell_number(int ip, int jp, int n, int halo) {
  const int m = n + 2 * halo;
  const int64_t band = (int64_t)halo * m;
  if (ip < halo) return (int64_t)ip * m + jp;
  if (ip >= n + halo) return band + (int64_t)(ip - n - halo) * m + jp;
  return 2 * band + (int64_t)(ip - halo) * 2 * halo + (jp < halo ? jp : jp - n);
}

__global__ __launch_bounds__(256) void duo_plan_kernel(int n, int halo, DuoEntry* __restrict__ plan) {
  const int m = n + 2 * halo;
  const int64_t per_face = (int64_t)m * m - (int64_t)n * n;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= 6 * per_face) return;
  const int f = (int)(idx / per_face);
  int ip, jp;
  halo_cell_position(idx % per_face, n, halo, &ip, &jp);
  int fp, rows[4], cols[4];
  double w[4];
  halo_neighbours(f, ip - halo, jp - halo, n, &fp, rows, cols, w);
  DuoEntry e;
  for (int k = 0; k < 4; ++k) {
    e.w[k] = w[k];
    e.cell[k] = rows[k] * n + cols[k];
  }
  e.face = fp;
  e.unused[0] = e.unused[1] = e.unused[2] = 0;
  plan[idx] = e;
}

// the n interior cells of a padded row at every level, in W-byte words
template <typename W>
__device__ __forceinline__ void copy_span(const char* src, char* dst, int64_t bytes, int P, int64_t plane_in,
                                          int64_t plane_out) {
  const int64_t words = bytes / (int64_t)sizeof(W);
  for (int p = 0; p < P; ++p) {
    const W* s = reinterpret_cast<const W*>(src + p * plane_in);
    W* d = reinterpret_cast<W*>(dst + p * plane_out);
    for (int64_t x = threadIdx.x; x < words; x += blockDim.x) d[x] = s[x];
  }
}

// One block per padded row (f, ip), all P levels.  Halo cells are gathered
// through the plan with the same weights and summation order as the
// on-the-fly kernel (identical results), G channels per access; the interior
// span of the row is copied in `word`-byte words.
template <typename T, int G>
__global__ __launch_bounds__(1024) void duo_apply_kernel(const T* __restrict__ in, const DuoEntry* __restrict__ plan,
                                                        int P, int n, int C, int halo, int word,
                                                        T* __restrict__ out) {
  const int m = n + 2 * halo;
  const int f = blockIdx.x / m, ip = blockIdx.x % m;
  const int groups = C / G;
  const int64_t plane_in = (int64_t)n * n * C, plane_out = (int64_t)m * m * C;
  const int64_t per_face = (int64_t)m * m - (int64_t)n * n;
  const bool band = ip < halo || ip >= n + halo;
  T* orow = out + (int64_t)f * P * plane_out + (int64_t)ip * m * C;
  // halo cells of this row: all m in a band row, else the 2 halo strip cells
  const int nh = band ? m : 2 * halo;
  for (int t = threadIdx.x; t < nh * groups; t += blockDim.x) {
    const int h = t / groups, c = (t - h * groups) * G;
    const int jp = band ? h : (h < halo ? h : n + h);
    const DuoEntry e = plan[(int64_t)f * per_face + halo_cell_number(ip, jp, n, halo)];
    // entries of a plan for other (n, halo) could point anywhere: skip them
    if (e.face < 0 || e.face > 5 || (e.cell[0] | e.cell[1] | e.cell[2] | e.cell[3]) < 0 ||
        max(max(e.cell[0], e.cell[1]), max(e.cell[2], e.cell[3])) >= n * n)
      continue;
    int64_t off[4];
    for (int k = 0; k < 4; ++k) off[k] = (int64_t)e.cell[k] * C;
    gather_group<T, G>(in + (int64_t)e.face * P * plane_in + c, off, e.w, P, plane_in, plane_out,
                       orow + (int64_t)jp * C + c);
  }
  if (band) return;
  const char* src = reinterpret_cast<const char*>(in + (int64_t)f * P * plane_in + (int64_t)(ip - halo) * n * C);
  char* dst = reinterpret_cast<char*>(orow + (int64_t)halo * C);
  const int64_t bytes = (int64_t)n * C * sizeof(T), pin = plane_in * sizeof(T), pout = plane_out * sizeof(T);
  if (word == 16)
    copy_span<uint4>(src, dst, bytes, P, pin, pout);
  else if (word == 8)
    copy_span<uint2>(src, dst, bytes, P, pin, pout);
  else if (word == 4)
    copy_span<uint32_t>(src, dst, bytes, P, pin, pout);
  else
    copy_span<uint16_t>(src, dst, bytes, P, pin, pout);
}

// ---- the adjoint P^T -------------------------------------------------------
// Transposed entries, grouped by source cell and, within a source cell, in
// ascending padded-cell order (face, row, column), so every gradient sums in
// one fixed order.  Cells are packed as face << 28 | cell within the face (the
// plan requires n + 2 halo < 2^14).
struct alignas(16) DuoTEntry {
  int32_t src;   // source cell: f << 28 | r * n + c
  int32_t halo;  // halo cell of the padded faces: f << 28 | ip * m + jp
  double w;
};
constexpr int kFaceShift = 28;
constexpr int32_t kCellMask = (1 << kFaceShift) - 1;
static_assert(sizeof(DuoTEntry) == 16, "transposed entry layout");

// byte offsets of the plan's sections
struct PlanLayout {
  int64_t fwd, tent, cursor, sums, rank, hsums, heads, nheads, total;
};

__host__ __device__ inline int64_t align16(int64_t x) { return (x + 15) & ~(int64_t)15; }

inline PlanLayout plan_layout(int n, int halo) {
  const int64_t m = n + 2 * halo, nh = 6 * (m * m - (int64_t)n * n), cells = 6LL * n * n;
  PlanLayout L;
  L.fwd = 0;
  L.tent = align16(L.fwd + nh * (int64_t)sizeof(DuoEntry));
  L.cursor = align16(L.tent + 4 * nh * (int64_t)sizeof(DuoTEntry));
  L.sums = align16(L.cursor + cells * 4);
  L.rank = align16(L.sums + (cells + 1023) / 1024 * 4);  // segment-start flags, then their ranks
  L.hsums = align16(L.rank + 4 * nh * 4);
  L.heads = align16(L.hsums + (4 * nh + 1023) / 1024 * 4);  // first entry of each source cell
  L.nheads = align16(L.heads + 4 * nh * 4);
  L.total = align16(L.nheads + 4);
  return L;
}

__global__ __launch_bounds__(256) void zero_i32_kernel(int32_t* __restrict__ x, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
    x[i] = 0;
}

// entries per source cell (integer atomics: the counts are exact)
__global__ __launch_bounds__(256) void duo_count_kernel(const DuoEntry* __restrict__ plan, int64_t nh, int n,
                                                        int32_t* __restrict__ cursor) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= 4 * nh) return;
  const DuoEntry& e = plan[t >> 2];
  atomicAdd(&cursor[(int64_t)e.face * n * n + e.cell[t & 3]], 1);
}

// inclusive scan of one value per lane over a 64-lane wave
__device__ __forceinline__ int32_t wave_inclusive_scan(int32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t u = __shfl_up(v, d, 64);
    if (lane >= d) v += u;
  }
  return v;
}

// exclusive scan, pass 1: each block of 256 threads scans 1024 values in place
// and records its total
__global__ __launch_bounds__(256) void scan_blocks_kernel(int32_t* __restrict__ x, int64_t count,
                                                          int32_t* __restrict__ sums) {
  __shared__ int32_t wave_tot[4];
  const int64_t base = (int64_t)blockIdx.x * 1024 + threadIdx.x * 4;
  int32_t v[4], t = 0;
  for (int k = 0; k < 4; ++k) {
    v[k] = base + k < count ? x[base + k] : 0;
    t += v[k];
  }
  const int32_t inc = wave_inclusive_scan(t);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) wave_tot[w] = inc;
  __syncthreads();
  int32_t before = inc - t;
  for (int k = 0; k < w; ++k) before += wave_tot[k];
  for (int k = 0; k < 4; ++k) {
    if (base + k < count) x[base + k] = before;
    before += v[k];
  }
  if (threadIdx.x == 255) sums[blockIdx.x] = before;
}

// pass 2 (one block of 1024 threads): exclusive scan of the block totals
__global__ __launch_bounds__(1024) void scan_sums_kernel(int32_t* __restrict__ sums, int64_t nb) {
  __shared__ int32_t wave_tot[16];
  __shared__ int32_t carry_s;
  if (threadIdx.x == 0) carry_s = 0;
  __syncthreads();
  for (int64_t c0 = 0; c0 < nb; c0 += 1024) {
    const int64_t i = c0 + threadIdx.x;
    const int32_t v = i < nb ? sums[i] : 0;
    const int32_t inc = wave_inclusive_scan(v);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 63) wave_tot[w] = inc;
    __syncthreads();
    int32_t before = carry_s + inc - v;
    for (int k = 0; k < w; ++k) before += wave_tot[k];
    if (i < nb) sums[i] = before;
    __syncthreads();
    if (threadIdx.x == 1023) carry_s = before + v;
    __syncthreads();
  }
}

// pass 3: add each block's offset
__global__ __launch_bounds__(256) void scan_add_kernel(int32_t* __restrict__ x, int64_t count,
                                                       const int32_t* __restrict__ sums) {
  const int64_t base = (int64_t)blockIdx.x * 1024;
  const int32_t add = sums[blockIdx.x];
  for (int k = threadIdx.x; k < 1024; k += 256)
    if (base + k < count) x[base + k] += add;
}

// place every (halo cell, k) entry in its source cell's segment
__global__ __launch_bounds__(256) void duo_fill_kernel(const DuoEntry* __restrict__ plan, int64_t nh, int n, int halo,
                                                       int32_t* __restrict__ cursor, DuoTEntry* __restrict__ tent) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= 4 * nh) return;
  const DuoEntry& e = plan[t >> 2];
  const int32_t pos = atomicAdd(&cursor[(int64_t)e.face * n * n + e.cell[t & 3]], 1);
  if (pos < 0 || pos >= 4 * nh) return;  // cannot happen with a correct scan; keeps every store in bounds
  const int m = n + 2 * halo;
  const int64_t per_face = (int64_t)m * m - (int64_t)n * n;
  const int hf = (int)((t >> 2) / per_face);
  int ip, jp;
  halo_cell_position((t >> 2) - (int64_t)hf * per_face, n, halo, &ip, &jp);
  DuoTEntry o;
  o.src = (e.face << kFaceShift) | e.cell[t & 3];
  o.halo = (hf << kFaceShift) | (ip * m + jp);
  o.w = e.w[t & 3];
  tent[pos] = o;
}

// the segment starting at pos, if pos starts one: [pos, end)
__device__ __forceinline__ bool segment_at(const DuoTEntry* tent, int64_t total, int64_t pos, int64_t* end) {
  const int32_t src = tent[pos].src;
  if (pos > 0 && tent[pos - 1].src == src) return false;
  int64_t e = pos + 1;
  while (e < total && tent[e].src == src) ++e;
  *end = e;
  return true;
}

// order each segment by padded cell (segments are short: insertion sort;
// other threads only read the src fields, which a sort within a segment keeps)
__global__ __launch_bounds__(256) void duo_sort_kernel(DuoTEntry* __restrict__ tent, int64_t total) {
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= total) return;
  int64_t end;
  if (!segment_at(tent, total, pos, &end)) return;
  for (int64_t a = pos + 1; a < end; ++a) {
    const DuoTEntry x = tent[a];
    int64_t b = a;
    while (b > pos && tent[b - 1].halo > x.halo) {
      tent[b] = tent[b - 1];
      --b;
    }
    tent[b] = x;
  }
}

// 1 where an entry starts its source cell's segment
__global__ __launch_bounds__(256) void duo_head_flag_kernel(const DuoTEntry* __restrict__ tent, int64_t total,
                                                            int32_t* __restrict__ flag) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  flag[t] = (t == 0 || tent[t - 1].src != tent[t].src) ? 1 : 0;
}

// after the exclusive scan of the flags: the list of segment starts in
// ascending order, and its length
__global__ __launch_bounds__(256) void duo_head_list_kernel(const DuoTEntry* __restrict__ tent, int64_t total,
                                                            const int32_t* __restrict__ rank,
                                                            int32_t* __restrict__ heads,
                                                            int32_t* __restrict__ nheads) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  const bool head = t == 0 || tent[t - 1].src != tent[t].src;
  if (head) heads[rank[t]] = (int32_t)t;
  if (t == total - 1) *nheads = rank[t] + (head ? 1 : 0);
}

// P^T for one source cell with halo entries [pos, end), level p: its interior
// gradient plus the weighted gradients of those halo cells, in segment order,
// one rounding (float32 sums for bf16 data, float64 for float32 data).  The
// entries are taken 8 at a time, all loads issued before the sums.
template <typename T, int G>
__device__ __forceinline__ void vjp_segment(const T* gpad, const DuoTEntry* tent, int64_t pos, int64_t end, int p,
                                            int P, int n, int C, int halo, T* gfaces) {
  const int m = n + 2 * halo;
  const int64_t plane_in = (int64_t)n * n * C, plane_out = (int64_t)m * m * C;
  const int32_t src = tent[pos].src;
  const int f = src >> kFaceShift, cell = src & kCellMask;
  if (f > 5 || cell >= n * n) return;  // only a plan for other (n, halo) holds such entries
  const int r = cell / n, c = cell - r * n;
  const T* gi = gpad + ((int64_t)f * P + p) * plane_out + ((int64_t)(halo + r) * m + (halo + c)) * C;
  T* go = gfaces + ((int64_t)f * P + p) * plane_in + (int64_t)cell * C;
  using Acc = decltype(widen(T{}));
  for (int c0 = 0; c0 < C; c0 += G) {
    const Group<T, G> own = *reinterpret_cast<const Group<T, G>*>(gi + c0);
    Acc acc[G];
    for (int e = 0; e < G; ++e) acc[e] = widen(own.v[e]);
    for (int64_t q0 = pos; q0 < end; q0 += 8) {
      DuoTEntry x[8];
      Group<T, G> g[8];
      bool ok[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        ok[u] = q0 + u < end;
        if (ok[u]) x[u] = tent[q0 + u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (!ok[u]) continue;
        const int hf = x[u].halo >> kFaceShift, hcell = x[u].halo & kCellMask;
        ok[u] = hf <= 5 && hcell < m * m;  // only a plan for other (n, halo) holds others
        if (ok[u])
          g[u] = *reinterpret_cast<const Group<T, G>*>(gpad + ((int64_t)hf * P + p) * plane_out +
                                                       (int64_t)hcell * C + c0);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (!ok[u]) continue;
        const Acc wv = (Acc)x[u].w;
        for (int e = 0; e < G; ++e) acc[e] = fma(wv, widen(g[u].v[e]), acc[e]);
      }
    }
    Group<T, G> o;
    for (int e = 0; e < G; ++e) {
      if constexpr (sizeof(T) == 2)
        o.v[e] = f32_to_bf16(acc[e]);
      else
        o.v[e] = (float)acc[e];
    }
    *reinterpret_cast<Group<T, G>*>(go + c0) = o;
  }
}

// P^T, interior part: one block per face row (f, i), all levels, the row's
// interior span of the padded gradient copied in `word`-byte words
__global__ __launch_bounds__(1024) void duo_crop_kernel(const char* __restrict__ gpad, int P, int n, int C, int es,
                                                        int halo, int word, char* __restrict__ gfaces) {
  const int m = n + 2 * halo;
  const int f = blockIdx.x / n, i = blockIdx.x % n;
  const int64_t cell = (int64_t)C * es;
  const char* src = gpad + ((int64_t)f * P * m * m + (int64_t)(halo + i) * m + halo) * cell;
  char* dst = gfaces + ((int64_t)f * P * n * n + (int64_t)i * n) * cell;
  const int64_t bytes = n * cell, pin = (int64_t)m * m * cell, pout = (int64_t)n * n * cell;
  if (word == 16)
    copy_span<uint4>(src, dst, bytes, P, pin, pout);
  else if (word == 8)
    copy_span<uint2>(src, dst, bytes, P, pin, pout);
  else if (word == 4)
    copy_span<uint32_t>(src, dst, bytes, P, pin, pout);
  else
    copy_span<uint16_t>(src, dst, bytes, P, pin, pout);
}

// P^T, halo part (after the crop, on the same stream): one thread per (source
// cell with halo entries, level), each rewriting that cell's gradient at that
// level with the halo terms added
template <typename T, int G>
__global__ __launch_bounds__(256) void duo_vjp_halo_kernel(const T* __restrict__ gpad,
                                                           const DuoTEntry* __restrict__ tent,
                                                           const int32_t* __restrict__ heads,
                                                           const int32_t* __restrict__ nheads, int64_t total, int P,
                                                           int n, int C, int halo, T* __restrict__ gfaces) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int p = blockIdx.y;  // neighbouring lanes: neighbouring source cells of one level
  const int64_t count = min((int64_t)*nheads, total);
  if (k >= count) return;
  const int64_t pos = heads[k], end = k + 1 < count ? (int64_t)heads[k + 1] : total;
  if (pos < 0 || end > total || pos >= end) return;  // only a plan for other (n, halo) holds such entries
  vjp_segment<T, G>(gpad, tent, pos, end, p, P, n, C, halo, gfaces);
}

}  // namespace

void launch_duo_pad(const void* in, int P, int n, int C, int halo, void* out, strata_dtype dt, hipStream_t s) {
  const int64_t es = dt == STRATA_BF16 ? 2 : 4;
  const int64_t cell = C * es, row_bytes = (int64_t)n * cell, rows = 6LL * P * n;
  const int64_t m = n + 2 * halo, nh = 6 * (m * m - (int64_t)n * n);
  const int64_t halo_blocks = (nh + 255) / 256;
  const uintptr_t base = reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out);
  // widest copy word that divides every row start and length on both sides
  const uint64_t align = (uint64_t)row_bytes | (uint64_t)(halo * cell) | (uint64_t)(2 * halo * cell) | base;
  const int word = align % 16 == 0 ? 16 : align % 8 == 0 ? 8 : align % 4 == 0 ? 4 : 2;
  // channel groups of 4, 2 or 1, as the channel count and base addresses allow
  const int group = (C % 4 == 0 && base % (4 * es) == 0) ? 4 : (C % 2 == 0 && base % (2 * es) == 0) ? 2 : 1;
  const dim3 grid((unsigned)(halo_blocks + rows));
  if (dt == STRATA_BF16)
    hipLaunchKernelGGL((duo_pad_kernel<uint16_t>), grid, dim3(256), 0, s, static_cast<const uint16_t*>(in), P, n, C,
                       halo, group, word, halo_blocks, static_cast<uint16_t*>(out));
  else
    hipLaunchKernelGGL((duo_pad_kernel<float>), grid, dim3(256), 0, s, static_cast<const float*>(in), P, n, C, halo,
                       group, word, halo_blocks, static_cast<float*>(out));
}

int64_t duo_plan_bytes(int n, int halo) { return plan_layout(n, halo).total; }

void launch_duo_plan(int n, int halo, void* plan, hipStream_t s) {
  const PlanLayout L = plan_layout(n, halo);
  const int64_t m = n + 2 * halo, nh = 6 * (m * m - (int64_t)n * n), cells = 6LL * n * n;
  char* base = static_cast<char*>(plan);
  DuoEntry* fwd = reinterpret_cast<DuoEntry*>(base + L.fwd);
  DuoTEntry* tent = reinterpret_cast<DuoTEntry*>(base + L.tent);
  int32_t* cursor = reinterpret_cast<int32_t*>(base + L.cursor);
  int32_t* sums = reinterpret_cast<int32_t*>(base + L.sums);
  const int64_t nb = (cells + 1023) / 1024;
  const unsigned eb = (unsigned)((4 * nh + 255) / 256);
  hipLaunchKernelGGL(duo_plan_kernel, dim3((unsigned)((nh + 255) / 256)), dim3(256), 0, s, n, halo, fwd);
  // counters, block sums and the alignment tail: every byte of a plan is defined
  hipLaunchKernelGGL(zero_i32_kernel, dim3((unsigned)(nb < 4096 ? nb : 4096)), dim3(256), 0, s, cursor,
                     (L.total - L.cursor) / 4);
  hipLaunchKernelGGL(duo_count_kernel, dim3(eb), dim3(256), 0, s, fwd, nh, n, cursor);
  hipLaunchKernelGGL(scan_blocks_kernel, dim3((unsigned)nb), dim3(256), 0, s, cursor, cells, sums);
  hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(1024), 0, s, sums, nb);
  hipLaunchKernelGGL(scan_add_kernel, dim3((unsigned)nb), dim3(256), 0, s, cursor, cells, sums);
  hipLaunchKernelGGL(duo_fill_kernel, dim3(eb), dim3(256), 0, s, fwd, nh, n, halo, cursor, tent);
  hipLaunchKernelGGL(duo_sort_kernel, dim3(eb), dim3(256), 0, s, tent, 4 * nh);
  // the list of segment starts: flags, their exclusive scan, then the list
  int32_t* rank = reinterpret_cast<int32_t*>(base + L.rank);
  int32_t* hsums = reinterpret_cast<int32_t*>(base + L.hsums);
  const int64_t nb2 = (4 * nh + 1023) / 1024;
  hipLaunchKernelGGL(duo_head_flag_kernel, dim3(eb), dim3(256), 0, s, tent, 4 * nh, rank);
  hipLaunchKernelGGL(scan_blocks_kernel, dim3((unsigned)nb2), dim3(256), 0, s, rank, 4 * nh, hsums);
  hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(1024), 0, s, hsums, nb2);
  hipLaunchKernelGGL(scan_add_kernel, dim3((unsigned)nb2), dim3(256), 0, s, rank, 4 * nh, hsums);
  hipLaunchKernelGGL(duo_head_list_kernel, dim3(eb), dim3(256), 0, s, tent, 4 * nh, rank,
                     reinterpret_cast<int32_t*>(base + L.heads), reinterpret_cast<int32_t*>(base + L.nheads));
}

void launch_duo_pad_vjp(const void* gpad, const void* plan, int P, int n, int C, int halo, void* gfaces,
                        strata_dtype dt, hipStream_t s) {
  const PlanLayout L = plan_layout(n, halo);
  const int64_t es = dt == STRATA_BF16 ? 2 : 4, cell = C * es, m = n + 2 * halo;
  const int64_t nh = 6 * (m * m - (int64_t)n * n);
  const uintptr_t base = reinterpret_cast<uintptr_t>(gpad) | reinterpret_cast<uintptr_t>(gfaces);
  const uint64_t align = (uint64_t)(n * cell) | (uint64_t)(halo * cell) | (uint64_t)(m * cell) |
                         (uint64_t)((int64_t)n * n * cell) | (uint64_t)(m * m * cell) | base;
  const int word = align % 16 == 0 ? 16 : align % 8 == 0 ? 8 : align % 4 == 0 ? 4 : 2;
  hipLaunchKernelGGL(duo_crop_kernel, dim3((unsigned)(6 * n)), dim3(1024), 0, s, static_cast<const char*>(gpad), P,
                     n, C, (int)es, halo, word, static_cast<char*>(gfaces));
  const int group = (C % 4 == 0 && base % (4 * es) == 0) ? 4 : (C % 2 == 0 && base % (2 * es) == 0) ? 2 : 1;
  const char* pb = static_cast<const char*>(plan);
  const DuoTEntry* tent = reinterpret_cast<const DuoTEntry*>(pb + L.tent);
  const int32_t* heads = reinterpret_cast<const int32_t*>(pb + L.heads);
  const int32_t* nheads = reinterpret_cast<const int32_t*>(pb + L.nheads);
  const dim3 grid((unsigned)((4 * nh + 255) / 256), (unsigned)P);
#define STRATA_DUO_VJP(T, GG)                                                                                      \
  hipLaunchKernelGGL((duo_vjp_halo_kernel<T, GG>), grid, dim3(256), 0, s, static_cast<const T*>(gpad), tent, heads, \
                     nheads, 4 * nh, P, n, C, halo, static_cast<T*>(gfaces))
  if (dt == STRATA_BF16) {
    if (group == 4)
      STRATA_DUO_VJP(uint16_t, 4);
    else if (group == 2)
      STRATA_DUO_VJP(uint16_t, 2);
    else
      STRATA_DUO_VJP(uint16_t, 1);
  } else {
    if (group == 4)
      STRATA_DUO_VJP(float, 4);
    else if (group == 2)
      STRATA_DUO_VJP(float, 2);
    else
      STRATA_DUO_VJP(float, 1);
  }
#undef STRATA_DUO_VJP
}

void launch_duo_pad_planned(const void* in, const void* plan, int P, int n, int C, int halo, void* out,
                            strata_dtype dt, hipStream_t s) {
  const int64_t es = dt == STRATA_BF16 ? 2 : 4;
  const uintptr_t base = reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out);
  const int group = (C % 4 == 0 && base % (4 * es) == 0) ? 4 : (C % 2 == 0 && base % (2 * es) == 0) ? 2 : 1;
  // widest copy word dividing the interior span, its start in the padded row,
  // both row strides, both plane strides and the base addresses
  const int64_t cell = C * es, m = n + 2 * halo;
  const uint64_t align = (uint64_t)(n * cell) | (uint64_t)(halo * cell) | (uint64_t)(m * cell) |
                         (uint64_t)((int64_t)n * n * cell) | (uint64_t)(m * m * cell) | base;
  const int word = align % 16 == 0 ? 16 : align % 8 == 0 ? 8 : align % 4 == 0 ? 4 : 2;
  const dim3 grid((unsigned)(6 * m));
  const DuoEntry* pl = static_cast<const DuoEntry*>(plan);
#define STRATA_DUO_APPLY(T, GG)                                                                                   \
  hipLaunchKernelGGL((duo_apply_kernel<T, GG>), grid, dim3(1024), 0, s, static_cast<const T*>(in), pl, P, n, C, \
                     halo, word, static_cast<T*>(out))
  if (dt == STRATA_BF16) {
    if (group == 4)
      STRATA_DUO_APPLY(uint16_t, 4);
    else if (group == 2)
      STRATA_DUO_APPLY(uint16_t, 2);
    else
      STRATA_DUO_APPLY(uint16_t, 1);
  } else {
    if (group == 4)
      STRATA_DUO_APPLY(float, 4);
    else if (group == 2)
      STRATA_DUO_APPLY(float, 2);
    else
      STRATA_DUO_APPLY(float, 1);
  }
#undef STRATA_DUO_APPLY
}

}  // namespace strata

// Block groups of the balanced key-stationary dK/dV kernel (na3d_mfma_kvp.hip):
// which 4-wide key blocks of an axis share a workgroup, and which 4-aligned
// runs of 4 query positions ("squares") their query boxes span.  Host and
// device code, no HIP runtime calls (a host test compiles it on its own).
#pragma once

namespace strata {
namespace kvp {

// queries whose (border-clamped) window holds position j of an axis of extent L
__host__ __device__ __forceinline__ int inv_lo(int j, int k) { return j < k ? 0 : j - (k >> 1); }
__host__ __device__ __forceinline__ int inv_hi(int j, int L, int k) { return j >= L - k ? L - 1 : j + (k >> 1); }

// One axis of a workgroup: its blocks and the squares their query boxes span.
// Entry e of the square list is square base + e for e < n0, else base1 + e - n0.
struct AxisGroup {
  int nblk;            // blocks in the group (1 or 2)
  int blk0, blk1;      // block indices (blk1 valid when nblk == 2)
  int base, n0, base1, n;
  int run0, len0, run1, len1;  // each block's run of entries
};

// The blocks of group i on an axis of nb blocks: group 0 pairs the two edge
// blocks; the interior blocks 1 .. nb-2 go in pairs that start at block 1 at
// the low border and end at block nb-2 at the high one (the pairs whose query
// boxes fit four squares next to a border).  With an odd number of interior
// blocks one block near the middle, c (odd), stands alone between the two runs.
__host__ __device__ __forceinline__ void group_blocks(int i, int nb, int& b0, int& b1, int& nblk) {
  if (i == 0) {
    b0 = 0;
    b1 = nb - 1;
    nblk = nb > 1 ? 2 : 1;
    return;
  }
  const int c = ((nb - 2) & 1) ? 2 * ((nb - 1) / 4) + 1 : nb;  // the lone block, if any
  const int il = (c + 1) / 2;                                  // its group
  nblk = 2;
  if (i < il) {
    b0 = 2 * i - 1;
  } else if (i == il) {
    b0 = c;
    nblk = 1;
  } else {
    b0 = c + 1 + 2 * (i - il - 1);
  }
  b1 = b0 + 1;
}

__host__ __device__ __forceinline__ AxisGroup axis_group(int i, int L, int k) {
  const int nb = (L + 3) >> 2;
  AxisGroup r;
  group_blocks(i, nb, r.blk0, r.blk1, r.nblk);
  const int a0 = inv_lo(4 * r.blk0, k) >> 2;
  const int a1 = inv_hi(min(4 * r.blk0 + 3, L - 1), L, k) >> 2;
  r.base = a0;
  r.run0 = 0;
  r.len0 = a1 - a0 + 1;
  r.run1 = 0;
  r.len1 = 0;
  r.n0 = r.n = r.len0;
  r.base1 = a0;
  if (r.nblk == 2) {
    const int c0 = inv_lo(4 * r.blk1, k) >> 2;
    const int c1 = inv_hi(min(4 * r.blk1 + 3, L - 1), L, k) >> 2;
    r.len1 = c1 - c0 + 1;
    if (c0 <= a1 + 1) {  // the runs overlap or touch: one run of squares
      r.n0 = r.n = max(a1, c1) - a0 + 1;
      r.run1 = c0 - a0;
    } else {
      r.n0 = r.len0;
      r.n = r.len0 + r.len1;
      r.base1 = c0;
      r.run1 = r.len0;
    }
  }
  return r;
}

__host__ __device__ __forceinline__ int sq_abs(const AxisGroup& r, int e) {
  return e < r.n0 ? r.base + e : r.base1 + e - r.n0;
}

__host__ __device__ __forceinline__ int n_groups(int L) { return 1 + (((L + 3) >> 2) - 1) / 2; }

// every group of every axis fits the staged grid (at most four squares), and
// each block's run along x is 2, 3 or 4 squares wide (the unrolled walks)
inline bool groups_fit(int L, int k, bool x_axis) {
  for (int i = 0; i < n_groups(L); ++i) {
    const AxisGroup r = axis_group(i, L, k);
    if (r.n > 4) return false;
    if (x_axis && (r.len0 < 2 || (r.nblk == 2 && r.len1 < 2))) return false;
  }
  return true;
}

}  // namespace kvp
}  // namespace strata

/*
 * CPU oracle for the STRATA hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, float64 reference of what the hot path computes.  Only the
 * tests, the smoke check and the bench's CPU-baseline leg use it; the HIP
 * library shares no code with it.  Every function evaluates the definition
 * directly: no blocking, no fusion, no reordering beyond what the definition
 * states.
 *
 * Tensor layout everywhere: [B, heads, Z, H, W, d], d innermost, row-major.
 * Token positions inside a tile are (z, y, x) = (level, row, column).
 *
 * Sources (arxiv 2606.31248):
 *   - neighbourhood attention in local (x, y, level) windows, NATTEN-style
 *     (Sec. 3.2 "Transformer backbone");
 *   - StereoRoPE: axial 2D rotary embedding driven by the stereographic
 *     coordinates of Eq. 1 (Sec. 3.3);
 *   - tile stitching S = D^-1 P^T W with D = P^T W 1 (App. F, "Tile stitching"
 *     and Eq. (stitch));
 *   - QK RMSNorm and the sigmoid output gate of every attention block
 *     (App. B.5).
 * Readings where the paper is silent are stated at each function.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define IDX6(b, h, z, y, x, HEADS, Z, H, W) \
  (((((int64_t)(b) * (HEADS) + (h)) * (Z) + (z)) * (H) + (y)) * (W) + (x))

/* ---------------------------------------------------------------------------
 * Neighbourhood window on one axis (NATTEN border-clamped rule, dilation 1).
 * A query at i sees the k consecutive positions [s, s+k) with
 * s = clamp(i - (k-1)/2, 0, L-k): the window is centred on i and shifted
 * inward at the borders, so every query sees exactly k positions.
 * ------------------------------------------------------------------------- */
static int win_start(int i, int L, int k) {
  int s = i - (k - 1) / 2;
  if (s < 0) s = 0;
  if (s > L - k) s = L - k;
  return s;
}

static int in_window(int j, int i, int L, int k) {
  int s = win_start(i, L, k);
  return j >= s && j < s + k;
}

/* A window size is valid when it is odd and fits the axis, or when it is the
 * whole axis (any parity: the rule above then gives every query all L
 * positions; column-wise attention over all levels is that case). */
static int window_ok(int L, int k) { return L > 0 && k > 0 && k <= L && ((k % 2) == 1 || k == L); }

/* starts[i] for every query position, and for every key position j the
 * inclusive range [qlo[j], qhi[j]] of queries whose window holds j
 * (found by scanning all queries; qlo = L, qhi = -1 if none). */
int oracle_axis_index(int L, int k, int32_t* starts, int32_t* qlo, int32_t* qhi) {
  if (!window_ok(L, k)) return 1;
  for (int i = 0; i < L; ++i) starts[i] = win_start(i, L, k);
  for (int j = 0; j < L; ++j) {
    int lo = L, hi = -1;
    for (int i = 0; i < L; ++i)
      if (in_window(j, i, L, k)) {
        if (i < lo) lo = i;
        if (i > hi) hi = i;
      }
    qlo[j] = lo;
    qhi[j] = hi;
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * StereoRoPE (Sec. 3.3): the stereographic (x, y) of a token replaces the
 * row/column index of axial 2D RoPE.  Reading: pairs (2t, 2t+1); the first
 * d/4 pairs turn by x * w_t, the last d/4 pairs by y * w_t, with
 * w_t = base^(-t/(d/4)); the level axis is not rotated.  A pair (a, b) turns
 * by angle th to (a cos th - b sin th, a sin th + b cos th); the transpose
 * turns by -th.
 * ------------------------------------------------------------------------- */
static double rope_angle(double cx, double cy, int t, int d, double base) {
  int q = d / 4;
  if (t < q) return cx * pow(base, -(double)t / (double)q);
  return cy * pow(base, -(double)(t - q) / (double)q);
}

/* Phase table (cos, sin) per (b, y, x, pair), float64. */
static double* build_phases(const float* coords, int B, int H, int W, int d, double base) {
  int np = d / 2;
  double* ph = (double*)malloc(sizeof(double) * 2 * (size_t)B * H * W * np);
  if (!ph) return NULL;
  for (int64_t p = 0; p < (int64_t)B * H * W; ++p) {
    double cx = (double)coords[2 * p + 0];
    double cy = (double)coords[2 * p + 1];
    for (int t = 0; t < np; ++t) {
      double th = rope_angle(cx, cy, t, d, base);
      ph[(p * np + t) * 2 + 0] = cos(th);
      ph[(p * np + t) * 2 + 1] = sin(th);
    }
  }
  return ph;
}

static void rotate(const double* in, const double* ph, int d, double sign, double* out) {
  for (int t = 0; t < d / 2; ++t) {
    double c = ph[2 * t], s = sign * ph[2 * t + 1];
    double a = in[2 * t], b = in[2 * t + 1];
    out[2 * t] = a * c - b * s;
    out[2 * t + 1] = a * s + b * c;
  }
}

/* Phase table export: ph[b, y, x, t] = (cos th, sin th) in float64. */
int oracle_rope_phases(const float* coords, int B, int H, int W, int d, double base, double* out) {
  if (d % 4 != 0) return 1;
  double* ph = build_phases(coords, B, H, W, d, base);
  if (!ph) return 2;
  memcpy(out, ph, sizeof(double) * 2 * (size_t)B * H * W * (d / 2));
  free(ph);
  return 0;
}

int oracle_rope_apply(const double* x, const float* coords, int B, int heads, int Z, int H,
                      int W, int d, double base, int transpose, double* y) {
  if (d % 4 != 0) return 1;
  double* ph = build_phases(coords, B, H, W, d, base);
  if (!ph) return 2;
  double sign = transpose ? -1.0 : 1.0;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < heads; ++h)
      for (int z = 0; z < Z; ++z)
        for (int yy = 0; yy < H; ++yy)
          for (int xx = 0; xx < W; ++xx) {
            int64_t tok = IDX6(b, h, z, yy, xx, heads, Z, H, W);
            int64_t pos = ((int64_t)b * H + yy) * W + xx;
            rotate(x + tok * d, ph + pos * (d / 2) * 2, d, sign, y + tok * d);
          }
  free(ph);
  return 0;
}

/* ---------------------------------------------------------------------------
 * Neighbourhood attention forward for one query (b, h, z, y, x):
 *   s_j   = scale * <q~, k~_j>  for the kz*ky*kx keys j of its window,
 *   LSE   = m + ln sum_j exp(s_j - m),   m = max_j s_j,
 *   out   = sum_j exp(s_j - LSE) v_j,
 * with q~ = R q, k~ = R k when coordinates are given (StereoRoPE), else q, k.
 * ------------------------------------------------------------------------- */
typedef struct {
  int B, heads, Z, H, W, d, kz, ky, kx;
  double scale;
} na_dims;

static void na_query(const na_dims* D, const double* q, const double* k, const double* v,
                     const double* ph, int64_t qi, double* o, double* lse_out,
                     double* s /* K scratch */, double* qr, double* kr) {
  const int d = D->d;
  int64_t r = qi;
  int x = (int)(r % D->W); r /= D->W;
  int y = (int)(r % D->H); r /= D->H;
  int z = (int)(r % D->Z); r /= D->Z;
  int h = (int)(r % D->heads); r /= D->heads;
  int b = (int)r;
  const double* qv = q + qi * d;
  if (ph) {
    rotate(qv, ph + (((int64_t)b * D->H + y) * D->W + x) * (d / 2) * 2, d, 1.0, qr);
    qv = qr;
  }
  int zs = win_start(z, D->Z, D->kz), ys = win_start(y, D->H, D->ky), xs = win_start(x, D->W, D->kx);
  int n = 0;
  double m = -INFINITY;
  for (int kz = zs; kz < zs + D->kz; ++kz)
    for (int ky = ys; ky < ys + D->ky; ++ky)
      for (int kx = xs; kx < xs + D->kx; ++kx) {
        int64_t kj = IDX6(b, h, kz, ky, kx, D->heads, D->Z, D->H, D->W);
        const double* kv = k + kj * d;
        if (ph) {
          rotate(kv, ph + (((int64_t)b * D->H + ky) * D->W + kx) * (d / 2) * 2, d, 1.0, kr);
          kv = kr;
        }
        double acc = 0.0;
        for (int e = 0; e < d; ++e) acc += qv[e] * kv[e];
        s[n] = D->scale * acc;
        if (s[n] > m) m = s[n];
        ++n;
      }
  double sum = 0.0;
  for (int j = 0; j < n; ++j) sum += exp(s[j] - m);
  double lse = m + log(sum);
  for (int e = 0; e < d; ++e) o[e] = 0.0;
  n = 0;
  for (int kz = zs; kz < zs + D->kz; ++kz)
    for (int ky = ys; ky < ys + D->ky; ++ky)
      for (int kx = xs; kx < xs + D->kx; ++kx) {
        int64_t kj = IDX6(b, h, kz, ky, kx, D->heads, D->Z, D->H, D->W);
        double p = exp(s[n++] - lse);
        for (int e = 0; e < d; ++e) o[e] += p * v[kj * d + e];
      }
  if (lse_out) *lse_out = lse;
}

static int check_dims(const na_dims* D) {
  if (D->B <= 0 || D->heads <= 0 || D->Z <= 0 || D->H <= 0 || D->W <= 0 || D->d <= 0) return 1;
  if (!window_ok(D->Z, D->kz) || !window_ok(D->H, D->ky) || !window_ok(D->W, D->kx)) return 1;
  if (!(D->scale > 0.0)) return 1;
  return 0;
}

/* Forward for the queries listed in sel[0..nsel) (flat indices into
 * [B, heads, Z, H, W]); sel == NULL means every query in order.
 * out[i*d ...] and lse[i] belong to the i-th listed query. */
int oracle_na3d_fwd(const double* q, const double* k, const double* v, const float* coords,
                    double base, int B, int heads, int Z, int H, int W, int d, int kz, int ky,
                    int kx, double scale, int64_t nsel, const int64_t* sel, double* out,
                    double* lse) {
  na_dims D = {B, heads, Z, H, W, d, kz, ky, kx, scale};
  if (check_dims(&D)) return 1;
  if (coords && d % 4 != 0) return 1;
  int64_t nq = (int64_t)B * heads * Z * H * W;
  if (!sel) nsel = nq;
  double* ph = NULL;
  if (coords) {
    ph = build_phases(coords, B, H, W, d, base);
    if (!ph) return 2;
  }
  int K = kz * ky * kx;
  int err = 0;
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * K);
    double* qr = (double*)malloc(sizeof(double) * d);
    double* kr = (double*)malloc(sizeof(double) * d);
    if (!s || !qr || !kr) {
#pragma omp atomic write
      err = 2;
    } else {
#pragma omp for schedule(dynamic, 64)
      for (int64_t i = 0; i < nsel; ++i) {
        int64_t qi = sel ? sel[i] : i;
        na_query(&D, q, k, v, ph, qi, out + i * d, lse ? lse + i : NULL, s, qr, kr);
      }
    }
    free(s);
    free(qr);
    free(kr);
  }
  free(ph);
  return err;
}

/* ---------------------------------------------------------------------------
 * Neighbourhood attention backward: the gradient of the forward above with
 * respect to q, k, v for an upstream gradient dO, written out directly:
 *   P_ij  = exp(s_ij - LSE_i),      D_i = <dO_i, O_i>,
 *   dV_j  = sum_{i : j in N(i)} P_ij dO_i,
 *   dS_ij = P_ij (<dO_i, v_j> - D_i),
 *   dq~_i = scale sum_j dS_ij k~_j,   dk~_j = scale sum_i dS_ij q~_i,
 *   dq = R^T dq~, dk = R^T dk~.
 * The oracle recomputes O and LSE itself in float64.
 * dq is produced for the queries in selq, dk and dv for the keys in selk
 * (flat indices; NULL = all).
 * ------------------------------------------------------------------------- */
int oracle_na3d_bwd(const double* q, const double* k, const double* v, const float* coords,
                    double base, int B, int heads, int Z, int H, int W, int d, int kz, int ky,
                    int kx, double scale, const double* dout, int64_t nselq, const int64_t* selq,
                    int64_t nselk, const int64_t* selk, double* dq, double* dk, double* dv) {
  na_dims D = {B, heads, Z, H, W, d, kz, ky, kx, scale};
  if (check_dims(&D)) return 1;
  if (coords && d % 4 != 0) return 1;
  int64_t nq = (int64_t)B * heads * Z * H * W;
  if (!selq) nselq = nq;
  if (!selk) nselk = nq;
  double* ph = NULL;
  if (coords) {
    ph = build_phases(coords, B, H, W, d, base);
    if (!ph) return 2;
  }
  const int K = kz * ky * kx;
  int err = 0;
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * K);
    double* qr = (double*)malloc(sizeof(double) * d);
    double* kr = (double*)malloc(sizeof(double) * d);
    double* o = (double*)malloc(sizeof(double) * d);
    double* acc = (double*)malloc(sizeof(double) * d);
    double* acc2 = (double*)malloc(sizeof(double) * d);
    if (!s || !qr || !kr || !o || !acc || !acc2) {
#pragma omp atomic write
      err = 2;
    } else {
      /* dq */
#pragma omp for schedule(dynamic, 16)
      for (int64_t i = 0; i < nselq; ++i) {
        int64_t qi = selq ? selq[i] : i;
        double lse;
        na_query(&D, q, k, v, ph, qi, o, &lse, s, qr, kr);
        int64_t r = qi;
        int x = (int)(r % W); r /= W;
        int y = (int)(r % H); r /= H;
        int z = (int)(r % Z); r /= Z;
        int h = (int)(r % heads); r /= heads;
        int b = (int)r;
        const double* g = dout + qi * d;
        double Di = 0.0;
        for (int e = 0; e < d; ++e) Di += g[e] * o[e];
        for (int e = 0; e < d; ++e) acc[e] = 0.0;
        int zs = win_start(z, Z, kz), ys = win_start(y, H, ky), xs = win_start(x, W, kx);
        int n = 0;
        for (int jz = zs; jz < zs + kz; ++jz)
          for (int jy = ys; jy < ys + ky; ++jy)
            for (int jx = xs; jx < xs + kx; ++jx) {
              int64_t kj = IDX6(b, h, jz, jy, jx, heads, Z, H, W);
              double p = exp(s[n++] - lse);
              double dp = 0.0;
              for (int e = 0; e < d; ++e) dp += g[e] * v[kj * d + e];
              double ds = p * (dp - Di);
              const double* kv = k + kj * d;
              if (ph) {
                rotate(kv, ph + (((int64_t)b * H + jy) * W + jx) * (d / 2) * 2, d, 1.0, kr);
                kv = kr;
              }
              for (int e = 0; e < d; ++e) acc[e] += scale * ds * kv[e];
            }
        if (ph)
          rotate(acc, ph + (((int64_t)b * H + y) * W + x) * (d / 2) * 2, d, -1.0, dq + i * d);
        else
          memcpy(dq + i * d, acc, sizeof(double) * d);
      }
      /* dk, dv */
#pragma omp for schedule(dynamic, 4)
      for (int64_t t = 0; t < nselk; ++t) {
        int64_t kj = selk ? selk[t] : t;
        int64_t r = kj;
        int jx = (int)(r % W); r /= W;
        int jy = (int)(r % H); r /= H;
        int jz = (int)(r % Z); r /= Z;
        int h = (int)(r % heads); r /= heads;
        int b = (int)r;
        for (int e = 0; e < d; ++e) { acc[e] = 0.0; acc2[e] = 0.0; }
        const double* vj = v + kj * d;
        for (int iz = 0; iz < Z; ++iz) {
          if (!in_window(jz, iz, Z, kz)) continue;
          for (int iy = 0; iy < H; ++iy) {
            if (!in_window(jy, iy, H, ky)) continue;
            for (int ix = 0; ix < W; ++ix) {
              if (!in_window(jx, ix, W, kx)) continue;
              int64_t qi = IDX6(b, h, iz, iy, ix, heads, Z, H, W);
              double lse;
              na_query(&D, q, k, v, ph, qi, o, &lse, s, qr, kr);
              /* na_query left the rotated q of query qi in qr (when rotating). */
              const double* qv = ph ? qr : q + qi * d;
              /* position of key j inside query i's window, in window order */
              int zs = win_start(iz, Z, kz), ys = win_start(iy, H, ky), xs = win_start(ix, W, kx);
              int n = ((jz - zs) * ky + (jy - ys)) * kx + (jx - xs);
              double p = exp(s[n] - lse);
              const double* g = dout + qi * d;
              double Di = 0.0, dp = 0.0;
              for (int e = 0; e < d; ++e) { Di += g[e] * o[e]; dp += g[e] * vj[e]; }
              double ds = p * (dp - Di);
              for (int e = 0; e < d; ++e) {
                acc2[e] += p * g[e];
                acc[e] += scale * ds * qv[e];
              }
            }
          }
        }
        memcpy(dv + t * d, acc2, sizeof(double) * d);
        if (ph)
          rotate(acc, ph + (((int64_t)b * H + jy) * W + jx) * (d / 2) * 2, d, -1.0, dk + t * d);
        else
          memcpy(dk + t * d, acc, sizeof(double) * d);
      }
    }
    free(s); free(qr); free(kr); free(o); free(acc); free(acc2);
  }
  free(ph);
  return err;
}

/* ---------------------------------------------------------------------------
 * QK normalisation and gated attention (App. B.5, "QK normalization and gated
 * attention").
 *   - Every query and key vector (one token of one head, its d entries) is
 *     divided by its root mean square before the dot product, with no
 *     learnable scale:  x^ = x / sqrt(mean_e x_e^2 + eps).
 *   - The attention output of every (token, head) is multiplied by a sigmoid
 *     gate, sigmoid(g) = 1 / (1 + exp(-g)), of gate logits g given either once
 *     per (token, head) (gate_dim 1) or per channel (gate_dim d).
 * Readings where the paper is silent: eps is an argument; the norm comes
 * before the rotary embedding (a rotation keeps every pair's sum of squares,
 * so the order does not change the result); the gate logits are inputs
 * (whatever produces them lies outside attention); the lse stays that of the
 * softmax, before the gate.
 * ------------------------------------------------------------------------- */
static double sigmoid(double g) { return 1.0 / (1.0 + exp(-g)); }

/* y[i] = x[i] / sqrt(mean(x[i]^2) + eps) for every row i of n rows of d;
 * rinv[i] = 1 / sqrt(mean(x[i]^2) + eps).  Returns NULL on allocation failure. */
static double* rms_normalise(const double* x, int64_t n, int d, double eps, double* rinv) {
  double* y = (double*)malloc(sizeof(double) * (size_t)n * d);
  if (!y) return NULL;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double ss = 0.0;
    for (int e = 0; e < d; ++e) ss += x[i * d + e] * x[i * d + e];
    double r = 1.0 / sqrt(ss / d + eps);
    if (rinv) rinv[i] = r;
    for (int e = 0; e < d; ++e) y[i * d + e] = x[i * d + e] * r;
  }
  return y;
}

static double gate_logit(const double* gate, int gate_dim, int d, int64_t qi, int e) {
  return gate_dim == 1 ? gate[qi] : gate[qi * d + e];
}

static int check_options(int d, int qk_norm, double eps, const double* gate, int gate_dim) {
  if (qk_norm && !(eps >= 0.0)) return 1;
  if (gate && gate_dim != 1 && gate_dim != d) return 1;
  return 0;
}

/* Forward with the options: the neighbourhood attention above on the
 * normalised q and k (when qk_norm), then the gate on its output (when gate
 * != NULL).  Selection, outputs and errors as in oracle_na3d_fwd. */
int oracle_na3d_fwd_ex(const double* q, const double* k, const double* v, const float* coords,
                       double base, int B, int heads, int Z, int H, int W, int d, int kz, int ky,
                       int kx, double scale, int qk_norm, double eps, const double* gate,
                       int gate_dim, int64_t nsel, const int64_t* sel, double* out, double* lse) {
  if (d <= 0 || check_options(d, qk_norm, eps, gate, gate_dim)) return 1;
  int64_t nq = (int64_t)B * heads * Z * H * W;
  if (nq <= 0) return 1;
  double *qn = NULL, *kn = NULL;
  if (qk_norm) {
    qn = rms_normalise(q, nq, d, eps, NULL);
    kn = rms_normalise(k, nq, d, eps, NULL);
    if (!qn || !kn) {
      free(qn);
      free(kn);
      return 2;
    }
  }
  int rc = oracle_na3d_fwd(qk_norm ? qn : q, qk_norm ? kn : k, v, coords, base, B, heads, Z, H, W,
                           d, kz, ky, kx, scale, nsel, sel, out, lse);
  free(qn);
  free(kn);
  if (rc || !gate) return rc;
  if (!sel) nsel = nq;
  for (int64_t i = 0; i < nsel; ++i) {
    int64_t qi = sel ? sel[i] : i;
    for (int e = 0; e < d; ++e) out[i * d + e] *= sigmoid(gate_logit(gate, gate_dim, d, qi, e));
  }
  return 0;
}

/* Backward with the options, by the chain rule through the steps of the
 * forward above, for upstream gradient dO of the gated output:
 *   gate:  out = s * A with s = sigmoid(g), so dA = s * dO and
 *          dg = s (1 - s) * dO * A  (per channel; gate_dim 1 sums over e);
 *   attention: the backward above on (q^, k^, v) with upstream gradient dA,
 *          giving dq^, dk^, dv;
 *   norm:  x^ = r x with r = (mean(x^2) + eps)^(-1/2), whose Jacobian gives
 *          dx = r (dx^ - x^ mean_e(dx^_e x^_e)).
 * dq and dgate rows follow selq, dk and dv rows follow selk (NULL = all);
 * dgate (shape of gate) is written when both gate and dgate are non-NULL. */
int oracle_na3d_bwd_ex(const double* q, const double* k, const double* v, const float* coords,
                       double base, int B, int heads, int Z, int H, int W, int d, int kz, int ky,
                       int kx, double scale, int qk_norm, double eps, const double* gate,
                       int gate_dim, const double* dout, int64_t nselq, const int64_t* selq,
                       int64_t nselk, const int64_t* selk, double* dq, double* dk, double* dv,
                       double* dgate) {
  if (d <= 0 || check_options(d, qk_norm, eps, gate, gate_dim)) return 1;
  int64_t nq = (int64_t)B * heads * Z * H * W;
  if (nq <= 0) return 1;
  if (!selq) nselq = nq;
  if (!selk) nselk = nq;
  double *qn = NULL, *kn = NULL, *rq = NULL, *rk = NULL, *da = NULL, *A = NULL;
  int rc = 2;
  if (qk_norm) {
    rq = (double*)malloc(sizeof(double) * nq);
    rk = (double*)malloc(sizeof(double) * nq);
    if (!rq || !rk) goto done;
    qn = rms_normalise(q, nq, d, eps, rq);
    kn = rms_normalise(k, nq, d, eps, rk);
    if (!qn || !kn) goto done;
  }
  const double* qq = qk_norm ? qn : q;
  const double* kk = qk_norm ? kn : k;
  if (gate) {
    da = (double*)malloc(sizeof(double) * (size_t)nq * d);
    if (!da) goto done;
    for (int64_t i = 0; i < nq; ++i)
      for (int e = 0; e < d; ++e) da[i * d + e] = sigmoid(gate_logit(gate, gate_dim, d, i, e)) * dout[i * d + e];
  }
  rc = oracle_na3d_bwd(qq, kk, v, coords, base, B, heads, Z, H, W, d, kz, ky, kx, scale,
                       gate ? da : dout, nselq, selq, nselk, selk, dq, dk, dv);
  if (rc) goto done;
  if (qk_norm) {
    for (int64_t i = 0; i < nselq; ++i) {
      int64_t qi = selq ? selq[i] : i;
      double c = 0.0;
      for (int e = 0; e < d; ++e) c += dq[i * d + e] * qn[qi * d + e];
      c /= d;
      for (int e = 0; e < d; ++e) dq[i * d + e] = rq[qi] * (dq[i * d + e] - qn[qi * d + e] * c);
    }
    for (int64_t t = 0; t < nselk; ++t) {
      int64_t kj = selk ? selk[t] : t;
      double c = 0.0;
      for (int e = 0; e < d; ++e) c += dk[t * d + e] * kn[kj * d + e];
      c /= d;
      for (int e = 0; e < d; ++e) dk[t * d + e] = rk[kj] * (dk[t * d + e] - kn[kj * d + e] * c);
    }
  }
  if (gate && dgate) {
    /* the ungated attention output A of the selected queries */
    A = (double*)malloc(sizeof(double) * (size_t)nselq * d);
    if (!A) {
      rc = 2;
      goto done;
    }
    rc = oracle_na3d_fwd(qq, kk, v, coords, base, B, heads, Z, H, W, d, kz, ky, kx, scale,
                         nselq, selq, A, NULL);
    if (rc) goto done;
    for (int64_t i = 0; i < nselq; ++i) {
      int64_t qi = selq ? selq[i] : i;
      if (gate_dim == 1) {
        double s = sigmoid(gate[qi]), acc = 0.0;
        for (int e = 0; e < d; ++e) acc += dout[qi * d + e] * A[i * d + e];
        dgate[i] = s * (1.0 - s) * acc;
      } else {
        for (int e = 0; e < d; ++e) {
          double s = sigmoid(gate[qi * d + e]);
          dgate[i * d + e] = s * (1.0 - s) * dout[qi * d + e] * A[i * d + e];
        }
      }
    }
  }
done:
  free(qn);
  free(kn);
  free(rq);
  free(rk);
  free(da);
  free(A);
  return rc;
}

/* ---------------------------------------------------------------------------
 * Tile stitching S = D^-1 P^T W (App. F).  On a regular tiling, tile (a, b)
 * has origin (a*stride_y, b*stride_x); P^T W sums, for every face cell, the
 * window-weighted values of the tiles that cover it, D sums the weights, and
 * the output is their quotient.  A cell no tile weights (D == 0) is 0.
 *
 * Operation order (fixed so that results are reproducible bit for bit):
 * tiles in ascending a, then ascending b; acc = fma(w, value, acc) and
 * D = D + w from 0; out = acc / D correctly rounded.  bf16 data accumulate
 * in float32 and round the quotient to bf16 (nearest-even); float32 data
 * accumulate in float64 and round the quotient to float32.
 * ------------------------------------------------------------------------- */
static uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static float bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static int blend_args(int nty, int ntx, int P, int Ht, int Wt, int C, int sy, int sx, int Hf, int Wf) {
  if (nty <= 0 || ntx <= 0 || P <= 0 || Ht <= 0 || Wt <= 0 || C <= 0 || sy <= 0 || sx <= 0)
    return 1;
  if (Hf <= 0 || Wf <= 0) return 1;
  if ((int64_t)(nty - 1) * sy + Ht > Hf || (int64_t)(ntx - 1) * sx + Wt > Wf) return 1;
  return 0;
}

int oracle_tile_blend(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C,
                      int sy, int sx, const float* window, void* out, int Hf, int Wf,
                      int is_bf16) {
  if (blend_args(nty, ntx, P, Ht, Wt, C, sy, sx, Hf, Wf)) return 1;
#pragma omp parallel for collapse(2) schedule(static)
  for (int p = 0; p < P; ++p)
    for (int y = 0; y < Hf; ++y)
      for (int x = 0; x < Wf; ++x)
        for (int c = 0; c < C; ++c) {
          int64_t o = (((int64_t)p * Hf + y) * Wf + x) * C + c;
          if (is_bf16) {
            float acc = 0.0f, Dw = 0.0f;
            for (int a = 0; a < nty; ++a) {
              int ly = y - a * sy;
              if (ly < 0 || ly >= Ht) continue;
              for (int b = 0; b < ntx; ++b) {
                int lx = x - b * sx;
                if (lx < 0 || lx >= Wt) continue;
                int64_t t = (int64_t)a * ntx + b;
                float w = window[ly * Wt + lx];
                float val = bf16_to_f32(((const uint16_t*)tiles)[(((t * P + p) * Ht + ly) * Wt + lx) * C + c]);
                acc = fmaf(w, val, acc);
                Dw = Dw + w;
              }
            }
            float r = (Dw == 0.0f) ? 0.0f : acc / Dw;
            ((uint16_t*)out)[o] = f32_to_bf16_rne(r);
          } else {
            double acc = 0.0, Dw = 0.0;
            for (int a = 0; a < nty; ++a) {
              int ly = y - a * sy;
              if (ly < 0 || ly >= Ht) continue;
              for (int b = 0; b < ntx; ++b) {
                int lx = x - b * sx;
                if (lx < 0 || lx >= Wt) continue;
                int64_t t = (int64_t)a * ntx + b;
                double w = (double)window[ly * Wt + lx];
                double val = (double)((const float*)tiles)[(((t * P + p) * Ht + ly) * Wt + lx) * C + c];
                acc = fma(w, val, acc);
                Dw = Dw + w;
              }
            }
            double r = (Dw == 0.0) ? 0.0 : acc / Dw;
            ((float*)out)[o] = (float)r;
          }
        }
  return 0;
}

/* Tile extraction P on a regular tiling (the inverse direction of the blend):
 * tiles[t, p, i, j, c] = face[p, a*stride_y + i, b*stride_x + j, c], t = a*ntx + b. */
int oracle_tile_extract(const void* face, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                        int sx, int Hf, int Wf, void* tiles, int elem_bytes) {
  if (blend_args(nty, ntx, P, Ht, Wt, C, sy, sx, Hf, Wf)) return 1;
  if (elem_bytes != 2 && elem_bytes != 4) return 1;
  for (int a = 0; a < nty; ++a)
    for (int b = 0; b < ntx; ++b)
      for (int p = 0; p < P; ++p)
        for (int i = 0; i < Ht; ++i)
          for (int j = 0; j < Wt; ++j) {
            int64_t t = (int64_t)a * ntx + b;
            int64_t dst = (((t * P + p) * Ht + i) * Wt + j) * C;
            int64_t src = (((int64_t)p * Hf + (a * sy + i)) * Wf + (b * sx + j)) * C;
            memcpy((char*)tiles + dst * elem_bytes, (const char*)face + src * elem_bytes,
                   (size_t)C * elem_bytes);
          }
  return 0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Thread count of the OpenMP loops that follow (timing runs on one core). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  extern void omp_set_num_threads(int);
  omp_set_num_threads(n > 0 ? n : 1);
#else
  (void)n;
#endif
}

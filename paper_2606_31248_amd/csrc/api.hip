// The C ABI of libstrata: argument validation, kernel selection, error reporting.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "common.h"
#include "kernels.h"

namespace strata {

static thread_local char g_err[512] = "";

strata_status set_error(strata_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

strata_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(STRATA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return STRATA_OK;
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE(cond, ...)                                          \
  do {                                                              \
    if (!(cond)) return set_error(STRATA_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)

#define REQUIRE_PTR(p)                                                              \
  do {                                                                              \
    if (!(p)) return set_error(STRATA_ERR_INVALID_ARG, "%s: null pointer", #p);     \
    if (!aligned16(p)) return set_error(STRATA_ERR_INVALID_ARG, "%s: not 16-byte aligned", #p); \
  } while (0)

static const int64_t kMaxElems = (int64_t)1 << 40;

// odd and inside the axis, or the whole axis (any parity)
static bool window_ok(int L, int k) { return k > 0 && k <= L && ((k & 1) || k == L); }

static strata_status check_desc(const strata_na3d_desc* d) {
  REQUIRE(d, "desc: null pointer");
  REQUIRE(d->B > 0 && d->heads > 0 && d->Z > 0 && d->H > 0 && d->W > 0 && d->head_dim > 0,
          "desc: every size must be positive (B=%d heads=%d Z=%d H=%d W=%d head_dim=%d)", d->B,
          d->heads, d->Z, d->H, d->W, d->head_dim);
  REQUIRE(d->kz > 0 && d->ky > 0 && d->kx > 0, "desc: window sizes must be positive (%d, %d, %d)", d->kz,
          d->ky, d->kx);
  REQUIRE(d->kz <= d->Z && d->ky <= d->H && d->kx <= d->W,
          "desc: window (%d, %d, %d) larger than the grid (%d, %d, %d)", d->kz, d->ky, d->kx, d->Z,
          d->H, d->W);
  REQUIRE(window_ok(d->Z, d->kz) && window_ok(d->H, d->ky) && window_ok(d->W, d->kx),
          "desc: window sizes must be odd or span their whole axis (%d, %d, %d) on (%d, %d, %d)", d->kz,
          d->ky, d->kx, d->Z, d->H, d->W);
  REQUIRE(d->scale > 0.f && isfinite(d->scale), "desc: scale must be finite and > 0");
  REQUIRE(d->dtype == STRATA_F32 || d->dtype == STRATA_BF16, "desc: unknown dtype %d", (int)d->dtype);
  int64_t n = (int64_t)d->B * d->heads * d->Z * d->H * d->W;
  REQUIRE(n * d->head_dim < kMaxElems, "desc: tensor too large");
  if (d->head_dim != 32 && d->head_dim != 64 && d->head_dim != 128)
    return set_error(STRATA_ERR_UNSUPPORTED, "head_dim %d not supported (32, 64 or 128)", d->head_dim);
  return STRATA_OK;
}

// Options of the attention block; NULL = plain attention.
static strata_status check_opts(const strata_na3d_desc* d, const strata_na3d_opts* o, NaOpts& out) {
  out = NaOpts{};
  if (!o) return STRATA_OK;
  if (o->qk_norm) {
    REQUIRE(isfinite(o->eps) && o->eps >= 0.f, "opts: eps must be finite and >= 0");
    out.qk_norm = 1;
    out.eps = o->eps;
  }
  if (o->gate) {
    REQUIRE(o->gate_dim == 1 || o->gate_dim == d->head_dim,
            "opts: gate_dim must be 1 or head_dim (%d), got %d", d->head_dim, o->gate_dim);
    REQUIRE(aligned16(o->gate), "opts.gate: not 16-byte aligned");
    out.gate = o->gate;
    out.gate_dim = o->gate_dim;
  }
  return STRATA_OK;
}

// Backward workspace: D, the per-(batch, head) exponent of the largest |dO|,
// then (with a gate) dA = sigmoid(g) dO as its rounded value hi and, for bf16,
// the remainder lo; every region starts on a 256-byte boundary.
struct BwdLayout {
  size_t dvec, emax, da_hi, da_lo, total;
};

static BwdLayout bwd_layout(const strata_na3d_desc& d, const NaOpts& o) {
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t n = (size_t)d.B * d.heads * d.Z * d.H * d.W;
  const size_t rowb = n * d.head_dim * (d.dtype == STRATA_BF16 ? 2 : 4);
  BwdLayout L = {};
  size_t off = al(n * sizeof(float));
  L.emax = off;
  off += al((size_t)d.B * d.heads * sizeof(int));
  L.da_hi = off;
  if (o.gate) off += al(rowb);
  L.da_lo = off;
  if (o.gate && d.dtype == STRATA_BF16) off += al(rowb);
  L.total = off;
  return L;
}

// the forward kernel for the problem's shape
static void launch_fwd(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k, const void* v,
                       const float* cs, void* out, float* lse, hipStream_t s) {
  if (!launch_na3d_fwd_col(d, o, q, k, v, out, lse, s) && !launch_na3d_fwd_zs(d, o, q, k, v, cs, out, lse, s) &&
      !launch_na3d_fwd_lsg(d, o, q, k, v, cs, out, lse, s) && !launch_na3d_fwd_mfma(d, o, q, k, v, cs, out, lse, s) &&
      !launch_na3d_fwd_d128(d, o, q, k, v, cs, out, lse, s))
    launch_na3d_fwd_ref(d, o, q, k, v, cs, out, lse, s);
}

static strata_status na3d_fwd_impl(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                   const void* q, const void* k, const void* v, const float* cs,
                                   void* out, float* lse, void* stream) {
  strata_status st = check_desc(desc);
  if (st != STRATA_OK) return st;
  NaOpts o;
  st = check_opts(desc, opts, o);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(q);
  REQUIRE_PTR(k);
  REQUIRE_PTR(v);
  REQUIRE_PTR(out);
  if (cs) REQUIRE(aligned16(cs), "cs: not 16-byte aligned");
  if (lse) REQUIRE(aligned16(lse), "lse: not 16-byte aligned");
  launch_fwd(*desc, o, q, k, v, cs, out, lse, (hipStream_t)stream);
  return check_launch(opts ? "strata_na3d_fwd_ex" : "strata_na3d_fwd");
}

static size_t bwd_workspace_impl(const strata_na3d_desc* desc, const strata_na3d_opts* opts) {
  NaOpts o;
  if (!desc || check_desc(desc) != STRATA_OK || check_opts(desc, opts, o) != STRATA_OK) return 0;
  return bwd_layout(*desc, o).total;
}

// The backward's kernels after the arguments have been checked: D (and, with a
// gate, dA) live in `ws`, laid out as bwd_layout says.
static strata_status na3d_bwd_launch(const strata_na3d_desc* desc, const strata_na3d_opts* opts, const NaOpts& o,
                                     const void* q, const void* k, const void* v, const float* cs, const void* out,
                                     const void* dout, const float* lse, void* dq, void* dk, void* dv, void* dgate,
                                     char* ws, hipStream_t s);

static strata_status na3d_bwd_impl(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                   const void* q, const void* k, const void* v, const float* cs,
                                   const void* out, const void* dout, const float* lse, void* dq,
                                   void* dk, void* dv, void* dgate, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  strata_status st = check_desc(desc);
  if (st != STRATA_OK) return st;
  NaOpts o;
  st = check_opts(desc, opts, o);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(q);
  REQUIRE_PTR(k);
  REQUIRE_PTR(v);
  REQUIRE_PTR(out);
  REQUIRE_PTR(dout);
  REQUIRE_PTR(lse);
  REQUIRE_PTR(dq);
  REQUIRE_PTR(dk);
  REQUIRE_PTR(dv);
  if (o.gate) REQUIRE_PTR(dgate);
  if (cs) REQUIRE(aligned16(cs), "cs: not 16-byte aligned");
  const BwdLayout L = bwd_layout(*desc, o);
  if (!workspace || workspace_bytes < L.total)
    return set_error(STRATA_ERR_WORKSPACE, "workspace: need %zu bytes, got %zu", L.total,
                     workspace ? workspace_bytes : (size_t)0);
  REQUIRE(aligned16(workspace), "workspace: not 16-byte aligned");
  return na3d_bwd_launch(desc, opts, o, q, k, v, cs, out, dout, lse, dq, dk, dv, dgate, static_cast<char*>(workspace),
                         (hipStream_t)stream);
}

static strata_status na3d_bwd_launch(const strata_na3d_desc* desc, const strata_na3d_opts* opts, const NaOpts& o,
                                     const void* q, const void* k, const void* v, const float* cs, const void* out,
                                     const void* dout, const float* lse, void* dq, void* dk, void* dv, void* dgate,
                                     char* ws, hipStream_t s) {
  const BwdLayout L = bwd_layout(*desc, o);
  float* dvec = reinterpret_cast<float*>(ws + L.dvec);
  // the attention backward runs with upstream gradient dA (dO without a gate);
  // QK RMSNorm happens inside its kernels
  BwdOpts bo;
  bo.qk_norm = o.qk_norm;
  bo.eps = o.eps;
  const void* ga = dout;
  // D = rowsum(dO * O): from the gate's pass, from the MFMA dq pass (which reads
  // O beside the dO rows it loads anyway), or from a pass of its own
  const bool fuse_d = !o.gate && na3d_bwd_dq_mfma_takes(*desc);
  if (o.gate) {
    void* lo = desc->dtype == STRATA_BF16 ? ws + L.da_lo : nullptr;
    launch_na3d_bwd_gate_prep(*desc, o, out, dout, dvec, ws + L.da_hi, lo, dgate, s);
    ga = ws + L.da_hi;
    bo.dout_lo = lo;
  } else if (!fuse_d) {
    launch_na3d_bwd_ref(0, *desc, bo, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
  }
  if (launch_na3d_bwd_col(*desc, bo, q, k, v, ga, lse, dvec, dq, dk, dv, s))
    return check_launch(opts ? "strata_na3d_bwd_ex" : "strata_na3d_bwd");
  // the MFMA dq pass also records the largest |dO| exponent per (batch, head)
  // when the balanced dk/dv pass, which scales its float16 copy of dO by it,
  // takes the problem
  int* emax = na3d_bwd_dkdv_kvp_takes(*desc, bo) ? reinterpret_cast<int*>(ws + L.emax) : nullptr;
  if (!launch_na3d_bwd_dq_mfma(*desc, bo, q, k, v, cs, ga, lse, dvec, fuse_d ? out : nullptr, emax, dq, s)) {
    emax = nullptr;
    if (fuse_d) launch_na3d_bwd_ref(0, *desc, bo, q, k, v, cs, out, dout, lse, dq, dk, dv, dvec, s);
    if (!launch_na3d_bwd_dq_d128(*desc, bo, q, k, v, cs, ga, lse, dvec, dq, s))
      launch_na3d_bwd_ref(1, *desc, bo, q, k, v, cs, out, ga, lse, dq, dk, dv, dvec, s);
  }
  if (!launch_na3d_bwd_dkdv_kvp(*desc, bo, q, k, v, cs, ga, lse, dvec, emax, dk, dv, s) &&
      !launch_na3d_bwd_dkdv_mfma(*desc, bo, q, k, v, cs, ga, lse, dvec, dk, dv, s) &&
      !launch_na3d_bwd_dkdv_d128(*desc, bo, q, k, v, cs, ga, lse, dvec, dk, dv, s))
    launch_na3d_bwd_ref(2, *desc, bo, q, k, v, cs, out, ga, lse, dq, dk, dv, dvec, s);
  return check_launch(opts ? "strata_na3d_bwd_ex" : "strata_na3d_bwd");
}

// ---- backward without a caller workspace ---------------------------------------
// D = rowsum(dO * O) of a plain backward and the per-(batch, head) exponent of
// the largest |dO| live in this file-scope device array instead of a
// workspace: every device the library runs on holds its own copy for the life
// of the process.  In host code `scratch` only names the symbol;
// its device address is looked up once per device (hipGetSymbolAddress, with
// the device current) and that address is what the kernels receive.
constexpr int64_t kMaxTokenHeads = (int64_t)1 << 23, kMaxBatchHeads = (int64_t)1 << 16;
constexpr int64_t kScratchFloats = kMaxTokenHeads + kMaxBatchHeads;  // 32 MiB + 256 KiB
static __device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 64;
static std::once_flag g_scratch_once[kMaxDevices];
static float* g_scratch_ptr[kMaxDevices];
static hipError_t g_scratch_err[kMaxDevices];

// this device's copy of `scratch`, or nullptr (with the HIP error in *err)
static float* device_scratch(int dev, hipError_t* err) {
  std::call_once(g_scratch_once[dev], [dev] {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? static_cast<float*>(p) : nullptr;
  });
  *err = g_scratch_err[dev];
  return g_scratch_ptr[dev];
}

static strata_status na3d_bwd_noalloc_impl(const strata_na3d_desc* desc, const void* q, const void* k,
                                           const void* v, const float* cs, const void* out, const void* dout,
                                           const float* lse, void* dq, void* dk, void* dv, void* stream) {
  strata_status st = check_desc(desc);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(q);
  REQUIRE_PTR(k);
  REQUIRE_PTR(v);
  REQUIRE_PTR(out);
  REQUIRE_PTR(dout);
  REQUIRE_PTR(lse);
  REQUIRE_PTR(dq);
  REQUIRE_PTR(dk);
  REQUIRE_PTR(dv);
  if (cs) REQUIRE(aligned16(cs), "cs: not 16-byte aligned");
  const int64_t bh = (int64_t)desc->B * desc->heads, n = bh * desc->Z * desc->H * desc->W;
  REQUIRE(n <= kMaxTokenHeads && bh <= kMaxBatchHeads,
          "bwd_noalloc: %lld token-heads (%lld batch-heads) exceed the static scratch of %lld (%lld) (use "
          "strata_na3d_bwd with a workspace)",
          (long long)n, (long long)bh, (long long)kMaxTokenHeads, (long long)kMaxBatchHeads);
  const NaOpts o;
  REQUIRE(bwd_layout(*desc, o).total <= (size_t)kScratchFloats * sizeof(float), "bwd_noalloc: static scratch layout");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(STRATA_ERR_HIP, "bwd_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(STRATA_ERR_UNSUPPORTED, "bwd_noalloc: device %d beyond the %d this build tracks", dev,
                     kMaxDevices);
  float* ws = device_scratch(dev, &e);
  if (!ws) return set_error(STRATA_ERR_HIP, "bwd_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
  return na3d_bwd_launch(desc, nullptr, o, q, k, v, cs, out, dout, lse, dq, dk, dv, nullptr,
                         reinterpret_cast<char*>(ws), (hipStream_t)stream);
}

}  // namespace strata

using namespace strata;

extern "C" {

const char* strata_status_string(strata_status st) {
  switch (st) {
    case STRATA_OK: return "ok";
    case STRATA_ERR_INVALID_ARG: return "invalid argument";
    case STRATA_ERR_UNSUPPORTED: return "unsupported";
    case STRATA_ERR_WORKSPACE: return "workspace too small";
    case STRATA_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* strata_last_error(void) { return g_err; }

strata_status strata_na_axis_index(int32_t L, int32_t k, int32_t* starts, int32_t* qlo,
                                   int32_t* qhi, void* stream) {
  REQUIRE(L > 0 && window_ok(L, k), "axis: need odd 1 <= k <= L or k == L (L=%d, k=%d)", L, k);
  REQUIRE_PTR(starts);
  REQUIRE_PTR(qlo);
  REQUIRE_PTR(qhi);
  launch_axis_index(L, k, starts, qlo, qhi, (hipStream_t)stream);
  return check_launch("strata_na_axis_index");
}

strata_status strata_stereo_coords(const int32_t* tile_face, const int32_t* tile_oy,
                                   const int32_t* tile_ox, int32_t B, int32_t H, int32_t W,
                                   int32_t face_cells, int32_t patch, double l_scale,
                                   float* coords, void* stream) {
  REQUIRE(B > 0 && H > 0 && W > 0, "coords: sizes must be positive");
  REQUIRE(face_cells > 0 && patch > 0 && face_cells % patch == 0,
          "coords: face_cells must be a positive multiple of patch");
  REQUIRE(H * (int64_t)patch <= face_cells && W * (int64_t)patch <= face_cells,
          "coords: tile larger than the face");
  REQUIRE(l_scale == 0.0 || (l_scale > 0.0 && isfinite(l_scale)), "coords: l_scale must be 0 or finite and > 0");
  // Eq. 1's length sqrt(4 pi / N_total), N_total = the native cells of the six faces
  if (l_scale == 0.0) l_scale = sqrt(4.0 * M_PI / (6.0 * (double)face_cells * (double)face_cells));
  REQUIRE_PTR(tile_face);
  REQUIRE_PTR(tile_oy);
  REQUIRE_PTR(tile_ox);
  REQUIRE_PTR(coords);
  launch_stereo_coords(tile_face, tile_oy, tile_ox, B, H, W, face_cells, patch, l_scale, coords,
                       (hipStream_t)stream);
  return check_launch("strata_stereo_coords");
}

strata_status strata_wind_tile_frame(const void* field, int32_t face, int32_t face_cells, int32_t nty,
                                     int32_t ntx, int32_t P, int32_t Ht, int32_t Wt, int32_t stride_y,
                                     int32_t stride_x, void* tiles, strata_dtype dtype, void* stream) {
  REQUIRE(face >= 0 && face < 6, "wind: face %d not in 0..5", face);
  REQUIRE(face_cells > 0 && nty > 0 && ntx > 0 && P > 0 && Ht > 0 && Wt > 0 && stride_y > 0 && stride_x > 0,
          "wind: sizes and strides must be positive");
  REQUIRE((int64_t)(nty - 1) * stride_y + Ht <= face_cells && (int64_t)(ntx - 1) * stride_x + Wt <= face_cells,
          "wind: tiles extend past the face");
  REQUIRE(dtype == STRATA_F32 || dtype == STRATA_BF16, "wind: unknown dtype %d", (int)dtype);
  REQUIRE((int64_t)P * face_cells * face_cells * 2 < kMaxElems &&
              (int64_t)nty * ntx * P * Ht * Wt * 2 < kMaxElems && (int64_t)nty * ntx * Ht * Wt < ((int64_t)1 << 31) * 256,
          "wind: tensor too large");
  REQUIRE_PTR(field);
  REQUIRE_PTR(tiles);
  launch_wind_tile_frame(field, face, face_cells, nty, ntx, P, Ht, Wt, stride_y, stride_x, tiles, dtype,
                         (hipStream_t)stream);
  return check_launch("strata_wind_tile_frame");
}

strata_status strata_stereorope_phases(const float* coords, int32_t B, int32_t H, int32_t W,
                                       int32_t head_dim, double base, float* cs, void* stream) {
  REQUIRE(B > 0 && H > 0 && W > 0, "phases: sizes must be positive");
  REQUIRE(head_dim > 0 && head_dim % 4 == 0, "phases: head_dim %d must be a positive multiple of 4",
          head_dim);
  REQUIRE(base > 0.0 && isfinite(base), "phases: base must be finite and > 0");
  REQUIRE_PTR(coords);
  REQUIRE_PTR(cs);
  launch_rope_phases(coords, B, H, W, head_dim, base, cs, (hipStream_t)stream);
  return check_launch("strata_stereorope_phases");
}

strata_status strata_stereorope_apply(const void* x, void* y, const float* cs, int32_t B,
                                      int32_t heads, int32_t Z, int32_t H, int32_t W,
                                      int32_t head_dim, strata_dtype dtype, int32_t transpose,
                                      void* stream) {
  REQUIRE(B > 0 && heads > 0 && Z > 0 && H > 0 && W > 0 && head_dim > 0,
          "rope: sizes must be positive");
  REQUIRE(head_dim % 4 == 0, "rope: head_dim %d must be a multiple of 4", head_dim);
  REQUIRE(dtype == STRATA_F32 || dtype == STRATA_BF16, "rope: unknown dtype %d", (int)dtype);
  REQUIRE((int64_t)B * heads * Z * H * W * head_dim < kMaxElems, "rope: tensor too large");
  REQUIRE_PTR(x);
  REQUIRE_PTR(y);
  REQUIRE_PTR(cs);
  if (head_dim % 8 != 0)
    return set_error(STRATA_ERR_UNSUPPORTED, "rope: head_dim %d not a multiple of 8", head_dim);
  launch_rope_apply(x, y, cs, B, heads, Z, H, W, head_dim, dtype, transpose, (hipStream_t)stream);
  return check_launch("strata_stereorope_apply");
}

strata_status strata_na3d_fwd(const strata_na3d_desc* desc, const void* q, const void* k,
                              const void* v, const float* cs, void* out, float* lse,
                              void* stream) {
  return na3d_fwd_impl(desc, nullptr, q, k, v, cs, out, lse, stream);
}

strata_status strata_na3d_fwd_ex(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                 const void* q, const void* k, const void* v, const float* cs,
                                 void* out, float* lse, void* stream) {
  return na3d_fwd_impl(desc, opts, q, k, v, cs, out, lse, stream);
}

size_t strata_na3d_bwd_workspace_size(const strata_na3d_desc* desc) {
  return bwd_workspace_impl(desc, nullptr);
}

size_t strata_na3d_bwd_ex_workspace_size(const strata_na3d_desc* desc,
                                         const strata_na3d_opts* opts) {
  return bwd_workspace_impl(desc, opts);
}

strata_status strata_na3d_bwd(const strata_na3d_desc* desc, const void* q, const void* k,
                              const void* v, const float* cs, const void* out, const void* dout,
                              const float* lse, void* dq, void* dk, void* dv, void* workspace,
                              size_t workspace_bytes, void* stream) {
  return na3d_bwd_impl(desc, nullptr, q, k, v, cs, out, dout, lse, dq, dk, dv, nullptr, workspace,
                       workspace_bytes, stream);
}

strata_status strata_na3d_bwd_ex(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                 const void* q, const void* k, const void* v, const float* cs,
                                 const void* out, const void* dout, const float* lse, void* dq,
                                 void* dk, void* dv, void* dgate, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  return na3d_bwd_impl(desc, opts, q, k, v, cs, out, dout, lse, dq, dk, dv, dgate, workspace,
                       workspace_bytes, stream);
}

strata_status strata_na3d_bwd_noalloc(const strata_na3d_desc* desc, const void* q, const void* k, const void* v,
                                      const float* cs, const void* out, const void* dout, const float* lse, void* dq,
                                      void* dk, void* dv, void* stream) {
  return na3d_bwd_noalloc_impl(desc, q, k, v, cs, out, dout, lse, dq, dk, dv, stream);
}

static strata_status check_tiling(int32_t nty, int32_t ntx, int32_t P, int32_t Ht, int32_t Wt,
                                  int32_t C, int32_t sy, int32_t sx, int32_t Hf, int32_t Wf,
                                  strata_dtype dt) {
  REQUIRE(nty > 0 && ntx > 0 && P > 0 && Ht > 0 && Wt > 0 && C > 0 && sy > 0 && sx > 0 && Hf > 0 &&
              Wf > 0,
          "tiling: sizes and strides must be positive");
  REQUIRE((int64_t)(nty - 1) * sy + Ht <= Hf && (int64_t)(ntx - 1) * sx + Wt <= Wf,
          "tiling: tiles extend past the face ((%d-1)*%d+%d > %d or (%d-1)*%d+%d > %d)", nty, sy, Ht,
          Hf, ntx, sx, Wt, Wf);
  REQUIRE(dt == STRATA_F32 || dt == STRATA_BF16, "tiling: unknown dtype %d", (int)dt);
  REQUIRE((int64_t)nty * ntx * P * Ht * Wt * C < kMaxElems &&
              (int64_t)P * Hf * Wf * C < kMaxElems,
          "tiling: tensor too large");
  return STRATA_OK;
}

strata_status strata_tile_blend(const void* tiles, int32_t nty, int32_t ntx, int32_t P,
                                int32_t Ht, int32_t Wt, int32_t C, int32_t stride_y,
                                int32_t stride_x, const float* window, void* out, int32_t Hf,
                                int32_t Wf, strata_dtype dtype, void* stream) {
  strata_status st = check_tiling(nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf, dtype);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(tiles);
  REQUIRE_PTR(window);
  REQUIRE_PTR(out);
  // one block per 256 items of a face row: the grid and in-row indices are 32-bit
  REQUIRE((int64_t)Wf * C < ((int64_t)1 << 31) &&
              (int64_t)P * Hf * (((int64_t)Wf * C + 255) / 256) < ((int64_t)1 << 31),
          "tile_blend: face too large for one launch");
  launch_tile_blend(tiles, nty, ntx, P, Ht, Wt, C, stride_y, stride_x, window, out, Hf, Wf, dtype,
                    (hipStream_t)stream);
  return check_launch("strata_tile_blend");
}

// A bf16 tiling whose overlap cells the overlap-only stitch handles: the tiles
// cover the face, and no cell lies in more than two tiles along an axis.
static bool overlap_form(int32_t nty, int32_t ntx, int32_t Ht, int32_t Wt, int32_t C, int32_t sy, int32_t sx,
                         int32_t Hf, int32_t Wf, strata_dtype dt) {
  return dt == STRATA_BF16 && C % 8 == 0 && sy <= Ht && Ht <= 2 * sy && sx <= Wt && Wt <= 2 * sx &&
         (int64_t)(nty - 1) * sy + Ht == Hf && (int64_t)(ntx - 1) * sx + Wt == Wf;
}

strata_status strata_tile_blend_overlap(const void* tiles, int32_t nty, int32_t ntx, int32_t P, int32_t Ht,
                                        int32_t Wt, int32_t C, int32_t stride_y, int32_t stride_x,
                                        const float* window, void* out, int32_t Hf, int32_t Wf,
                                        strata_dtype dtype, void* stream) {
  strata_status st = check_tiling(nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf, dtype);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(tiles);
  REQUIRE_PTR(window);
  REQUIRE_PTR(out);
  REQUIRE((int64_t)Wf * C < ((int64_t)1 << 31) &&
              (int64_t)P * Hf * (((int64_t)Wf * C + 255) / 256) < ((int64_t)1 << 31),
          "tile_blend_overlap: face too large for one launch");
  if (overlap_form(nty, ntx, Ht, Wt, C, stride_y, stride_x, Hf, Wf, dtype))
    launch_tile_blend_overlap(tiles, nty, ntx, P, Ht, Wt, C, stride_y, stride_x, window, out, Hf, Wf,
                              (hipStream_t)stream);
  else
    launch_tile_blend(tiles, nty, ntx, P, Ht, Wt, C, stride_y, stride_x, window, out, Hf, Wf, dtype,
                      (hipStream_t)stream);
  return check_launch("strata_tile_blend_overlap");
}

strata_status strata_na3d_fwd_stitch(const strata_na3d_desc* desc, const strata_na3d_opts* opts, const void* q,
                                     const void* k, const void* v, const float* cs, void* tiles, float* lse,
                                     int32_t nty, int32_t ntx, int32_t stride_y, int32_t stride_x,
                                     const float* window, void* face, int32_t Hf, int32_t Wf, void* stream) {
  strata_status st = check_desc(desc);
  if (st != STRATA_OK) return st;
  NaOpts o;
  st = check_opts(desc, opts, o);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(q);
  REQUIRE_PTR(k);
  REQUIRE_PTR(v);
  REQUIRE_PTR(tiles);
  REQUIRE_PTR(window);
  REQUIRE_PTR(face);
  if (cs) REQUIRE(aligned16(cs), "cs: not 16-byte aligned");
  if (lse) REQUIRE(aligned16(lse), "lse: not 16-byte aligned");
  REQUIRE((int64_t)nty * ntx == desc->B, "fwd_stitch: the batch (%d tiles) is not the %d x %d tiling", desc->B,
          nty, ntx);
  REQUIRE((int64_t)desc->heads * desc->Z < ((int64_t)1 << 31), "fwd_stitch: heads * Z planes exceed 32 bits");
  const int32_t P = desc->heads * desc->Z, Ht = desc->H, Wt = desc->W, C = desc->head_dim;
  st = check_tiling(nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf, desc->dtype);
  if (st != STRATA_OK) return st;
  REQUIRE((int64_t)Wf * C < ((int64_t)1 << 31) &&
              (int64_t)P * Hf * (((int64_t)Wf * C + 255) / 256) < ((int64_t)1 << 31),
          "fwd_stitch: face too large for one launch");
  hipStream_t s = (hipStream_t)stream;
  const StitchArgs sa = {face, window, nty, ntx, stride_y, stride_x, Hf, Wf};
  const bool fused = overlap_form(nty, ntx, Ht, Wt, C, stride_y, stride_x, Hf, Wf, desc->dtype) &&
                     launch_na3d_fwd_zs(*desc, o, q, k, v, cs, tiles, lse, s, &sa);
  if (!fused) {  // every tile output, then the whole stitch
    launch_fwd(*desc, o, q, k, v, cs, tiles, lse, s);
    launch_tile_blend(tiles, nty, ntx, P, Ht, Wt, C, stride_y, stride_x, window, face, Hf, Wf, desc->dtype, s);
  }
  return check_launch("strata_na3d_fwd_stitch");
}

strata_status strata_duo_pad(const void* faces, int32_t P, int32_t n, int32_t C, int32_t halo, void* padded,
                             strata_dtype dtype, void* stream) {
  REQUIRE(P > 0 && C > 0, "duo: P and C must be positive");
  REQUIRE(n >= 16 && halo > 0 && halo <= n / 4, "duo: need n >= 16 and 1 <= halo <= n/4 (n=%d, halo=%d)", n, halo);
  REQUIRE(dtype == STRATA_F32 || dtype == STRATA_BF16, "duo: unknown dtype %d", (int)dtype);
  const int64_t m = (int64_t)n + 2 * halo;
  REQUIRE(6LL * P * m * m * C < kMaxElems, "duo: tensor too large");
  // one block per interior row plus one per 256 halo cells
  REQUIRE(6LL * P * n + (6 * (m * m - (int64_t)n * n) + 255) / 256 < INT32_MAX, "duo: too many rows (P*n=%lld)",
          (long long)P * n);
  REQUIRE_PTR(faces);
  REQUIRE_PTR(padded);
  launch_duo_pad(faces, P, n, C, halo, padded, dtype, (hipStream_t)stream);
  return check_launch("strata_duo_pad");
}

// the plan packs a cell of a (padded) face in 28 bits and counts transposed
// entries with int32
static bool duo_plan_fits(int32_t n, int32_t halo) {
  const int64_t m = (int64_t)n + 2 * halo;
  return m < (1 << 14) && 4 * 6 * (m * m - (int64_t)n * n) < INT32_MAX;
}

size_t strata_duo_plan_bytes(int32_t n, int32_t halo) {
  if (n < 16 || halo < 1 || halo > n / 4 || !duo_plan_fits(n, halo)) return 0;
  return (size_t)duo_plan_bytes(n, halo);
}

strata_status strata_duo_plan(int32_t n, int32_t halo, void* plan, size_t plan_bytes, void* stream) {
  REQUIRE(n >= 16 && halo > 0 && halo <= n / 4, "duo plan: need n >= 16 and 1 <= halo <= n/4 (n=%d, halo=%d)", n,
          halo);
  REQUIRE(duo_plan_fits(n, halo), "duo plan: n=%d too large for a plan", n);
  REQUIRE_PTR(plan);
  REQUIRE(reinterpret_cast<uintptr_t>(plan) % 16 == 0, "duo plan: plan must be 16-byte aligned");
  REQUIRE(plan_bytes >= (size_t)duo_plan_bytes(n, halo), "duo plan: plan_bytes %zu < %lld", plan_bytes,
          (long long)duo_plan_bytes(n, halo));
  launch_duo_plan(n, halo, plan, (hipStream_t)stream);
  return check_launch("strata_duo_plan");
}

strata_status strata_duo_pad_planned(const void* faces, int32_t P, int32_t n, int32_t C, int32_t halo,
                                     const void* plan, size_t plan_bytes, void* padded, strata_dtype dtype,
                                     void* stream) {
  REQUIRE(P > 0 && C > 0, "duo: P and C must be positive");
  REQUIRE(n >= 16 && halo > 0 && halo <= n / 4, "duo: need n >= 16 and 1 <= halo <= n/4 (n=%d, halo=%d)", n, halo);
  REQUIRE(dtype == STRATA_F32 || dtype == STRATA_BF16, "duo: unknown dtype %d", (int)dtype);
  const int64_t m = (int64_t)n + 2 * halo;
  REQUIRE(6LL * P * m * m * C < kMaxElems, "duo: tensor too large");
  REQUIRE_PTR(faces);
  REQUIRE_PTR(padded);
  REQUIRE_PTR(plan);
  REQUIRE(reinterpret_cast<uintptr_t>(plan) % 16 == 0, "duo: plan must be 16-byte aligned");
  REQUIRE(plan_bytes >= (size_t)duo_plan_bytes(n, halo), "duo: plan_bytes %zu < %lld (a plan for other n, halo?)",
          plan_bytes, (long long)duo_plan_bytes(n, halo));
  launch_duo_pad_planned(faces, plan, P, n, C, halo, padded, dtype, (hipStream_t)stream);
  return check_launch("strata_duo_pad_planned");
}

strata_status strata_duo_pad_vjp(const void* grad_padded, int32_t P, int32_t n, int32_t C, int32_t halo,
                                 const void* plan, size_t plan_bytes, void* grad_faces, strata_dtype dtype,
                                 void* stream) {
  REQUIRE(P > 0 && C > 0 && P <= 65535, "duo vjp: need 0 < P <= 65535 and C > 0 (P=%d, C=%d)", P, C);
  REQUIRE(n >= 16 && halo > 0 && halo <= n / 4, "duo vjp: need n >= 16 and 1 <= halo <= n/4 (n=%d, halo=%d)", n,
          halo);
  REQUIRE(dtype == STRATA_F32 || dtype == STRATA_BF16, "duo vjp: unknown dtype %d", (int)dtype);
  REQUIRE(duo_plan_fits(n, halo), "duo vjp: n=%d too large for a plan", n);
  const int64_t m = (int64_t)n + 2 * halo;
  REQUIRE(6LL * P * m * m * C < kMaxElems, "duo vjp: tensor too large");
  REQUIRE_PTR(grad_padded);
  REQUIRE_PTR(grad_faces);
  REQUIRE_PTR(plan);
  REQUIRE(reinterpret_cast<uintptr_t>(plan) % 16 == 0, "duo vjp: plan must be 16-byte aligned");
  REQUIRE(plan_bytes >= (size_t)duo_plan_bytes(n, halo), "duo vjp: plan_bytes %zu < %lld (a plan for other n, halo?)",
          plan_bytes, (long long)duo_plan_bytes(n, halo));
  launch_duo_pad_vjp(grad_padded, plan, P, n, C, halo, grad_faces, dtype, (hipStream_t)stream);
  return check_launch("strata_duo_pad_vjp");
}

strata_status strata_kbd_window(int32_t Ht, int32_t Wt, int32_t overlap, double beta, float* window,
                                void* stream) {
  REQUIRE(Ht > 0 && Wt > 0 && (int64_t)Ht * Wt < ((int64_t)1 << 31), "kbd: sizes must be positive");
  REQUIRE(overlap > 0 && overlap <= Ht && overlap <= Wt, "kbd: need 1 <= overlap <= min(Ht, Wt) (got %d)", overlap);
  REQUIRE(beta >= 0.0 && beta <= 700.0, "kbd: beta must lie in [0, 700]");
  REQUIRE_PTR(window);
  launch_kbd_window(Ht, Wt, overlap, beta, window, (hipStream_t)stream);
  return check_launch("strata_kbd_window");
}

strata_status strata_tile_extract(const void* face, int32_t nty, int32_t ntx, int32_t P,
                                  int32_t Ht, int32_t Wt, int32_t C, int32_t stride_y,
                                  int32_t stride_x, int32_t Hf, int32_t Wf, void* tiles,
                                  strata_dtype dtype, void* stream) {
  strata_status st = check_tiling(nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf, dtype);
  if (st != STRATA_OK) return st;
  REQUIRE_PTR(face);
  REQUIRE_PTR(tiles);
  launch_tile_extract(face, nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf, tiles, dtype,
                      (hipStream_t)stream);
  return check_launch("strata_tile_extract");
}

}  // extern "C"

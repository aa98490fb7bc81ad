// Launchers of the HIP kernels behind the C ABI.  Each returns after enqueueing
// work on `stream`; argument validation happens in api.hip before these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "strata.h"

namespace strata {

// Options of the attention block (App. B.5): RMS normalisation of q and k (no
// learnable scale) and a sigmoid gate on the output, with logits of the
// problem's dtype, one per (token, head) (gate_dim 1) or per channel.
struct NaOpts {
  int qk_norm = 0;
  float eps = 0.f;
  const void* gate = nullptr;
  int gate_dim = 0;
};

void launch_axis_index(int L, int k, int32_t* starts, int32_t* qlo, int32_t* qhi, hipStream_t s);

void launch_stereo_coords(const int32_t* face, const int32_t* oy, const int32_t* ox, int B, int H,
                          int W, int face_cells, int patch, double l_scale, float* coords,
                          hipStream_t s);

void launch_wind_tile_frame(const void* field, int face, int n_cells, int nty, int ntx, int P, int Ht, int Wt,
                            int sy, int sx, void* tiles, strata_dtype dt, hipStream_t s);

void launch_rope_phases(const float* coords, int B, int H, int W, int head_dim, double base,
                        float* cs, hipStream_t s);

void launch_rope_apply(const void* x, void* y, const float* cs, int B, int heads, int Z, int H,
                       int W, int head_dim, strata_dtype dt, int transpose, hipStream_t s);

// Plain per-query forward (float32 arithmetic), any supported dtype / head_dim.
void launch_na3d_fwd_ref(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                         const void* v, const float* cs, void* out, float* lse, hipStream_t s);

// bf16 MFMA forward sweeping the key levels once per head (window 3x7x7, Z = 8);
// returns false for any other problem.
// A regular tiling of one face that a forward stitches into: tile (a, b) of
// the batch (index a ntx + b) has its origin at (a sy, b sx) of the face
// [heads Z, Hf, Wf, head_dim]; `window` [H, W] holds the stitch weights.
struct StitchArgs {
  void* face;
  const float* window;
  int nty, ntx, sy, sx, Hf, Wf;
};

bool launch_na3d_fwd_zs(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                        const void* v, const float* cs, void* out, float* lse, hipStream_t s,
                        const StitchArgs* st = nullptr);

// bf16 level sweep over groups of query levels (head_dim 64, windows 3x7x7 and
// 5x9x9, any Z); returns false for any other problem.
bool launch_na3d_fwd_lsg(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                         const void* v, const float* cs, void* out, float* lse, hipStream_t s);

// bf16 column-wise forward, windows (kz, 1, 1) with Z <= 32, head_dim 64;
// returns false for any other problem.
bool launch_na3d_fwd_col(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                         const void* v, void* out, float* lse, hipStream_t s);

// bf16 MFMA forward; returns false when the problem has no MFMA variant.
// head_dim-128 forward (bf16, window 9x9x9, options included); false if not applicable
bool launch_na3d_fwd_d128(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                          const void* v, const float* cs, void* out, float* lse, hipStream_t s);
bool launch_na3d_fwd_mfma(const strata_na3d_desc& d, const NaOpts& o, const void* q, const void* k,
                          const void* v, const float* cs, void* out, float* lse, hipStream_t s);

// Options of the attention backward kernels: QK RMSNorm (applied to q and k
// as they are loaded, its Jacobian applied to dq and dk before the store) and
// the low part of an upstream gradient given as two terms dO = hi + lo of the
// problem's dtype (the gated dA = sigmoid(g) dO split exactly enough that its
// rounding does not show); dout_lo = nullptr: dO is `dout` alone.
struct BwdOpts {
  int qk_norm = 0;
  float eps = 0.f;
  const void* dout_lo = nullptr;
};

// Plain backward (float32 arithmetic), one part per call: 0 = D = rowsum(dO * O)
// into dvec, 1 = dq, 2 = dk and dv (parts 1 and 2 read dvec).
void launch_na3d_bwd_ref(int part, const strata_na3d_desc& d, const BwdOpts& o, const void* q,
                         const void* k, const void* v, const float* cs, const void* out,
                         const void* dout, const float* lse, void* dq, void* dk, void* dv,
                         float* dvec, hipStream_t s);

// Row pass of the gated backward (one 16-byte piece per lane): D = rowsum(dO *
// out) into dvec, dA = sigmoid(g) dO as da_hi (+ da_lo for bf16: the rounding
// remainder, so that hi + lo carries dA to ~2^-16), and dgate.
void launch_na3d_bwd_gate_prep(const strata_na3d_desc& d, const NaOpts& o, const void* out,
                               const void* dout, float* dvec, void* da_hi, void* da_lo, void* dgate,
                               hipStream_t s);

// bf16 MFMA backward parts; each returns false when the problem has no MFMA variant.
// dq: query-stationary (the forward's decomposition); dk/dv: key-stationary.
// With `out` (the forward's O) set, the dq pass also forms D = rowsum(dO * O)
// itself and stores it to dvec for the dk/dv pass (not with a two-term dO);
// with `emax` set ([B * heads] int32) it stores there, per (batch, head), the
// largest frexp exponent of |dO| (kEmaxEmpty where every dO is zero), which the
// balanced dk/dv pass scales dO by.  na3d_bwd_dq_mfma_takes is its test of
// whether it takes the problem.
constexpr int kEmaxEmpty = -1000;
bool na3d_bwd_dq_mfma_takes(const strata_na3d_desc& d);
bool launch_na3d_bwd_dq_mfma(const strata_na3d_desc& d, const BwdOpts& o, const void* q,
                             const void* k, const void* v, const float* cs, const void* dout,
                             const float* lse, float* dvec, const void* out, int* emax, void* dq,
                             hipStream_t s);
// bf16 column-wise backward (dq, dk, dv together), windows (kz, 1, 1) with Z <= 32,
// head_dim 64; false for any other problem.
bool launch_na3d_bwd_col(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                         const void* v, const void* dout, const float* lse, const float* dvec, void* dq,
                         void* dk, void* dv, hipStream_t s);
// dK/dV with two key levels x four 4x4 blocks per workgroup (bf16, head_dim 64,
// windows 5x9x9 and 9x9x9, no two-term dO); false if not applicable
// (emax: the dO exponents the MFMA dq pass recorded; na3d_bwd_dkdv_kvp_takes
// is the launcher's test of whether it takes the problem)
bool na3d_bwd_dkdv_kvp_takes(const strata_na3d_desc& d, const BwdOpts& o);
bool launch_na3d_bwd_dkdv_kvp(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                              const void* v, const float* cs, const void* dout, const float* lse,
                              const float* dvec, const int* emax, void* dk, void* dv, hipStream_t s);
bool launch_na3d_bwd_dkdv_mfma(const strata_na3d_desc& d, const BwdOpts& o, const void* q,
                               const void* k, const void* v, const float* cs, const void* dout,
                               const float* lse, const float* dvec, void* dk, void* dv,
                               hipStream_t s);
// head_dim-128 backward passes (bf16, window 9x9x9, no options); false if not applicable
bool launch_na3d_bwd_dq_d128(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                             const void* v, const float* cs, const void* dout, const float* lse,
                             const float* dvec, void* dq, hipStream_t s);
bool launch_na3d_bwd_dkdv_d128(const strata_na3d_desc& d, const BwdOpts& o, const void* q, const void* k,
                               const void* v, const float* cs, const void* dout, const float* lse,
                               const float* dvec, void* dk, void* dv, hipStream_t s);

// Stitch of the cells covered by two or more tiles along y or x of a bf16
// tiling with sy <= Ht <= 2 sy, sx <= Wt <= 2 sx, C % 8 == 0, whose tiles
// cover the face ((nty-1) sy + Ht == Hf, (ntx-1) sx + Wt == Wf).
void launch_tile_blend_overlap(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                               int sx, const float* window, void* out, int Hf, int Wf, hipStream_t s);
void launch_tile_blend(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                       int sx, const float* window, void* out, int Hf, int Wf, strata_dtype dt,
                       hipStream_t s);

void launch_duo_pad(const void* in, int P, int n, int C, int halo, void* out, strata_dtype dt, hipStream_t s);
int64_t duo_plan_bytes(int n, int halo);
void launch_duo_plan(int n, int halo, void* plan, hipStream_t s);
void launch_duo_pad_planned(const void* in, const void* plan, int P, int n, int C, int halo, void* out,
                            strata_dtype dt, hipStream_t s);
void launch_duo_pad_vjp(const void* gpad, const void* plan, int P, int n, int C, int halo, void* gfaces,
                        strata_dtype dt, hipStream_t s);

void launch_kbd_window(int Ht, int Wt, int overlap, double beta, float* window, hipStream_t s);

void launch_tile_extract(const void* face, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                         int sx, int Hf, int Wf, void* tiles, strata_dtype dt, hipStream_t s);

}  // namespace strata

// Launchers of the HIP kernels behind the C ABI.  Each returns after enqueueing
// work on `stream`; argument validation happens in api.hip before these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "strata.h"

namespace strata {

void launch_axis_index(int L, int k, int32_t* starts, int32_t* qlo, int32_t* qhi, hipStream_t s);

void launch_stereo_coords(const int32_t* face, const int32_t* oy, const int32_t* ox, int B, int H,
                          int W, int face_cells, int patch, double l_scale, float* coords,
                          hipStream_t s);

void launch_rope_phases(const float* coords, int B, int H, int W, int head_dim, double base,
                        float* cs, hipStream_t s);

void launch_rope_apply(const void* x, void* y, const float* cs, int B, int heads, int Z, int H,
                       int W, int head_dim, strata_dtype dt, int transpose, hipStream_t s);

// Plain per-query forward (float32 arithmetic), any supported dtype / head_dim.
void launch_na3d_fwd_ref(const strata_na3d_desc& d, const void* q, const void* k, const void* v,
                         const float* cs, void* out, float* lse, hipStream_t s);

// bf16 MFMA forward sweeping the key levels once per head (window 3x7x7, Z = 8);
// returns false for any other problem.
bool launch_na3d_fwd_zs(const strata_na3d_desc& d, const void* q, const void* k, const void* v,
                        const float* cs, void* out, float* lse, hipStream_t s);

// bf16 MFMA forward; returns false when the problem has no MFMA variant.
bool launch_na3d_fwd_mfma(const strata_na3d_desc& d, const void* q, const void* k, const void* v,
                          const float* cs, void* out, float* lse, hipStream_t s);

// Plain backward (float32 arithmetic), one part per call: 0 = D = rowsum(dO * O)
// into dvec, 1 = dq, 2 = dk and dv (parts 1 and 2 read dvec).
void launch_na3d_bwd_ref(int part, const strata_na3d_desc& d, const void* q, const void* k,
                         const void* v, const float* cs, const void* out, const void* dout,
                         const float* lse, void* dq, void* dk, void* dv, float* dvec, hipStream_t s);

// bf16 MFMA backward parts; each returns false when the problem has no MFMA variant.
// dq: query-stationary (the forward's decomposition); dk/dv: key-stationary.
bool launch_na3d_bwd_dq_mfma(const strata_na3d_desc& d, const void* q, const void* k, const void* v,
                             const float* cs, const void* dout, const float* lse,
                             const float* dvec, void* dq, hipStream_t s);
bool launch_na3d_bwd_dkdv_mfma(const strata_na3d_desc& d, const void* q, const void* k,
                               const void* v, const float* cs, const void* dout, const float* lse,
                               const float* dvec, void* dk, void* dv, hipStream_t s);

void launch_tile_blend(const void* tiles, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                       int sx, const float* window, void* out, int Hf, int Wf, strata_dtype dt,
                       hipStream_t s);

void launch_tile_extract(const void* face, int nty, int ntx, int P, int Ht, int Wt, int C, int sy,
                         int sx, int Hf, int Wf, void* tiles, strata_dtype dt, hipStream_t s);

}  // namespace strata

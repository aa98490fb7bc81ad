/*
 * strata.h -- C ABI of the STRATA hot path on AMD Instinct MI355X (gfx950).
 *
 * What it computes (arxiv 2606.31248, "Scaling Storm-Resolving Atmospheric AI
 * Simulation to the Entire Planet"):
 *   - the tile-centred stereographic coordinates of every token (Sec. 3.3, Eq. 1);
 *   - StereoRoPE: axial 2D rotary embedding driven by those coordinates (Sec. 3.3);
 *   - 3D neighbourhood attention over the (level, y, x) token grid of each tile
 *     with NATTEN's border-clamped windows (Sec. 3.2), forward and backward;
 *   - the overlapping-tile stitch S = D^-1 P^T W and its extraction P
 *     (App. F, "Tile stitching", "Linear operator interpretation");
 *   - QK RMSNorm and the sigmoid output gate of the attention block (App. B.5);
 *   - the wind vectors of each tile in its centre's East-North frame (Sec. 3.3,
 *     Eq. 2);
 *   - the Duo-grid halo padding across cube faces and the Kaiser-Bessel-derived
 *     blend window (App. F).
 *
 * Conventions shared by every call:
 *   - Pointers are DEVICE pointers owned by the caller unless stated otherwise.
 *     The library never allocates device memory and never frees caller memory.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream).  Arguments are validated synchronously before any launch; on a
 *     validation error nothing is launched.
 *   - Activations are [B, heads, Z, H, W, head_dim], contiguous, head_dim
 *     innermost: B tiles, Z vertical levels, H x W horizontal tokens.
 *   - Element types: STRATA_F32 (IEEE binary32) or STRATA_BF16 (bfloat16 bit
 *     patterns in uint16 storage).  Results are rounded to nearest-even.
 *   - Every call returns a strata_status; a non-OK status leaves a message
 *     retrievable with strata_last_error() on the calling thread.  Nothing
 *     throws across the ABI.  Device pointers must be 16-byte aligned.
 */
#ifndef STRATA_H_
#define STRATA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  STRATA_OK = 0,
  STRATA_ERR_INVALID_ARG = 1, /* null pointer, bad size, misalignment, bad window */
  STRATA_ERR_UNSUPPORTED = 2, /* valid arguments this build has no kernel for */
  STRATA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  STRATA_ERR_HIP = 4          /* the HIP runtime reported an error at launch */
} strata_status;

typedef enum { STRATA_F32 = 0, STRATA_BF16 = 1 } strata_dtype;

/* Neighbourhood-attention problem.  Window (kz, ky, kx): odd, 1 <= k <= extent
 * on its axis, dilation 1.  A query at position i of an axis of extent L sees
 * the k positions [s, s + k) with s = min(max(i - (k-1)/2, 0), L - k): centred,
 * shifted inward at the borders, so every query sees exactly kz*ky*kx keys. */
typedef struct {
  int32_t B, heads, Z, H, W, head_dim;
  int32_t kz, ky, kx;
  float scale;        /* logit scale, > 0 (usually 1/sqrt(head_dim)) */
  strata_dtype dtype; /* element type of q, k, v, out, dout, dq, dk, dv */
} strata_na3d_desc;

/* ---- a1: stereographic tile coordinates (Sec. 3.3, Eq. 1) -----------------
 * For tile b on the equiangular cubed sphere (faces of face_cells^2 cells,
 * tokens of patch x patch cells), token (y, x) of the tile has face token
 * (tile_oy[b] + y, tile_ox[b] + x) on face tile_face[b] (0..5).  Its
 * (lat, lon) is projected stereographically about the tile centre (the point
 * at the mean angles of the tile's first and last token) and divided by
 * l_scale, Eq. 1's length sqrt(4 pi / N_total); l_scale == 0 selects
 * sqrt(4 pi / (6 face_cells^2)) (N_total = the native cells of the six faces),
 * any other value must be finite and > 0:
 *   coords[b, y, x, 0] = x_east / l_scale,  coords[b, y, x, 1] = y_north / l_scale.
 * Face f with a = tan(alpha) (columns), c = tan(beta) (rows) is the cube point
 *   0:(1,a,c) 1:(-a,1,c) 2:(-1,-a,c) 3:(a,-1,c) 4:(-c,a,1) 5:(c,a,-1).
 * Computed in float64, stored as float32.  tile_face/oy/ox: device int32[B];
 * coords: device float32[B, H, W, 2].  Tiles must fit on the face. */
strata_status strata_stereo_coords(const int32_t* tile_face, const int32_t* tile_oy,
                                   const int32_t* tile_ox, int32_t B, int32_t H, int32_t W,
                                   int32_t face_cells, int32_t patch, double l_scale,
                                   float* coords, void* stream);

/* ---- wind vectors into the tile-centre frame (Sec. 3.3, Eq. 2) -------------
 * Cuts tiles from one cube face's horizontal wind and expresses every wind
 * vector in the East-North frame at its tile's centre:
 *   v = U e + V n  with the unit East and North vectors (e, n) at the cell's
 *   (lat, lon);  v_perp = v - (v . r0) r0;  U_loc = v_perp . e0,
 *   V_loc = v_perp . n0  with (e0, n0, r0) at the tile centre.
 * field: [P, face_cells, face_cells, 2] of dtype, (U, V) per cell of face
 * `face` (0..5, orientation as in strata_stereo_coords) for P planes (levels);
 * cell (i, j) has angles alpha = -pi/4 + (j + 1/2) (pi/2)/face_cells (columns)
 * and beta likewise from the row i.  Tile t = a*ntx + b covers the Ht x Wt
 * cells from (a*stride_y, b*stride_x); its centre is the point at the mean
 * angles of its first and last cell on each axis (at a pole the frame is the
 * formula's at the computed longitude).  tiles: [nty*ntx, P, Ht, Wt, 2] of
 * dtype.  Geometry and the 2x2 rotation in float32 for bf16 data, in float64
 * for float32 data.  Tiles must fit on the face. */
strata_status strata_wind_tile_frame(const void* field, int32_t face, int32_t face_cells, int32_t nty,
                                     int32_t ntx, int32_t P, int32_t Ht, int32_t Wt, int32_t stride_y,
                                     int32_t stride_x, void* tiles, strata_dtype dtype, void* stream);

/* ---- a2: StereoRoPE phase table (Sec. 3.3) --------------------------------
 * cs[b, y, x, t] = (cos th, sin th) for pair t < head_dim/2, with
 *   th = coords[b,y,x,0] * base^(-t/(head_dim/4))               for t <  head_dim/4,
 *   th = coords[b,y,x,1] * base^(-(t-head_dim/4)/(head_dim/4))  for t >= head_dim/4.
 * Built in float64, stored as float32 pairs.  coords: float32[B, H, W, 2];
 * cs: float32[B, H, W, head_dim/2, 2].  head_dim % 4 == 0, base > 0. */
strata_status strata_stereorope_phases(const float* coords, int32_t B, int32_t H, int32_t W,
                                       int32_t head_dim, double base, float* cs, void* stream);

/* ---- a2: StereoRoPE application (Sec. 3.3) --------------------------------
 * Rotates every pair (x[2t], x[2t+1]) of every token by its phase:
 *   y[2t] = x[2t] cos - x[2t+1] sin,  y[2t+1] = x[2t] sin + x[2t+1] cos;
 * transpose != 0 rotates by the opposite angle (R^T, used for gradients).
 * All levels and heads of a column share the phase of (b, y, x).
 * x, y: [B, heads, Z, H, W, head_dim] of dtype; y may equal x (in place).
 * Arithmetic in float32. */
strata_status strata_stereorope_apply(const void* x, void* y, const float* cs, int32_t B,
                                      int32_t heads, int32_t Z, int32_t H, int32_t W,
                                      int32_t head_dim, strata_dtype dtype, int32_t transpose,
                                      void* stream);

/* ---- a3-a6: neighbourhood attention forward (Sec. 3.2) --------------------
 * For every query i (all heads, tiles, positions):
 *   s_ij = scale * <R_i q_i, R_j k_j>  over the kz*ky*kx keys j of i's window,
 *   lse_i = ln sum_j exp(s_ij),   out_i = sum_j exp(s_ij - lse_i) v_j,
 * where R is the StereoRoPE rotation from the phase table `cs` (float32
 * [B, H, W, head_dim/2, 2]), or the identity when cs == NULL.
 * q, k, v, out: [B, heads, Z, H, W, head_dim] of desc->dtype;
 * lse: float32 [B, heads, Z, H, W] (natural log) or NULL when not needed.
 * Supported: head_dim 32, 64 or 128 in either dtype.  Kernels: bf16 at
 * head_dim 64 runs on MFMA for the windows (3,7,7), (5,9,9), (9,9,9) and every
 * column window (kz,1,1) with Z <= 32 (level sweeps for (3,7,7) and (5,9,9), a
 * query-stationary kernel for (9,9,9)); bf16 at head_dim 128 on MFMA for (9,9,9);
 * every other case (f32, head_dim 32, other windows) on plain kernels in
 * float32 (one thread per query, or one wave per query below 2^18 queries).
 * Softmax and accumulation in float32.
 * Contraction precision: on the MFMA paths the logits q.k are float16 products
 * (wider mantissa than bf16) of float16 copies of the rotated, normalised and
 * scaled q and k, accumulated in float32; P.V is a float16 product (weights and
 * V in float16) on the level-sweep kernels (3x7x7, 5x9x9), a bf16 one on the
 * others; V of magnitude above 65504 then saturates and below 2^-14 keeps
 * float16's subnormal spacing.  Input range:
 * with M = max(1, 2 scale log2(e)), inputs with M |q| <= 32000 and
 * M |k| <= 32000 (q^, k^ after the QK norm) keep every float16 operand inside
 * its range; beyond that each path saturates its float16 copies (results stay
 * finite) and the paths may give different results. */
strata_status strata_na3d_fwd(const strata_na3d_desc* desc, const void* q, const void* k,
                              const void* v, const float* cs, void* out, float* lse,
                              void* stream);

/* ---- a7: neighbourhood attention backward ----------------------------------
 * Gradients of the forward above for upstream gradient dout, with the lse the
 * forward wrote and its output `out`:
 *   P_ij = exp(s_ij - lse_i),   D_i = <dout_i, out_i>,
 *   dv_j = sum_{i: j in N(i)} P_ij dout_i,    dS_ij = P_ij (<dout_i, v_j> - D_i),
 *   dq_i = R_i^T scale sum_j dS_ij R_j k_j,    dk_j = R_j^T scale sum_i dS_ij R_i q_i.
 * Deterministic (the one atomic operation is an integer maximum, whose result
 * does not depend on order).  workspace: device memory of at least
 * strata_na3d_bwd_workspace_size(desc) bytes (holds D, one word per (batch,
 * head) and, with a gate, dA), owned by the caller.
 * Kernels and input range as strata_na3d_fwd; on the MFMA paths the dS products
 * (dq, dk) are float16 with exact power-of-two scaling; P.dO and dO.V^T are
 * float16 products with dO scaled by a power of two per (batch, head) in the
 * dK/dV kernel of the 9-wide windows (V then saturates at 65504 and keeps
 * float16's subnormal spacing below 2^-14, as in the level-sweep forward);
 * elsewhere they are bf16 products, P.dO with P in two bf16 terms in the
 * one-block dK/dV kernel (3x7x7, planes of 17-20 positions; one term with the
 * gate's two-term dA) and with P rounded to bf16 once in the column and
 * head_dim-128 kernels. */
size_t strata_na3d_bwd_workspace_size(const strata_na3d_desc* desc);
strata_status strata_na3d_bwd(const strata_na3d_desc* desc, const void* q, const void* k,
                              const void* v, const float* cs, const void* out, const void* dout,
                              const float* lse, void* dq, void* dk, void* dv, void* workspace,
                              size_t workspace_bytes, void* stream);

/* ---- backward for callers that cannot allocate --------------------------------
 * For code under HIP graph capture, tight training loops and harnesses that
 * forbid hipMalloc: strata_na3d_bwd without a workspace.  Same arguments,
 * results and kernels as strata_na3d_bwd (plain attention, no options); D and
 * one word per (batch, head) live in a static device array of the library
 * (32 MiB + 256 KiB), one per device, held until the process ends.  Limits:
 * B*heads*Z*H*W <= 2^23 token-heads and B*heads <= 2^16, otherwise
 * STRATA_ERR_INVALID_ARG and nothing is launched.  Nothing is allocated; the
 * array's device address is looked up once per device on the first call.
 * Every call on a device shares that device's array: calls that overlap on one
 * device (two streams, two threads) race and must be ordered by the caller. */
strata_status strata_na3d_bwd_noalloc(const strata_na3d_desc* desc, const void* q, const void* k,
                                      const void* v, const float* cs, const void* out,
                                      const void* dout, const float* lse, void* dq, void* dk,
                                      void* dv, void* stream);

/* ---- QK normalisation and the output gate (App. B.5) -----------------------
 * Options of the attention block beyond plain neighbourhood attention; a
 * zero-initialised struct (or a NULL pointer) selects plain attention.
 *   qk_norm != 0: every query and key vector (one token of one head, its
 *     head_dim entries) is divided by its root mean square before the dot
 *     product, with no learnable scale:  x^ = x / sqrt(mean_e x_e^2 + eps).
 *     The norm precedes the StereoRoPE rotation (the two commute: a rotation
 *     keeps every pair's sum of squares).  eps: finite, >= 0 (with eps = 0 an
 *     all-zero vector gives inf/NaN).
 *   gate != NULL: the attention output of every (token, head) is multiplied by
 *     sigmoid(g) = 1 / (1 + exp(-g)) of the gate logits g (device memory of
 *     desc->dtype): gate_dim == 1 -> g is [B, heads, Z, H, W], one logit per
 *     token and head; gate_dim == head_dim -> g is [B, heads, Z, H, W,
 *     head_dim], one per channel.  The logits are inputs: whatever produces
 *     them (a projection of the block input) lies outside this library. */
typedef struct {
  int32_t qk_norm;
  float eps;
  const void* gate;
  int32_t gate_dim;
} strata_na3d_opts;

/* Forward with options: s_ij = scale <R_i q^_i, R_j k^_j> (q^ = q, k^ = k when
 * qk_norm == 0), lse_i = ln sum_j exp(s_ij) (the softmax's, before the gate),
 * out_i = sigmoid(g_i) * sum_j exp(s_ij - lse_i) v_j (no factor without a
 * gate).  Everything else as strata_na3d_fwd; opts == NULL is strata_na3d_fwd. */
strata_status strata_na3d_fwd_ex(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                 const void* q, const void* k, const void* v, const float* cs,
                                 void* out, float* lse, void* stream);

/* Backward with options, for dout = d(loss)/d(out) of the gated output, with the
 * out and lse the forward wrote.  By the chain rule through the forward:
 *   gate: a = sigmoid(g), dA = a * dout, dgate = (1 - a) * dout * out per
 *     channel (gate_dim == head_dim) or (1 - a) * <dout_i, out_i>
 *     (gate_dim == 1);
 *   attention: the backward of strata_na3d_bwd on (q^, k^, v) with upstream
 *     gradient dA (its D_i = <dA_i, A_i> equals <dout_i, out_i>);
 *   norm: dx = r (dx^ - x^ mean_e(dx^_e x^_e)), r = (mean(x^2) + eps)^(-1/2),
 *     for x = q and x = k.
 * dgate: same shape and dtype as the gate, required when opts->gate is set
 * (NULL otherwise).  workspace: at least strata_na3d_bwd_ex_workspace_size(desc,
 * opts) bytes of device memory owned by the caller; it holds D and, with a
 * gate, dA (for bf16 as two bf16 terms whose sum carries it to ~2^-16).  The
 * norm is applied inside the attention kernels.  The library allocates
 * nothing. */
size_t strata_na3d_bwd_ex_workspace_size(const strata_na3d_desc* desc,
                                         const strata_na3d_opts* opts);
strata_status strata_na3d_bwd_ex(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                 const void* q, const void* k, const void* v, const float* cs,
                                 const void* out, const void* dout, const float* lse, void* dq,
                                 void* dk, void* dv, void* dgate, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* ---- a8: tile stitch S = D^-1 P^T W (App. F, Eq. stitch) -------------------
 * Regular tiling: tile t = a*ntx + b has origin (a*stride_y, b*stride_x) on the
 * face.  tiles: [nty*ntx, P, Ht, Wt, C] of dtype; window: float32 [Ht*Wt],
 * >= 0; out: [P, Hf, Wf, C] of dtype.  For every face cell:
 *   out = (sum_t w_t * value_t) / (sum_t w_t)  over the tiles t covering it,
 * summed in ascending a, then b, with fused multiply-adds from zero, divided
 * with correct rounding; bf16 data accumulate in float32, f32 data in float64.
 * Cells no tile weights (sum 0) are written as 0.  Requires
 * (nty-1)*stride_y + Ht <= Hf and (ntx-1)*stride_x + Wt <= Wf.  Bit-exact. */
strata_status strata_tile_blend(const void* tiles, int32_t nty, int32_t ntx, int32_t P,
                                int32_t Ht, int32_t Wt, int32_t C, int32_t stride_y,
                                int32_t stride_x, const float* window, void* out, int32_t Hf,
                                int32_t Wf, strata_dtype dtype, void* stream);

/* ---- a4-a6 + a8: face step with the stitch fused into the forward ----------
 * (Sec. 3.2 attention on each tile of one face, App. F, Eq. stitch.)  The
 * batch of `desc` is the nty x ntx tiling of one face, tile t = a*ntx + b at
 * origin (a*stride_y, b*stride_x), P = heads*Z planes, Ht = H, Wt = W,
 * C = head_dim, window float32 [H*W] >= 0, face [heads*Z, Hf, Wf, head_dim]
 * of the problem's dtype.  Two calls on one stream give
 *   strata_tile_blend(strata_na3d_fwd_ex(...))      bit for bit:
 * strata_na3d_fwd_stitch, then strata_tile_blend_overlap with the same tiles,
 * tiling, window and face.  The first writes the attention output (options
 * and lse as in strata_na3d_fwd_ex) and stores every cell that one tile alone
 * covers straight into `face`, computed as the stitch computes it: the tile's
 * value fma(w, v, +0) / w rounded to the dtype, which for 2^-8 <= w <= 1 (the
 * linear ramp's range) is v itself with -0 turned into +0, and 0 where w = 0.  The other cells go to `tiles`
 * ([B, heads, Z, H, W, head_dim], caller-owned scratch; the contents of
 * single-cover cells are unspecified).  The second stitches the cells that two
 * or more tiles cover and leaves the rest of the face as it is.  The fusion
 * applies to bf16 tilings whose tiles cover the face with
 * stride <= extent <= 2 stride on both axes, at the shape of the level-sweep
 * forward (3x7x7, Z = 8, head_dim 64); elsewhere the first call writes every
 * tile output and stitches the whole face, and the second re-stitches cells
 * with the same values.  tiles, face and the inputs must not overlap.
 * Validation as strata_na3d_fwd_ex and strata_tile_blend, plus B = nty*ntx.
 * One or two kernel launches per call; nothing is allocated. */
strata_status strata_na3d_fwd_stitch(const strata_na3d_desc* desc, const strata_na3d_opts* opts,
                                     const void* q, const void* k, const void* v, const float* cs,
                                     void* tiles, float* lse, int32_t nty, int32_t ntx,
                                     int32_t stride_y, int32_t stride_x, const float* window,
                                     void* face, int32_t Hf, int32_t Wf, void* stream);
strata_status strata_tile_blend_overlap(const void* tiles, int32_t nty, int32_t ntx, int32_t P,
                                        int32_t Ht, int32_t Wt, int32_t C, int32_t stride_y,
                                        int32_t stride_x, const float* window, void* out,
                                        int32_t Hf, int32_t Wf, strata_dtype dtype, void* stream);

/* ---- Duo-grid halo padding P (App. F, "DUO-style boundary padding") --------
 * faces: [6, P, n, n, C] of dtype (P planes of n x n cells with C channels per
 * face, orientation as in strata_stereo_coords); padded: [6, P, n + 2 halo,
 * n + 2 halo, C].  Interior cells are copied.  Halo cell (i, j) of face f
 * (i or j outside [0, n)) extends f's equiangular mesh on f's own plane
 * (angles -pi/4 + (index + 1/2)(pi/2)/n), is projected to the sphere, and
 * takes the inverse great-circle-distance weighted average of the 4 cells
 * nearest to that point on the face containing it (the face of its largest
 * coordinate; a point on an edge or corner, where face scores are equal on a
 * 1e-12 grid, belongs to the lowest-numbered face); distances equal on a
 * 1e-12-radian grid are ordered by (row, column), a cell at distance 0 takes
 * the whole weight.  Sums nearest first, in float32 for bf16 data, float64 for
 * float32 data.  Both buffers are device memory owned by the caller and must
 * not overlap.  n >= 16, 1 <= halo <= n/4, 6 P n rows plus one block per 256
 * halo cells below 2^31; otherwise STRATA_ERR_INVALID_ARG and nothing is
 * launched.  One kernel launch on `stream`. */
strata_status strata_duo_pad(const void* faces, int32_t P, int32_t n, int32_t C, int32_t halo, void* padded,
                             strata_dtype dtype, void* stream);

/* The same padding operator P built once and applied many times (App. F: P is a
 * fixed sparse matrix with 4 non-zeros per halo cell, so a model that pads
 * every layer of a rollout reuses it), and its transpose for gradients.
 *
 * strata_duo_plan_bytes: size of the plan for (n, halo), 0 if the pair is
 * invalid or too large (n + 2 halo < 2^14, 4 entries per halo cell below
 * 2^31).  strata_duo_plan: writes the plan (geometry only, no field
 * data: P and its transpose) into `plan`, caller-owned device memory of at
 * least that many bytes, 16-byte aligned; its contents are opaque and valid
 * for this (n, halo) only.  The build is deterministic.
 * strata_duo_pad_planned: as strata_duo_pad, with the neighbours and weights
 * read from a plan written by strata_duo_plan for the same (n, halo); results
 * are identical to strata_duo_pad's.
 * strata_duo_pad_vjp: the adjoint, grad_faces = P^T grad_padded
 * (grad_padded: [6, P, n + 2 halo, n + 2 halo, C], grad_faces: [6, P, n, n,
 * C], both of dtype, not overlapping): every face cell's interior gradient
 * plus, for each halo cell whose 4 neighbours include it, that halo cell's
 * gradient times the weight, summed in ascending padded-cell order (face,
 * row, column) after the interior term, with fused multiply-adds; float32
 * sums for bf16 data, float64 for float32 data; one rounding.  Deterministic.
 * P <= 65535.
 * Errors: STRATA_ERR_INVALID_ARG for the rules of strata_duo_pad, a NULL or
 * misaligned plan, or plan_bytes below strata_duo_plan_bytes(n, halo); nothing
 * is launched then. */
size_t strata_duo_plan_bytes(int32_t n, int32_t halo);
strata_status strata_duo_plan(int32_t n, int32_t halo, void* plan, size_t plan_bytes, void* stream);
strata_status strata_duo_pad_planned(const void* faces, int32_t P, int32_t n, int32_t C, int32_t halo,
                                     const void* plan, size_t plan_bytes, void* padded, strata_dtype dtype,
                                     void* stream);
strata_status strata_duo_pad_vjp(const void* grad_padded, int32_t P, int32_t n, int32_t C, int32_t halo,
                                 const void* plan, size_t plan_bytes, void* grad_faces, strata_dtype dtype,
                                 void* stream);

/* ---- a8: Kaiser-Bessel-derived blend window (App. F, "Tile stitching") -----
 * window[y * Wt + x] = w(y, Ht) * w(x, Wt) (float32 [Ht * Wt], device) with,
 * per axis of length L, w(i) = 1 in the interior and, over the `overlap` cells
 * at each end, the rising half of the KBD window of length 2*overlap:
 *   w(i) = sqrt(sum_{j<=i} k_j / sum_{j<=overlap} k_j),
 *   k_j = I0(beta sqrt(1 - (2j/overlap - 1)^2)),  j = 0..overlap,
 * mirrored at the far end (the smaller value where both ends reach).  The
 * paper gives no alpha or taper length: beta (= pi alpha) is an argument and
 * the taper spans the overlap, as the linear ramp does.  1 <= overlap <=
 * min(Ht, Wt); 0 <= beta <= 700.  Computed in float64, rounded once. */
strata_status strata_kbd_window(int32_t Ht, int32_t Wt, int32_t overlap, double beta, float* window,
                                void* stream);

/* ---- a8': tile extraction P (App. F) ---------------------------------------
 * tiles[t, p, i, j, c] = face[p, a*stride_y + i, b*stride_x + j, c] (exact copy). */
strata_status strata_tile_extract(const void* face, int32_t nty, int32_t ntx, int32_t P,
                                  int32_t Ht, int32_t Wt, int32_t C, int32_t stride_y,
                                  int32_t stride_x, int32_t Hf, int32_t Wf, void* tiles,
                                  strata_dtype dtype, void* stream);

/* ---- a3: window indexing of one axis (Sec. 3.2, NATTEN's border-clamped ----
 * neighbourhood; bit-exact integer export).  For an axis of extent L and
 * window k (odd with 1 <= k <= L, or k == L): starts[i] = min(max(i - (k-1)/2,
 * 0), L - k) is the first position of query i's window [starts[i],
 * starts[i] + k); [qlo[j], qhi[j]] is the contiguous range of queries whose
 * window holds position j.  starts, qlo, qhi: device int32[L] each, written by
 * one launch on `stream`; STRATA_ERR_INVALID_ARG for other (L, k) or a NULL /
 * misaligned pointer, with nothing launched. */
strata_status strata_na_axis_index(int32_t L, int32_t k, int32_t* starts, int32_t* qlo,
                                   int32_t* qhi, void* stream);

/* ---- status ---------------------------------------------------------------- */
const char* strata_status_string(strata_status status);
/* Detail of the last non-OK status returned on the calling thread ("" if none). */
const char* strata_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* STRATA_H_ */

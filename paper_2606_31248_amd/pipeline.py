"""One pass of the hot path on device tensors, as a sequence of libstrata calls.

coordinates (Eq. 1) -> StereoRoPE phases -> neighbourhood attention forward
with the rotation fused into the Q/K loads -> tile stitch S = D^-1 P^T W.
PyTorch only allocates device memory and supplies the stream.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

from . import binding as B

ROPE_BASE = 100.0


@dataclasses.dataclass
class TileGeometry:
    face: torch.Tensor   # int32 [B] on device
    oy: torch.Tensor     # int32 [B] token row of the tile origin
    ox: torch.Tensor     # int32 [B] token column of the tile origin
    face_cells: int = 2048
    patch: int = 4


def stereo_phases(geom: TileGeometry, H: int, W: int, head_dim: int,
                  coords: Optional[torch.Tensor] = None, cs: Optional[torch.Tensor] = None,
                  base: float = ROPE_BASE):
    """Coordinates [B, H, W, 2] and phase table [B, H, W, head_dim/2, 2] (float32)."""
    Bt = geom.face.shape[0]
    dev = geom.face.device
    if coords is None:
        coords = torch.empty((Bt, H, W, 2), dtype=torch.float32, device=dev)
    if cs is None:
        cs = torch.empty((Bt, H, W, head_dim // 2, 2), dtype=torch.float32, device=dev)
    B.strata_stereo_coords(geom.face, geom.oy, geom.ox, H, W, geom.face_cells, geom.patch,
                           0.0, coords)  # 0: the library's Eq. 1 length for these faces
    B.strata_stereorope_phases(coords, head_dim, base, cs)
    return coords, cs


def na3d_forward(q, k, v, window, scale, cs=None, out=None, lse=None):
    if out is None:
        out = torch.empty_like(q)
    desc = B.desc_for(q, window, scale)
    B.strata_na3d_fwd(desc, q, k, v, cs, out, lse)
    return out


def face_step(q, k, v, geom: TileGeometry, window, scale, tiling, blend_window, face_out,
              coords=None, cs=None, out=None, fused: bool = True, opts=None):
    """One face rollout step: per-tile NA3D forward with StereoRoPE, then the stitch.

    q, k, v: [T, heads, Z, Ht, Wt, d]; tiling = (nty, ntx, stride_y, stride_x);
    the tile outputs are viewed as [T, heads*Z, Ht, Wt, d] planes for the blend;
    face_out: [heads*Z, Hf, Wf, d].  fused: the forward stores the cells one tile
    alone covers straight into the face and the stitch visits only the overlaps
    (the same face bit for bit); `out` then holds only the overlap cells."""
    T, heads, Z, Ht, Wt, d = q.shape
    coords, cs = stereo_phases(geom, Ht, Wt, d, coords, cs)
    if out is None:
        out = torch.empty_like(q)
    nty, ntx, sy, sx = tiling
    planes = out.view(T, heads * Z, Ht, Wt, d)
    desc = B.desc_for(q, window, scale)
    if fused:
        B.strata_na3d_fwd_stitch(desc, opts, q, k, v, cs, out, None, nty, ntx, sy, sx, blend_window, face_out)
        B.strata_tile_blend_overlap(planes, nty, ntx, sy, sx, blend_window, face_out)
    else:
        B.strata_na3d_fwd_ex(desc, opts, q, k, v, cs, out, None)
        B.strata_tile_blend(planes, nty, ntx, sy, sx, blend_window, face_out)
    return face_out

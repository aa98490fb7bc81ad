"""Seeded synthetic inputs shared by the HIP path, the CPU oracle, tests and bench.

This module holds no arithmetic of the method itself: it only draws random
numbers, rounds them to the storage type the kernels consume, places tiles on
the cubed sphere and lists the workload shapes.  Everything the method
computes (stereographic coordinates, rotary phases, neighbourhood attention,
the tile blend) lives separately in the oracle and in the HIP kernels.

Random streams: ``numpy.random.default_rng([seed, stream])`` with
stream ids Q=0, K=1, V=2, dOut=3, tile placement=4, blend field=5.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np

STREAM_Q, STREAM_K, STREAM_V, STREAM_DO, STREAM_PLACE, STREAM_FIELD, STREAM_GATE = 0, 1, 2, 3, 4, 5, 6

# Cubed-sphere grid of the 4.9-km workload: 6 faces of 2048 x 2048 native cells,
# tokens are 4 x 4 horizontal patches (one vertical level per token).
FACE_CELLS = 2048
PATCH = 4
FACE_TOKENS = FACE_CELLS // PATCH  # 512
N_FACES = 6


def rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); returns uint16 bit patterns.

    Storage conversion of the synthetic draws (finite inputs only: the largest
    finite pattern plus 0x8000 stays below 2^32, so 32-bit integers suffice).
    Converted in chunks, so a multi-GB draw needs no wide temporaries."""
    xa = np.ascontiguousarray(x, dtype=np.float32)
    b = xa.reshape(-1).view(np.uint32)
    out = np.empty(b.size, np.uint16)
    step = 1 << 24
    for i in range(0, b.size, step):
        c = b[i:i + step]
        out[i:i + step] = ((c + ((c >> 16) & np.uint32(1)) + np.uint32(0x7FFF)) >> 16).astype(np.uint16)
    return out.reshape(xa.shape)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def gaussian(shape, seed: int, stream: int, dtype: str, mult: float = 1.0) -> np.ndarray:
    """iid N(0,1) draws (times ``mult``) in float32, stored as ``dtype``.

    dtype "f32" -> float32 array; dtype "bf16" -> uint16 array of bf16 bits (RNE)."""
    x = rng(seed, stream).standard_normal(size=shape, dtype=np.float32)
    if mult != 1.0:
        x = (x * np.float32(mult)).astype(np.float32)
    if dtype == "f32":
        return x
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    raise ValueError(f"unknown dtype {dtype!r}")


@dataclasses.dataclass(frozen=True)
class TilePlacement:
    """Where each tile of tokens sits on the cubed sphere.

    ``face[b]`` is the cube face (0..5), ``oy[b]``, ``ox[b]`` the token row /
    column of the tile's first token on that face (token grid FACE_TOKENS^2)."""
    face: np.ndarray
    oy: np.ndarray
    ox: np.ndarray

    def as_int32(self) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        return (self.face.astype(np.int32), self.oy.astype(np.int32), self.ox.astype(np.int32))


def random_placement(n_tiles: int, tile_h: int, tile_w: int, seed: int,
                     face_tokens: int = FACE_TOKENS) -> TilePlacement:
    """Faces uniform over the 6 cube faces, token origins uniform so the tile fits the face."""
    g = rng(seed, STREAM_PLACE)
    face = g.integers(0, N_FACES, size=n_tiles)
    oy = g.integers(0, face_tokens - tile_h + 1, size=n_tiles)
    ox = g.integers(0, face_tokens - tile_w + 1, size=n_tiles)
    return TilePlacement(face.astype(np.int64), oy.astype(np.int64), ox.astype(np.int64))


def corner_placement(tile_h: int, tile_w: int) -> TilePlacement:
    """One tile at the corner of face 0 (strongest equiangular distortion)."""
    z = np.zeros(1, dtype=np.int64)
    return TilePlacement(z.copy(), z.copy(), z.copy())


def face_tiling(face: int, n_ty: int, n_tx: int, stride_y: int, stride_x: int) -> TilePlacement:
    """Regular overlapping tiling of one face: tile (a, b) has origin (a*stride_y, b*stride_x)."""
    a, b = np.meshgrid(np.arange(n_ty), np.arange(n_tx), indexing="ij")
    n = n_ty * n_tx
    return TilePlacement(np.full(n, face, dtype=np.int64),
                         (a.reshape(-1) * stride_y).astype(np.int64),
                         (b.reshape(-1) * stride_x).astype(np.int64))


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload of the hot path (shapes follow the paper's tiles)."""
    name: str
    seed: int
    dtype: str            # "f32" or "bf16"
    B: int                # tiles
    heads: int
    Z: int
    H: int
    W: int
    d: int
    kz: int
    ky: int
    kx: int
    rope: bool = True
    qkv_mult: float = 1.0           # multiplier applied to the N(0,1) draws
    # regular face tiling (face rollout step) or random placement
    tiling: Optional[Tuple[int, int, int, int]] = None   # (n_ty, n_tx, stride_y, stride_x)
    corner: bool = False

    @property
    def N(self) -> int:
        return self.Z * self.H * self.W

    @property
    def K(self) -> int:
        return self.kz * self.ky * self.kx

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))

    def shape(self) -> Tuple[int, ...]:
        return (self.B, self.heads, self.Z, self.H, self.W, self.d)

    def placement(self) -> TilePlacement:
        if self.tiling is not None:
            n_ty, n_tx, sy, sx = self.tiling
            return face_tiling(0, n_ty, n_tx, sy, sx)
        if self.corner:
            return corner_placement(self.H, self.W)
        return random_placement(self.B, self.H, self.W, self.seed)

    def qkv(self):
        s = self.shape()
        return tuple(gaussian(s, self.seed, st, self.dtype, self.qkv_mult)
                     for st in (STREAM_Q, STREAM_K, STREAM_V))

    def dout(self):
        return gaussian(self.shape(), self.seed, STREAM_DO, self.dtype)


# The five workloads of the hot path.  Seeds are 1000 + workload number.
TINY_F32 = Workload("tiny_f32_1x4x16x16_h4_d32_w3x7x7", 1001, "f32",
                    1, 4, 4, 16, 16, 32, 3, 7, 7, corner=True)
SMALL_BF16 = Workload("bf16_8x8x32x32_h8_d64_w3x7x7", 1002, "bf16",
                      8, 8, 8, 32, 32, 64, 3, 7, 7)
TRAIN_TILE = Workload("bf16_16x8x64x64_h16_d64_w5x9x9", 1003, "bf16",
                      16, 16, 8, 64, 64, 64, 5, 9, 9)
TRAIN_TILE_BWD = Workload("bf16_bwd_16x8x64x64_h16_d64_w5x9x9", 1004, "bf16",
                          16, 16, 8, 64, 64, 64, 5, 9, 9)
# One cube face of 2048^2 cells at 4x4 patches = 512^2 tokens x 8 levels, cut into
# 64x64-token tiles overlapping by 8 tokens: stride 56, 9 x 9 = 81 tiles.
FACE_ROLLOUT = Workload("face_rollout_81x16x8x64x64_d64_w3x7x7", 1005, "bf16",
                        81, 16, 8, 64, 64, 64, 3, 7, 7, tiling=(9, 9, 56, 56))

WORKLOADS = {w.name: w for w in (TINY_F32, SMALL_BF16, TRAIN_TILE, TRAIN_TILE_BWD, FACE_ROLLOUT)}

# The paper's own shapes (App. B.1): 24 levels, NA3D window 9x9x9 on tiles of
# 64x64 or 128x128 cells = 16x16 or 32x32 tokens (16 heads, head_dim 64); the
# column-wise blocks attend along all 24 levels of a column (window 24x1x1);
# the de-aliasing decoder's NA3D runs at full resolution, 64x64 pixels x 24
# levels, with width 128 (one head of 128 channels here).
PAPER_TILE16 = Workload("paper_96x16x24x16x16_d64_w9x9x9", 1006, "bf16",
                        96, 16, 24, 16, 16, 64, 9, 9, 9)
PAPER_TILE32 = Workload("paper_24x16x24x32x32_d64_w9x9x9", 1007, "bf16",
                        24, 16, 24, 32, 32, 64, 9, 9, 9)
PAPER_COLUMN = Workload("paper_column_96x16x24x16x16_d64_w24x1x1", 1008, "bf16",
                        96, 16, 24, 16, 16, 64, 24, 1, 1)
PAPER_DECODER = Workload("paper_decoder_2x1x24x64x64_d128_w9x9x9", 1009, "bf16",
                         2, 1, 24, 64, 64, 128, 9, 9, 9)
# The 3x7x7 window of the face workload at the paper's 24 levels (the window
# sweep of App. B.2 at full depth), on the 32x32-token tiles above.
Z24_TILE = Workload("paper_24x16x24x32x32_d64_w3x7x7", 1010, "bf16",
                    24, 16, 24, 32, 32, 64, 3, 7, 7)
PAPER_WORKLOADS = {w.name: w for w in (PAPER_TILE16, PAPER_TILE32, PAPER_COLUMN, PAPER_DECODER, Z24_TILE)}

FACE_OVERLAP = 8  # tokens shared by neighbouring tiles of the face rollout step


def ramp_window_1d(L: int, overlap: int) -> np.ndarray:
    """Per-axis linear ramp sampled at cell centres, 1 in the interior.

    w(i) = min(1, (i + 1/2)/overlap, (L - i - 1/2)/overlap); for overlap 8 every value
    is a multiple of 1/16, so 2D products are exact in float32."""
    i = np.arange(L, dtype=np.float64)
    w = np.minimum(1.0, np.minimum((i + 0.5) / overlap, (L - i - 0.5) / overlap))
    return w


def ramp_window_2d(Ht: int, Wt: int, overlap: int) -> np.ndarray:
    """Separable 2D linear-ramp window [Ht*Wt] float32 (the blend's W)."""
    w = np.outer(ramp_window_1d(Ht, overlap), ramp_window_1d(Wt, overlap))
    return w.astype(np.float32).reshape(-1)


def tophat_window_2d(Ht: int, Wt: int, halo: int) -> np.ndarray:
    """2D top-hat window: 1 in the interior, 0 in a halo of ``halo`` cells."""
    w = np.zeros((Ht, Wt), dtype=np.float32)
    w[halo:Ht - halo, halo:Wt - halo] = 1.0
    return w.reshape(-1)

"""Host checks of the bench's algorithmic byte counts (no GPU)."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402


def brute_overlap_bytes(nty, ntx, Ht, Wt, sy, sx, P, C, elem=2):
    """Tile by tile: every tile value of a cell some other tile also covers is read once;
    every such face cell is written once."""
    Hf, Wf = (nty - 1) * sy + Ht, (ntx - 1) * sx + Wt
    cover = np.zeros((Hf, Wf), int)
    for a in range(nty):
        for b in range(ntx):
            cover[a * sy:a * sy + Ht, b * sx:b * sx + Wt] += 1
    multi = np.zeros((Hf, Wf), bool)
    for a in range(nty):
        for b in range(ntx):
            ys = np.arange(a * sy, a * sy + Ht)
            xs = np.arange(b * sx, b * sx + Wt)
            ny = np.array([sum(t * sy <= y < t * sy + Ht for t in range(nty)) for y in ys])
            nx = np.array([sum(t * sx <= x < t * sx + Wt for t in range(ntx)) for x in xs])
            multi[np.ix_(ys, xs)] |= (ny[:, None] > 1) | (nx[None, :] > 1)
    reads = cover[multi].sum()
    return float((reads + multi.sum()) * P * C * elem)


def test_overlap_stitch_bytes_match_brute_force():
    for case in [(3, 3, 32, 32, 24, 24), (2, 3, 36, 36, 28, 28), (2, 2, 16, 16, 16, 16), (3, 4, 20, 24, 14, 17)]:
        assert bench.overlap_stitch_bytes(*case, 2, 8) == brute_overlap_bytes(*case, 2, 8)


def test_face_tiling_overlap_stitch_bytes():
    # 9 x 9 tiles of 64 x 64 cells at stride 56 on a 512 x 512 face, 128 planes x 64 bf16 channels
    b = bench.overlap_stitch_bytes(9, 9, 64, 64, 56, 56, 128, 64)
    assert b == brute_overlap_bytes(9, 9, 64, 64, 56, 56, 128, 64)
    multi_cells = 512 * 512 - 448 * 448   # cells outside the 48 x 48 single-cover interiors
    assert b == (131072 + multi_cells) * 128 * 64 * 2

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


def test_face_parity_reference_is_the_oracle_stitch():
    """The bench's sampled face reference (oracle forward of each covering tile's
    query, stitched in float64) equals the oracle's whole-tile forward stitched
    by brute force over every tile, at every sampled cell; the sample holds every
    cell category on every plane."""
    import oracle
    from oracle import geometry as G
    from paper_2606_31248_amd import inputs as I

    wl = I.Workload("face_small_9x2x8x32x32", 1205, "bf16", 9, 2, 8, 32, 32, 64, 3, 7, 7, tiling=(3, 3, 24, 24))
    qkv = wl.qkv()
    win = I.ramp_window_2d(wl.H, wl.W, 8)
    cells = bench.face_sample_cells(wl)
    ref, carried, meta = bench.face_reference(wl, qkv, cells, win)
    assert meta["planes"] == wl.heads * wl.Z and meta["n_cells"] == 16 * wl.heads * wl.Z
    pl = wl.placement()
    c32 = G.tile_coords(pl.face, pl.oy, pl.ox, wl.H, wl.W).astype(np.float32)
    ro, _ = oracle.na3d_fwd(*(oracle.widen(a, "bf16") for a in qkv), (3, 7, 7), wl.scale, coords=c32)
    nty, ntx, sy, sx = wl.tiling
    num = np.zeros((wl.heads * wl.Z, 80, 80, wl.d))
    den = np.zeros((80, 80, 1))
    w2 = win.reshape(wl.H, wl.W, 1).astype(np.float64)
    planes = ro.reshape(9, wl.heads * wl.Z, wl.H, wl.W, wl.d)
    for a in range(nty):
        for b in range(ntx):
            num[:, a * sy:a * sy + wl.H, b * sx:b * sx + wl.W] += w2 * planes[a * ntx + b]
            den[a * sy:a * sy + wl.H, b * sx:b * sx + wl.W] += w2
    brute = (num / den)[cells[0], cells[1], cells[2]]
    assert np.max(np.abs(ref - brute)) <= 1e-12 * np.max(np.abs(brute))
    assert np.all(carried > 0)
    # the categories: single-cover, y strip, x strip, 4-tile corner and face corners are all present
    ny = np.array([sum(0 <= y - t * sy < wl.H for t in range(nty)) for y in range(80)])
    nx = np.array([sum(0 <= x - t * sx < wl.W for t in range(ntx)) for x in range(80)])
    kinds = set(zip(ny[cells[1]], nx[cells[2]]))
    assert {(1, 1), (2, 1), (1, 2), (2, 2)} <= kinds
    assert np.any((cells[1] == 0) & (cells[2] == 0)) and np.any((cells[1] == 79) & (cells[2] == 79))

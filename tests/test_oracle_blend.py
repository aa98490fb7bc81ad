"""Pins of the oracle's tile stitching S = D^-1 P^T W and extraction P (App. F) -- CPU only."""
import numpy as np
import pytest

import oracle
from oracle import geometry as G
from paper_2606_31248_amd import inputs


def regular_P(nty, ntx, Ht, Wt, sy, sx, Hf, Wf):
    """Dense extraction operator P: (tile cells) x (face cells), built from index arithmetic."""
    rows = []
    for a in range(nty):
        for b in range(ntx):
            for i in range(Ht):
                for j in range(Wt):
                    rows.append((a * sy + i) * Wf + (b * sx + j))
    P = np.zeros((len(rows), Hf * Wf))
    P[np.arange(len(rows)), rows] = 1.0
    return P


def face_field(P, Hf, Wf, C, seed, dtype):
    return inputs.gaussian((P, Hf, Wf, C), seed, inputs.STREAM_FIELD, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_stitch_matches_operator_form(dtype):
    # S y = D^-1 P^T (W y), D = P^T W 1, written as explicit matrices (Eq. stitch).
    nty, ntx, Ht, Wt, sy, sx = 3, 4, 12, 10, 9, 7
    Hf, Wf, P_, C = (nty - 1) * sy + Ht, (ntx - 1) * sx + Wt, 2, 3
    T = nty * ntx
    tiles = inputs.gaussian((T, P_, Ht, Wt, C), 7, inputs.STREAM_FIELD, dtype)
    win = inputs.ramp_window_2d(Ht, Wt, 3)
    out = oracle.tile_blend(tiles, nty, ntx, sy, sx, win, Hf, Wf, dtype)
    Pm = regular_P(nty, ntx, Ht, Wt, sy, sx, Hf, Wf)
    Wd = np.tile(win.astype(np.float64), T)
    D = Pm.T @ Wd
    y = oracle.widen(tiles, dtype)                       # [T, P, Ht, Wt, C]
    y = np.moveaxis(y, 1, 0).reshape(P_, T * Ht * Wt, C)  # [P, tile cells, C]
    ref = (Pm.T @ (Wd[None, :, None] * y)) / D[None, :, None]
    ref = ref.reshape(P_, Hf, Wf, C)
    got = oracle.widen(out, dtype)
    tol = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -23
    np.testing.assert_allclose(got, ref, rtol=tol, atol=1e-30)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_constant_field_is_reproduced_exactly(dtype):
    nty, ntx, Ht, Wt, s = 3, 3, 16, 16, 12
    Hf = Wf = 2 * s + Ht
    val = inputs.gaussian((1,), 3, 0, dtype)[0]
    tiles = np.full((9, 2, Ht, Wt, 4), val)
    win = inputs.ramp_window_2d(Ht, Wt, 4)
    out = oracle.tile_blend(tiles, nty, ntx, s, s, win, Hf, Wf, dtype)
    assert np.all(out == val)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_round_trip_stitch_of_extract_is_identity(dtype):
    # S(P F) = F exactly for the face-rollout tiling geometry (scaled down in P and C).
    nty = ntx = 9
    Ht = Wt = 64
    s = 56
    Hf = Wf = 512
    F = face_field(2, Hf, Wf, 3, 11, dtype)
    tiles = oracle.tile_extract(F, nty, ntx, Ht, Wt, s, s)
    win = inputs.ramp_window_2d(Ht, Wt, inputs.FACE_OVERLAP)
    out = oracle.tile_blend(tiles, nty, ntx, s, s, win, Hf, Wf, dtype)
    assert np.array_equal(out, F)


def test_tophat_window_reduces_to_crop():
    # A top-hat window (1 inside, 0 in the halo) turns stitching into a crop of tile interiors.
    nty, ntx, Ht, Wt, halo = 3, 2, 12, 12, 2
    s = Ht - 2 * halo
    Hf, Wf = (nty - 1) * s + Ht, (ntx - 1) * s + Wt
    tiles = inputs.gaussian((nty * ntx, 1, Ht, Wt, 2), 5, inputs.STREAM_FIELD, "bf16")
    win = inputs.tophat_window_2d(Ht, Wt, halo)
    out = oracle.tile_blend(tiles, nty, ntx, s, s, win, Hf, Wf, "bf16")
    exp = np.zeros_like(out)
    for a in range(nty):
        for b in range(ntx):
            t = a * ntx + b
            exp[:, a * s + halo:a * s + Ht - halo, b * s + halo:b * s + Wt - halo] = \
                tiles[t, :, halo:Ht - halo, halo:Wt - halo]
    assert np.array_equal(out, exp)
    # the outer halo of the face is weighted by no tile: D == 0 -> 0
    assert np.all(out[:, :halo] == 0) and np.all(out[:, :, :halo] == 0)


def test_ramp_windows_partition_unity_on_face_tiling():
    # Overlapping ramps of neighbouring tiles sum to one; interior weights are one.
    w = inputs.ramp_window_1d(64, inputs.FACE_OVERLAP)
    acc = np.zeros(512)
    for a in range(9):
        acc[a * 56:a * 56 + 64] += w
    assert np.all(acc[8:-8] == 1.0)
    assert np.all(w * 256 == np.round(w * 256))


def test_extract_is_a_copy():
    F = face_field(3, 40, 50, 5, 13, "bf16")
    t = oracle.tile_extract(F, 2, 3, 24, 20, 16, 15)
    for a in range(2):
        for b in range(3):
            assert np.array_equal(t[a * 3 + b], F[:, a * 16:a * 16 + 24, b * 15:b * 15 + 20])


def test_blend_rejects_tiles_past_the_face():
    tiles = np.zeros((4, 1, 8, 8, 1), np.float32)
    with pytest.raises(ValueError):
        oracle.tile_blend(tiles, 2, 2, 8, 8, np.ones(64, np.float32), 15, 16, "f32")


# ----------------------------------------------------------------------------- KBD window

@pytest.mark.parametrize("overlap,beta", [(8, 4 * np.pi), (8, 2.0), (16, 10.0), (3, 1.0)])
def test_kbd_taper_is_scipys_kaiser_bessel_derived_half(overlap, beta):
    from scipy.signal.windows import kaiser_bessel_derived
    ref = kaiser_bessel_derived(2 * overlap, beta)[:overlap]
    np.testing.assert_allclose(G.kbd_taper(overlap, beta), ref, rtol=0, atol=1e-14)


def test_kbd_taper_is_power_complementary():
    # Princen-Bradley: w[n]^2 + w[overlap-1-n]^2 = 1 for the rising half and its mirror
    t = G.kbd_taper(8, 4 * np.pi)
    np.testing.assert_allclose(t ** 2 + t[::-1] ** 2, 1.0, atol=1e-14)


def test_kbd_window_2d_shape_and_interior():
    w = G.kbd_window_2d(64, 40, 8, 4 * np.pi).reshape(64, 40)
    assert np.all(w[8:56, 8:32] == 1.0)
    t = G.kbd_taper(8, 4 * np.pi)
    np.testing.assert_allclose(w[3, 20], t[3], atol=0)
    np.testing.assert_allclose(w[63, 39], t[0] * t[0], atol=1e-16)
    assert np.all(w > 0) and np.all(w <= 1)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_single_cover_cells_return_the_tile_value(dtype):
    """A face cell that one tile alone covers stitches to w v / w: the tile's own
    value bit for bit for any positive float32 weight (one rounding of the
    product, one of the quotient, then the store rounding), 0 where w = 0, and
    +0 for -0 (the multiply-add starts from +0).  The fused face step stores
    these cells from the forward on this basis."""
    nty, ntx, Ht, Wt, sy, sx = 3, 3, 12, 14, 9, 10
    Hf, Wf, P_, C = (nty - 1) * sy + Ht, (ntx - 1) * sx + Wt, 2, 4
    T = nty * ntx
    r = np.random.default_rng(90)
    tiles = inputs.gaussian((T, P_, Ht, Wt, C), 90, inputs.STREAM_FIELD, dtype)
    neg_zero = np.uint16(0x8000) if dtype == "bf16" else np.float32(-0.0)
    tiles[r.random(tiles.shape) < 0.05] = neg_zero
    # arbitrary positive float32 weights (not dyadic), some exactly 0
    win = r.uniform(0.01, 3.0, Ht * Wt).astype(np.float32)
    win[r.random(Ht * Wt) < 0.1] = 0.0
    out = oracle.tile_blend(tiles, nty, ntx, sy, sx, win, Hf, Wf, dtype)
    ny = np.array([sum(a * sy <= y < a * sy + Ht for a in range(nty)) for y in range(Hf)])
    nx = np.array([sum(b * sx <= x < b * sx + Wt for b in range(ntx)) for x in range(Wf)])
    bits = (lambda a: a) if dtype == "bf16" else (lambda a: a.view(np.uint32))
    zero = 0
    singles = 0
    for a in range(nty):
        for b in range(ntx):
            for i in range(Ht):
                for j in range(Wt):
                    y, x = a * sy + i, b * sx + j
                    if ny[y] != 1 or nx[x] != 1:
                        continue
                    singles += 1
                    v = bits(tiles[a * ntx + b, :, i, j, :])
                    expect = np.where(v == bits(np.array([neg_zero]))[0], zero, v)
                    if win[i * Wt + j] == 0.0:
                        expect = np.zeros_like(v)
                    assert np.array_equal(bits(out[:, y, x, :]), expect), (a, b, i, j)
    assert singles > 0.4 * Hf * Wf

"""GPU parity of the face step with the stitch fused into the forward.

strata_na3d_fwd_stitch followed by strata_tile_blend_overlap must give the face
that strata_na3d_fwd_ex followed by strata_tile_blend gives, bit for bit (the
stitch of a cell covered by one tile is w v / w = v, or 0 where w = 0, with -0
turned into +0 by the fused multiply-add from +0); and the face must match the
oracle's forward and stitch under the bf16 rule.  Cases: the fused kernel at
small tilings (overlaps that split query sub-blocks, ragged query blocks, no
overlap, a ragged head group, a window with zero weights, random non-dyadic
weights, every option with saturated gates) and at the full face-rollout size;
the shapes and tilings that fall back to forward + whole stitch; and the
overlap-only stitch on its own against the oracle, in its bf16 form and in the
forms where it stitches the whole face."""
import numpy as np
import pytest
import torch

import oracle
from oracle import geometry as G
from paper_2606_31248_amd import binding as B
from paper_2606_31248_amd import inputs as I
from paper_2606_31248_amd import pipeline
from _util import BF16_REL_RMS, bf16_half_ulp, dev_tensor, host_bits

pytestmark = pytest.mark.gpu


def tiling_case(nty, ntx, H, W, sy, sx, heads=2, Z=8, d=64, dtype="bf16", seed=70):
    T = nty * ntx
    shape = (T, heads, Z, H, W, d)
    q, k, v = (I.gaussian(shape, seed, s, dtype) for s in (I.STREAM_Q, I.STREAM_K, I.STREAM_V))
    Hf, Wf = (nty - 1) * sy + H, (ntx - 1) * sx + W
    # tile origins on face 0 at the token positions of the tiling (their coordinates)
    face = np.zeros(T, np.int64)
    oy = np.repeat(np.arange(nty) * sy, ntx)
    ox = np.tile(np.arange(ntx) * sx, nty)
    coords = G.tile_coords(face, oy, ox, H, W).astype(np.float32)
    return shape, (q, k, v), coords, Hf, Wf


def run_both(shape, qkv, coords, tiling, window, win, dtype="bf16", opts=None, scale=None):
    """Fused and unfused face steps on the same device inputs: (fused face, plain face, plain tiles, lse pair)."""
    T, heads, Z, H, W, d = shape
    nty, ntx, sy, sx = tiling
    Hf, Wf = (nty - 1) * sy + H, (ntx - 1) * sx + W
    qd, kd, vd = (dev_tensor(a, dtype) for a in qkv)
    c = torch.from_numpy(coords).cuda()
    cs = torch.empty((T, H, W, d // 2, 2), dtype=torch.float32, device="cuda")
    B.strata_stereorope_phases(c, d, pipeline.ROPE_BASE, cs)
    desc = B.desc_for(qd, window, scale or 1.0 / np.sqrt(d))
    wd = torch.from_numpy(win).cuda()
    tiles_a, tiles_b = torch.empty_like(qd), torch.empty_like(qd)
    face_a = torch.full((heads * Z, Hf, Wf, d), 7.0, dtype=qd.dtype, device="cuda")
    face_b = torch.empty_like(face_a)
    lse_a = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    lse_b = torch.empty_like(lse_a)
    B.strata_na3d_fwd_stitch(desc, opts, qd, kd, vd, cs, tiles_a, lse_a, nty, ntx, sy, sx, wd, face_a)
    B.strata_tile_blend_overlap(tiles_a.view(T, heads * Z, H, W, d), nty, ntx, sy, sx, wd, face_a)
    B.strata_na3d_fwd_ex(desc, opts, qd, kd, vd, cs, tiles_b, lse_b)
    B.strata_tile_blend(tiles_b.view(T, heads * Z, H, W, d), nty, ntx, sy, sx, wd, face_b)
    torch.cuda.synchronize()
    return face_a, face_b, tiles_b, (lse_a, lse_b)


@pytest.mark.parametrize("nty,ntx,H,W,sy,sx,heads", [
    (3, 3, 32, 32, 24, 24, 2),   # overlap 8 on whole 4x4 query sub-blocks
    (2, 3, 36, 36, 28, 28, 2),   # ragged 8x8 query blocks
    (2, 2, 32, 40, 27, 29, 2),   # overlaps of 5 and 11 cut through sub-blocks
    (2, 2, 16, 16, 16, 16, 2),   # no overlap: every cell goes straight to the face
    (1, 3, 24, 32, 24, 17, 2),   # one tile row
    (2, 2, 24, 24, 16, 16, 11),  # two head groups of 8 and 3 heads: face planes h Z + z
])
def test_fused_face_step_bit_exact(nty, ntx, H, W, sy, sx, heads):
    shape, qkv, coords, Hf, Wf = tiling_case(nty, ntx, H, W, sy, sx, heads=heads)
    win = I.ramp_window_2d(H, W, max(H - sy, W - sx, 1))
    fa, fb, _, (la, lb) = run_both(shape, qkv, coords, (nty, ntx, sy, sx), (3, 7, 7), win)
    assert np.array_equal(host_bits(fa), host_bits(fb))
    assert torch.equal(la, lb)


def test_fused_face_step_matches_oracle():
    """The fused face against the oracle's stitch of the oracle's exact tile outputs.

    The face stores the stitch of bf16 tile values, so beside the bf16 rule
    (half an ulp of the exact face value + 2e-2 RMS) each cell may carry the
    weighted average of its tiles' storage rounding: the oracle's stitch of half
    an ulp of each exact tile value."""
    nty, ntx, H, W, s = 3, 3, 32, 32, 24
    shape, qkv, coords, Hf, Wf = tiling_case(nty, ntx, H, W, s, s, seed=71)
    win = I.ramp_window_2d(H, W, I.FACE_OVERLAP)
    fa, _, _, _ = run_both(shape, qkv, coords, (nty, ntx, s, s), (3, 7, 7), win)
    ro, _ = oracle.na3d_fwd(*(oracle.widen(a, "bf16") for a in qkv), (3, 7, 7), 1.0 / 8.0, coords=coords)
    T, heads, Z, _, _, d = shape
    planes = (T, heads * Z, H, W, d)
    ref = oracle.tile_blend(ro.reshape(planes).astype(np.float32), nty, ntx, s, s, win, Hf, Wf, "f32")
    ref = ref.astype(np.float64)
    tile_round = oracle.tile_blend(bf16_half_ulp(ro).reshape(planes).astype(np.float32), nty, ntx, s, s, win,
                                   Hf, Wf, "f32").astype(np.float64)
    got = I.bf16_bits_to_f32(host_bits(fa)).astype(np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    excess = np.abs(got - ref) - bf16_half_ulp(ref) - tile_round
    assert float(np.max(excess)) <= BF16_REL_RMS * rms, (float(np.max(excess)), BF16_REL_RMS * rms)


def test_fused_face_step_zero_weights():
    """A top-hat window: cells one tile covers with weight 0 become 0, overlap cells with D = 0 as well."""
    nty, ntx, H, W, s = 3, 3, 32, 32, 24
    shape, qkv, coords, Hf, Wf = tiling_case(nty, ntx, H, W, s, s, seed=72)
    win = I.tophat_window_2d(H, W, 2)
    fa, fb, _, _ = run_both(shape, qkv, coords, (nty, ntx, s, s), (3, 7, 7), win)
    bits = host_bits(fa)
    assert np.array_equal(bits, host_bits(fb))
    assert np.all(bits[:, :2] == 0) and np.all(bits[:, :, :2] == 0)


def test_fused_face_step_arbitrary_weights():
    """Random positive float32 weights (not dyadic: the stitch rounds w v and w v / w), 10% of them 0."""
    nty, ntx, H, W, s = 3, 3, 32, 32, 24
    shape, qkv, coords, Hf, Wf = tiling_case(nty, ntx, H, W, s, s, seed=77)
    r = np.random.default_rng(77)
    win = r.uniform(0.01, 3.0, H * W).astype(np.float32)
    win[r.random(H * W) < 0.1] = 0.0
    fa, fb, _, _ = run_both(shape, qkv, coords, (nty, ntx, s, s), (3, 7, 7), win)
    assert np.array_equal(host_bits(fa), host_bits(fb))


@pytest.mark.parametrize("vmul,weights", [
    (2.0 ** 12, (2.0 ** 115, 2.0 ** 116, 0.75, 1.0)),  # w v overflows float32: the stitch gives inf
    (2.0 ** -120, (2.0 ** -20, 2.0 ** -9, 0.5)),  # w v underflows to float32 subnormals
    (1.0, (1e-3, 3e-40, 1.0, 7.0)),               # a subnormal weight, and weights outside [2^-8, 1]
])
def test_fused_face_step_weights_outside_unit_range(vmul, weights):
    """Single-cover cells with weights outside [2^-8, 1] take the stitch's own
    arithmetic fma(w, v, +0) / w in the fused forward: the face equals forward +
    whole stitch bit for bit, including overflow to inf and subnormal products."""
    nty, ntx, H, W, s = 2, 2, 32, 32, 24
    shape, (q, k, v), coords, Hf, Wf = tiling_case(nty, ntx, H, W, s, s, seed=79)
    v = I.f32_to_bf16_bits((I.bf16_bits_to_f32(v) * np.float32(vmul)).astype(np.float32))
    win = np.array(weights, np.float32)[np.arange(H * W) % len(weights)]
    fa, fb, _, _ = run_both(shape, (q, k, v), coords, (nty, ntx, s, s), (3, 7, 7), win)
    assert np.array_equal(host_bits(fa), host_bits(fb))
    if vmul > 1:
        assert np.any(np.isinf(I.bf16_bits_to_f32(host_bits(fa))))


@pytest.mark.parametrize("qk_norm,gate", [(True, None), (False, "token"), (True, "channel")])
def test_fused_face_step_options(qk_norm, gate):
    """QK RMSNorm and the gate; gate logits of -200 on some tokens drive outputs to +-0."""
    nty, ntx, H, W, s = 2, 2, 32, 32, 24
    shape, qkv, coords, Hf, Wf = tiling_case(nty, ntx, H, W, s, s, seed=73)
    g = None
    if gate is not None:
        gshape = shape[:-1] if gate == "token" else shape
        gf = I.bf16_bits_to_f32(I.gaussian(gshape, 73, I.STREAM_GATE, "bf16"))
        mask = np.random.default_rng(73).random(gshape[:5]) < 0.3
        gf = np.where(mask.reshape(mask.shape + (1,) * (len(gshape) - 5)), np.float32(-200.0), gf)
        g = dev_tensor(I.f32_to_bf16_bits(gf.astype(np.float32)), "bf16")
    opts = B.make_opts(qk_norm=qk_norm, eps=1e-6, gate=g)
    win = I.ramp_window_2d(H, W, I.FACE_OVERLAP)
    fa, fb, tiles_b, _ = run_both(shape, qkv, coords, (nty, ntx, s, s), (3, 7, 7), win, opts=opts)
    assert np.array_equal(host_bits(fa), host_bits(fb))
    if gate is not None:  # the case the zero-sign rule is for is present
        assert np.count_nonzero(host_bits(tiles_b) == 0x8000) > 0


@pytest.mark.parametrize("case", ["window_5x9x9", "f32", "extent_over_twice_stride", "uncovered_margin"])
def test_fused_face_step_fallbacks(case):
    """Shapes and tilings outside the fused kernel: forward + whole stitch, then the overlap call."""
    window, dtype = (3, 7, 7), "bf16"
    nty, ntx, H, W, sy, sx = 2, 2, 24, 24, 16, 16
    if case == "window_5x9x9":
        window = (5, 9, 9)
    elif case == "f32":
        dtype = "f32"
    elif case == "extent_over_twice_stride":
        nty, ntx, sy, sx = 3, 3, 10, 10
    shape, qkv, coords, Hf, Wf = tiling_case(nty, ntx, H, W, sy, sx, dtype=dtype, seed=74)
    win = I.ramp_window_2d(H, W, 8)
    if case == "uncovered_margin":  # a face wider than the tiling: not the overlap form
        T, heads, Z, _, _, d = shape
        qd, kd, vd = (dev_tensor(a, dtype) for a in qkv)
        desc = B.desc_for(qd, window, 0.125)
        wd = torch.from_numpy(win).cuda()
        tiles = torch.empty_like(qd)
        face_a = torch.full((heads * Z, Hf + 3, Wf + 2, d), 7.0, dtype=qd.dtype, device="cuda")
        face_b = torch.empty_like(face_a)
        B.strata_na3d_fwd_stitch(desc, None, qd, kd, vd, None, tiles, None, nty, ntx, sy, sx, wd, face_a)
        B.strata_tile_blend_overlap(tiles.view(T, heads * Z, H, W, d), nty, ntx, sy, sx, wd, face_a)
        B.strata_tile_blend(tiles.view(T, heads * Z, H, W, d), nty, ntx, sy, sx, wd, face_b)
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(face_a), host_bits(face_b))
        return
    fa, fb, _, (la, lb) = run_both(shape, qkv, coords, (nty, ntx, sy, sx), window, win, dtype=dtype)
    assert np.array_equal(host_bits(fa), host_bits(fb))
    assert torch.equal(la, lb)


def test_overlap_stitch_alone_against_oracle():
    """The overlap-only stitch writes the oracle's stitch at every cell two tiles cover and nothing else."""
    nty, ntx, Ht, Wt, sy, sx, P, C = 3, 4, 20, 24, 14, 17, 3, 16
    Hf, Wf = (nty - 1) * sy + Ht, (ntx - 1) * sx + Wt
    tiles = I.gaussian((nty * ntx, P, Ht, Wt, C), 75, I.STREAM_FIELD, "bf16")
    win = I.ramp_window_2d(Ht, Wt, 7)
    td = dev_tensor(tiles, "bf16")
    out = torch.full((P, Hf, Wf, C), 7.0, dtype=torch.bfloat16, device="cuda")
    B.strata_tile_blend_overlap(td, nty, ntx, sy, sx, torch.from_numpy(win).cuda(), out)
    ref = oracle.tile_blend(tiles, nty, ntx, sy, sx, win, Hf, Wf, "bf16")
    ny = np.array([sum(a * sy <= y < a * sy + Ht for a in range(nty)) for y in range(Hf)])
    nx = np.array([sum(b * sx <= x < b * sx + Wt for b in range(ntx)) for x in range(Wf)])
    multi = (ny[:, None] > 1) | (nx[None, :] > 1)
    got = host_bits(out)
    assert np.array_equal(got[:, multi], ref[:, multi])
    sentinel = np.uint16(0x40E0)  # bf16 7.0
    assert np.all(got[:, ~multi] == sentinel)


@pytest.mark.parametrize("dtype,C", [("f32", 4), ("bf16", 3), ("f32", 3)])
def test_overlap_stitch_fallback_stitches_every_cell(dtype, C):
    """Outside its bf16 / C % 8 == 0 form the overlap-only call stitches the whole face (oracle, bit for bit)."""
    nty, ntx, Ht, Wt, sy, sx, P = 3, 2, 12, 10, 9, 7, 2
    Hf, Wf = (nty - 1) * sy + Ht, (ntx - 1) * sx + Wt
    tiles = I.gaussian((nty * ntx, P, Ht, Wt, C), 78, I.STREAM_FIELD, dtype)
    win = I.ramp_window_2d(Ht, Wt, 3)
    td = dev_tensor(tiles, dtype)
    out = torch.full((P, Hf, Wf, C), 7.0, dtype=td.dtype, device="cuda")
    B.strata_tile_blend_overlap(td, nty, ntx, sy, sx, torch.from_numpy(win).cuda(), out)
    ref = oracle.tile_blend(tiles, nty, ntx, sy, sx, win, Hf, Wf, dtype)
    assert np.array_equal(host_bits(out), ref)


def test_fused_face_step_full_face_rollout():
    """The face-rollout step at full size (81 tiles x 16 heads x 8x64x64, 3x7x7): fused = plain, bit for bit."""
    wl = I.FACE_ROLLOUT
    nty, ntx, sy, sx = wl.tiling
    Hf, Wf = (nty - 1) * sy + wl.H, (ntx - 1) * sx + wl.W
    gen = torch.Generator(device="cuda").manual_seed(76)
    shape = wl.shape()
    q, k, v = (torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
               for _ in range(3))
    pl = wl.placement()
    geom = pipeline.TileGeometry(*(torch.from_numpy(a).cuda() for a in pl.as_int32()))
    _, cs = pipeline.stereo_phases(geom, wl.H, wl.W, wl.d)
    win = torch.from_numpy(I.ramp_window_2d(wl.H, wl.W, I.FACE_OVERLAP)).cuda()
    window = (wl.kz, wl.ky, wl.kx)
    fa = torch.empty((wl.heads * wl.Z, Hf, Wf, wl.d), dtype=torch.bfloat16, device="cuda")
    fb = torch.empty_like(fa)
    pipeline.face_step(q, k, v, geom, window, wl.scale, wl.tiling, win, fa, cs=cs, fused=True)
    pipeline.face_step(q, k, v, geom, window, wl.scale, wl.tiling, win, fb, cs=cs, fused=False)
    torch.cuda.synchronize()
    assert torch.equal(fa.view(torch.int16), fb.view(torch.int16))


def test_face_step_seeded_full_size_against_oracle():
    """The face-rollout step on the seeded inputs bench.py times (81 tiles x 16 heads
    x 8x64x64, 3x7x7, StereoRoPE, linear-ramp overlaps): 2048 face cells over all 128
    planes (face corners, single-cover cells, both overlap strips, four-tile corners)
    against the oracle's forward of the covering tiles' queries and its stitch
    (Sec. 3.2; App. F, Eq. stitch) -- the same check as the bench line's parity."""
    import bench  # the repository root is on sys.path (conftest)
    wl = I.FACE_ROLLOUT
    nty, ntx, sy, sx = wl.tiling
    Hf, Wf = (nty - 1) * sy + wl.H, (ntx - 1) * sx + wl.W
    qkv_host = wl.qkv()
    q, k, v = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda() for x in qkv_host)
    geom = pipeline.TileGeometry(*(torch.from_numpy(a).cuda() for a in wl.placement().as_int32()))
    win_np = I.ramp_window_2d(wl.H, wl.W, I.FACE_OVERLAP)
    face = torch.empty((wl.heads * wl.Z, Hf, Wf, wl.d), dtype=torch.bfloat16, device="cuda")
    pipeline.face_step(q, k, v, geom, (wl.kz, wl.ky, wl.kx), wl.scale, wl.tiling,
                       torch.from_numpy(win_np).cuda(), face, fused=True)
    torch.cuda.synchronize()
    del q, k, v
    cells = bench.face_sample_cells(wl)
    idx = torch.from_numpy((cells[0] * Hf + cells[1]) * Wf + cells[2]).cuda()
    rows = face.view(-1, wl.d).index_select(0, idx).float().cpu().numpy().astype(np.float64)
    par = bench.face_parity(wl, qkv_host, rows, cells, win_np)
    assert par["n_cells"] == 2048 and par["planes"] == wl.heads * wl.Z, par
    assert par["pass_r11"], par

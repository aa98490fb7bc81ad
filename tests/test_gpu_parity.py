"""GPU parity of every hot-path entry point against the CPU oracle (through the C ABI).

Rules: integer/index and blend/extract results bit-exact; float32 max abs error
<= 1e-5; bf16 max abs error <= 2e-2 * RMS of the oracle output; LSE (float32)
within 1e-5 (f32 inputs) or 2e-2 natural-log units (bf16 inputs)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import geometry as G
from paper_2606_31248_amd import binding as B
from paper_2606_31248_amd import inputs as I
from paper_2606_31248_amd import pipeline
from _util import LSE_ABS_BF16, bf16_half_ulp, check_close, dev_tensor, host_bits, host_f64, host_rows

pytestmark = pytest.mark.gpu

ROPE_BASE = pipeline.ROPE_BASE


def placement_dev(pl):
    f, oy, ox = pl.as_int32()
    return pipeline.TileGeometry(*(torch.from_numpy(a).cuda() for a in (f, oy, ox)))


def oracle_coords(pl, H, W):
    return G.tile_coords(pl.face, pl.oy, pl.ox, H, W).astype(np.float32)


def gpu_phases(coords32, d):
    c = torch.from_numpy(coords32).cuda()
    cs = torch.empty(coords32.shape[:3] + (d // 2, 2), dtype=torch.float32, device="cuda")
    B.strata_stereorope_phases(c, d, ROPE_BASE, cs)
    return cs


# ----------------------------------------------------------------------------- indexing

@pytest.mark.parametrize("L,k", [(1, 1), (7, 7), (8, 3), (8, 5), (16, 7), (32, 7), (64, 9), (64, 7),
                                 (512, 9), (5, 1), (13, 13)])
def test_axis_index_bit_exact(L, k):
    out = [torch.empty(L, dtype=torch.int32, device="cuda") for _ in range(3)]
    B.strata_na_axis_index(L, k, *out)
    ref = oracle.axis_index(L, k)
    for g, r in zip(out, ref):
        assert np.array_equal(g.cpu().numpy(), r)


# ----------------------------------------------------------------------------- coordinates

@pytest.mark.parametrize("wl", [I.TINY_F32, I.SMALL_BF16, I.FACE_ROLLOUT], ids=lambda w: w.name)
def test_stereo_coords_match_oracle(wl):
    pl = wl.placement()
    geom = placement_dev(pl)
    coords, _ = pipeline.stereo_phases(geom, wl.H, wl.W, wl.d)
    got = coords.cpu().numpy().astype(np.float64)
    ref = G.tile_coords(pl.face, pl.oy, pl.ox, wl.H, wl.W)
    # float64 arithmetic on both sides, stored as float32: within one float32 ulp
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(got - ref) <= ulp + 1e-30)


def test_phase_table_matches_oracle():
    wl = I.SMALL_BF16
    c32 = oracle_coords(wl.placement(), wl.H, wl.W)
    cs = gpu_phases(c32, wl.d).cpu().numpy().astype(np.float64)
    ref = oracle.rope_phases(c32, wl.d, ROPE_BASE)
    assert np.max(np.abs(cs - ref)) <= 1.2e-7


# ----------------------------------------------------------------------------- RoPE apply

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("transpose", [False, True])
def test_rope_apply_matches_oracle(dtype, transpose):
    shape = (3, 2, 3, 12, 20, 64)
    pl = I.random_placement(3, 12, 20, 77)
    c32 = oracle_coords(pl, 12, 20)
    x = I.gaussian(shape, 5, 0, dtype)
    xd = dev_tensor(x, dtype)
    y = torch.empty_like(xd)
    B.strata_stereorope_apply(xd, y, gpu_phases(c32, 64), transpose=transpose)
    ref = oracle.rope_apply(oracle.widen(x, dtype), c32, transpose=transpose, base=ROPE_BASE)
    check_close(host_f64(y), ref, dtype, "rope")
    if dtype == "bf16":  # one rounding of a float32 result: within 1 bf16 ulp of the exact value
        assert np.all(np.abs(host_f64(y) - ref) <= np.abs(ref) * 2.0 ** -7 + 1e-6)


def test_rope_apply_in_place_and_round_trip():
    shape = (2, 3, 2, 8, 8, 32)
    pl = I.random_placement(2, 8, 8, 78)
    cs = gpu_phases(oracle_coords(pl, 8, 8), 32)
    x = dev_tensor(I.gaussian(shape, 6, 0, "f32"), "f32")
    y = x.clone()
    B.strata_stereorope_apply(y, y, cs)
    B.strata_stereorope_apply(y, y, cs, transpose=True)
    assert torch.max(torch.abs(y - x)).item() <= 2e-6


# ----------------------------------------------------------------------------- NA3D forward

def run_fwd(wl_shape, window, dtype, seed, coords32=None, scale=None, want_lse=True):
    Bt, heads, Z, H, W, d = wl_shape
    q, k, v = (I.gaussian(wl_shape, seed, s, dtype) for s in (0, 1, 2))
    scale = scale or 1.0 / np.sqrt(d)
    qd, kd, vd = (dev_tensor(a, dtype) for a in (q, k, v))
    cs = gpu_phases(coords32, d) if coords32 is not None else None
    out = torch.empty_like(qd)
    lse = torch.empty(wl_shape[:-1], dtype=torch.float32, device="cuda") if want_lse else None
    B.strata_na3d_fwd(B.desc_for(qd, window, scale), qd, kd, vd, cs, out, lse)
    torch.cuda.synchronize()
    return (q, k, v), out, lse, scale


def test_fwd_tiny_f32_full():
    wl = I.TINY_F32
    c32 = oracle_coords(wl.placement(), wl.H, wl.W)
    (q, k, v), out, lse, scale = run_fwd(wl.shape(), (wl.kz, wl.ky, wl.kx), "f32", wl.seed, c32)
    ro, rl = oracle.na3d_fwd(*(oracle.widen(a, "f32") for a in (q, k, v)), (wl.kz, wl.ky, wl.kx), scale,
                             coords=c32)
    check_close(host_f64(out), ro, "f32", "out")
    assert np.max(np.abs(host_f64(lse) - rl)) <= 1e-5


@pytest.mark.parametrize("shape,window", [
    ((1, 2, 9, 10, 11, 64), (9, 9, 9)),   # 729 keys: every lane of a query's wave takes 11-12
    ((2, 1, 3, 5, 6, 32), (1, 3, 5)),     # 15 keys: most lanes of the wave take none
])
def test_fwd_f32_one_wave_per_query(shape, window):
    """Small float32 problems run one wave per query (the lanes split the window's
    keys and merge their softmax states): full grids against the oracle."""
    pl = I.random_placement(shape[0], shape[3], shape[4], 95)
    c32 = oracle_coords(pl, shape[3], shape[4])
    (q, k, v), out, lse, scale = run_fwd(shape, window, "f32", 47, c32)
    ro, rl = oracle.na3d_fwd(*(oracle.widen(a, "f32") for a in (q, k, v)), window, scale, coords=c32)
    check_close(host_f64(out), ro, "f32", "out")
    assert np.max(np.abs(host_f64(lse) - rl)) <= 1e-5


@pytest.mark.parametrize("shape,window", [
    ((2, 3, 5, 19, 21, 64), (3, 7, 7)),     # ragged against 8x8 query blocks
    ((1, 2, 6, 24, 24, 64), (5, 9, 9)),
    ((2, 2, 3, 16, 12, 32), (3, 5, 7)),
    ((1, 1, 8, 32, 32, 64), (3, 7, 7)),
    ((2, 3, 8, 19, 21, 64), (3, 7, 7)),     # level-sweep kernel, ragged blocks
    ((1, 11, 8, 16, 24, 64), (3, 7, 7)),    # level-sweep kernel, ragged head group
    ((2, 2, 8, 7, 7, 64), (3, 7, 7)),       # level-sweep kernel, window = whole plane
    ((1, 3, 8, 7, 9, 64), (3, 7, 7)),       # level-sweep kernel, one-column blocks
    ((1, 3, 24, 19, 21, 64), (3, 7, 7)),    # level-sweep kernel at 24 levels, ragged blocks
    ((2, 9, 24, 8, 12, 64), (3, 7, 7)),     # ... a head run cut short (9 heads)
    ((1, 2, 4, 9, 9, 64), (1, 9, 9)),       # window = whole plane
    # the grouped level sweep (4 query levels per group): groups cut short by Z,
    # border-clamped level windows, ragged position blocks, two head groups
    ((1, 3, 5, 19, 21, 64), (3, 7, 7)),
    ((1, 2, 10, 16, 16, 64), (3, 7, 7)),
    ((1, 2, 7, 20, 17, 64), (5, 9, 9)),
    ((1, 9, 6, 9, 11, 64), (5, 9, 9)),
    ((1, 2, 9, 16, 16, 64), (9, 9, 9)),
    ((1, 2, 13, 12, 20, 64), (9, 9, 9)),
])
@pytest.mark.parametrize("rope", [True, False])
def test_fwd_bf16_full_oracle(shape, window, rope):
    pl = I.random_placement(shape[0], shape[3], shape[4], 91)
    c32 = oracle_coords(pl, shape[3], shape[4]) if rope else None
    (q, k, v), out, lse, scale = run_fwd(shape, window, "bf16", 21, c32)
    ro, rl = oracle.na3d_fwd(*(oracle.widen(a, "bf16") for a in (q, k, v)), window, scale, coords=c32)
    check_close(host_f64(out), ro, "bf16", "out")
    assert np.max(np.abs(host_f64(lse) - rl)) <= LSE_ABS_BF16


def sample_queries(shape, n, seed, tiles=None):
    """Random flat query indices plus every grid corner of the chosen tiles."""
    Bt, heads, Z, H, W, _ = shape
    r = np.random.default_rng(seed)
    tiles = list(range(Bt)) if tiles is None else tiles
    b = r.choice(tiles, n)
    idx = np.stack([b, r.integers(0, heads, n), r.integers(0, Z, n), r.integers(0, H, n),
                    r.integers(0, W, n)], 1)
    corners = [(t, h, z, y, x) for t in tiles[:2] for h in (0, heads - 1) for z in (0, Z - 1)
               for y in (0, 1, H - 1) for x in (0, 2, W - 1)]
    idx = np.concatenate([idx, np.array(corners)], 0)
    flat = (((idx[:, 0] * heads + idx[:, 1]) * Z + idx[:, 2]) * H + idx[:, 3]) * W + idx[:, 4]
    return np.unique(flat)


@pytest.mark.parametrize("wl", [I.SMALL_BF16, I.TRAIN_TILE, I.FACE_ROLLOUT, I.Z24_TILE], ids=lambda w: w.name)
def test_fwd_full_size_sampled(wl):
    """Full-size launch (the configuration the bench times); sampled outputs vs oracle.

    The oracle sees only the tiles the samples fall in (tiles are independent)."""
    shape = wl.shape()
    window = (wl.kz, wl.ky, wl.kx)
    pl = wl.placement()
    c32 = oracle_coords(pl, wl.H, wl.W)
    (q, k, v), out, lse, scale = run_fwd(shape, window, "bf16", wl.seed, c32)
    tiles = sorted({0, shape[0] // 2, shape[0] - 1})
    sel = sample_queries(shape, 3000, wl.seed, tiles)
    per_tile = shape[1] * wl.N
    sub = lambda a: oracle.widen(a[tiles], "bf16")
    # re-index samples into the tile subset
    tb = sel // per_tile
    local = np.searchsorted(tiles, tb) * per_tile + sel % per_tile
    ro, rl = oracle.na3d_fwd(sub(q), sub(k), sub(v), window, scale, coords=c32[tiles], sel=local)
    got = host_rows(out, sel, wl.d)
    check_close(got, ro, "bf16", "out")
    assert np.max(np.abs(host_rows(lse, sel) - rl)) <= LSE_ABS_BF16
    # a global property at full size: every output is a convex combination of v rows
    o = out.float()
    assert torch.isfinite(o).all()
    vmax = float(np.max(np.abs(oracle.widen(v, "bf16"))))
    assert torch.max(torch.abs(o)).item() <= vmax * (1 + 2.0 ** -7)


@pytest.mark.parametrize("Z,H,W,window", [(6, 20, 23, (3, 7, 5)), (8, 20, 23, (3, 7, 7))])
def test_fwd_one_hot_probe_membership_bit_exact(Z, H, W, window):
    """Q = K = 0, V one-hot on 64 probe tokens: outputs are non-zero exactly where
    the probe lies in the query's window (membership compared bit for bit)."""
    d = 64
    shape = (1, 2, Z, H, W, d)
    N = Z * H * W
    r = np.random.default_rng(5)
    probes = r.choice(N, (2, d), replace=False) if N >= d else None
    v = np.zeros(shape, np.float32)
    for h in range(2):
        for c in range(d):
            v.reshape(2, N, d)[h, probes[h, c], c] = 1.0
    zeros = np.zeros(shape, np.float32)
    qd = dev_tensor(I.f32_to_bf16_bits(zeros), "bf16")
    vd = dev_tensor(I.f32_to_bf16_bits(v), "bf16")
    out = torch.empty_like(qd)
    B.strata_na3d_fwd(B.desc_for(qd, window, 0.125), qd, qd, vd, None, out, None)
    ro, _ = oracle.na3d_fwd(zeros.astype(np.float64), zeros.astype(np.float64), v.astype(np.float64),
                            window, 0.125)
    got = host_f64(out)
    assert np.array_equal(got != 0, ro != 0)
    check_close(got, ro, "bf16", "probe")


@pytest.mark.parametrize("scale", [0.5, 1.0])
def test_fwd_large_logits_move_the_maximum(scale):
    """Logit spread of ~6-12 log2 units per key level: the running maximum moves
    between key levels (rescaling O and the row sums) for many queries."""
    shape = (1, 2, 8, 24, 24, 64)
    pl = I.random_placement(1, 24, 24, 17)
    c32 = oracle_coords(pl, 24, 24)
    (q, k, v), out, lse, _ = run_fwd(shape, (3, 7, 7), "bf16", 33, c32, scale=scale)
    ro, rl = oracle.na3d_fwd(*(oracle.widen(a, "bf16") for a in (q, k, v)), (3, 7, 7), scale, coords=c32)
    check_close(host_f64(out), ro, "bf16", "out")
    assert np.max(np.abs(host_f64(lse) - rl)) <= LSE_ABS_BF16


@pytest.mark.parametrize("sign", [-1.0, 1.0])
@pytest.mark.parametrize("window", [(3, 7, 7), (5, 9, 9)])
def test_fwd_uniform_extreme_logits(sign, window):
    """Every logit equal and about 200 (log2 units) from zero: without moving the
    softmax reference the weights would underflow to 0 (-) or overflow (+); the
    result must be the window mean of V, the log-sum-exp logit + ln K."""
    shape = (1, 2, 8, 16, 16, 64)
    scale = 0.125
    logit = sign * 200.0 / 1.4426950408889634          # natural-log units
    alpha = logit / (64 * scale)                          # q = alpha * ones, k = ones
    q = I.f32_to_bf16_bits(np.full(shape, alpha, np.float32))
    k = I.f32_to_bf16_bits(np.ones(shape, np.float32))
    v = I.gaussian(shape, 77, 2, "bf16")
    qd, kd, vd = (dev_tensor(a, "bf16") for a in (q, k, v))
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(B.desc_for(qd, window, scale), qd, kd, vd, None, out, lse)
    torch.cuda.synchronize()
    ro, rl = oracle.na3d_fwd(*(oracle.widen(a, "bf16") for a in (q, k, v)), window, scale)
    got = host_f64(out)
    assert np.isfinite(got).all()
    check_close(got, ro, "bf16", "out")
    # the logits themselves carry the float16 rounding of the scaled query (2^-11
    # relative), so the log-sum-exp bound grows with their size
    assert np.max(np.abs(host_f64(lse) - rl)) <= LSE_ABS_BF16 + 2.0 ** -10 * float(np.max(np.abs(rl)))


def test_fwd_deterministic_and_lse_optional():
    shape = (2, 4, 8, 32, 32, 64)
    pl = I.random_placement(2, 32, 32, 3)
    c32 = oracle_coords(pl, 32, 32)
    (q, k, v), out1, lse1, scale = run_fwd(shape, (3, 7, 7), "bf16", 9, c32)
    _, out2, _, _ = run_fwd(shape, (3, 7, 7), "bf16", 9, c32)
    _, out3, lse3, _ = run_fwd(shape, (3, 7, 7), "bf16", 9, c32, want_lse=False)
    assert torch.equal(out1, out2) and torch.equal(out1, out3)


# ----------------------------------------------------------------------------- blend / extract

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_blend_and_extract_bit_exact_face_geometry(dtype):
    nty = ntx = 9
    Ht = Wt = 64
    s = 56
    Hf = Wf = 512
    P, C = 3, 64 if dtype == "bf16" else 12
    tiles = I.gaussian((81, P, Ht, Wt, C), 31, I.STREAM_FIELD, dtype)
    win = I.ramp_window_2d(Ht, Wt, I.FACE_OVERLAP)
    td = dev_tensor(tiles, dtype)
    wd = torch.from_numpy(win).cuda()
    out = torch.empty((P, Hf, Wf, C), dtype=td.dtype, device="cuda")
    B.strata_tile_blend(td, nty, ntx, s, s, wd, out)
    ref = oracle.tile_blend(tiles, nty, ntx, s, s, win, Hf, Wf, dtype)
    assert np.array_equal(host_bits(out), ref)
    back = torch.empty_like(td)
    B.strata_tile_extract(out, nty, ntx, s, s, back)
    assert np.array_equal(host_bits(back), oracle.tile_extract(ref, nty, ntx, Ht, Wt, s, s))


@pytest.mark.parametrize("C", [1, 3, 8])
def test_blend_ragged_channels_and_uncovered_cells(C):
    # odd channel counts take the scalar path; a top-hat window leaves D == 0 cells
    nty, ntx, Ht, Wt, sy, sx = 2, 3, 10, 9, 7, 6
    Hf, Wf = (nty - 1) * sy + Ht + 3, (ntx - 1) * sx + Wt + 2
    tiles = I.gaussian((6, 2, Ht, Wt, C), 32, I.STREAM_FIELD, "bf16")
    win = I.tophat_window_2d(Ht, Wt, 1)
    td = dev_tensor(tiles, "bf16")
    out = torch.empty((2, Hf, Wf, C), dtype=torch.bfloat16, device="cuda")
    B.strata_tile_blend(td, nty, ntx, sy, sx, torch.from_numpy(win).cuda(), out)
    ref = oracle.tile_blend(tiles, nty, ntx, sy, sx, win, Hf, Wf, "bf16")
    assert np.array_equal(host_bits(out), ref)


@pytest.mark.parametrize("dtype,C", [("bf16", 8), ("bf16", 3), ("f32", 4), ("f32", 3)])
def test_extract_ragged_tiling_bit_exact(dtype, C):
    """Extraction on a tiling that leaves face margins uncovered: rows of 16-byte pieces (C a multiple of
    8 bf16 or 4 f32 values) and the element-wise kernel (other C), against the oracle's copy."""
    nty, ntx, Ht, Wt, sy, sx = 2, 3, 10, 9, 7, 6
    Hf, Wf = (nty - 1) * sy + Ht + 3, (ntx - 1) * sx + Wt + 2
    face = I.gaussian((2, Hf, Wf, C), 34, I.STREAM_FIELD, dtype)
    fd = dev_tensor(face, dtype)
    tiles = torch.empty((nty * ntx, 2, Ht, Wt, C), dtype=fd.dtype, device="cuda")
    B.strata_tile_extract(fd, nty, ntx, sy, sx, tiles)
    assert np.array_equal(host_bits(tiles), oracle.tile_extract(face, nty, ntx, Ht, Wt, sy, sx))


def test_blend_full_face_rollout_planes():
    """The face-rollout blend at full size; planes 0, 63, 127 compared bit for bit."""
    wl = I.FACE_ROLLOUT
    P = wl.heads * wl.Z
    tiles = I.gaussian((81, P, 64, 64, 64), 33, I.STREAM_FIELD, "bf16")
    win = I.ramp_window_2d(64, 64, I.FACE_OVERLAP)
    td = dev_tensor(tiles, "bf16")
    out = torch.empty((P, 512, 512, 64), dtype=torch.bfloat16, device="cuda")
    B.strata_tile_blend(td, 9, 9, 56, 56, torch.from_numpy(win).cuda(), out)
    planes = [0, 63, P - 1]
    ref = oracle.tile_blend(np.ascontiguousarray(tiles[:, planes]), 9, 9, 56, 56, win, 512, 512, "bf16")
    assert np.array_equal(host_bits(out[planes]), ref)


# ----------------------------------------------------------------------------- NA3D backward

def run_bwd(shape, window, dtype, seed, coords32=None, g_exp=None):
    """GPU forward (for out and lse) then backward; returns host inputs and GPU grads.

    g_exp: optional integer exponents (one per token, shape[:-1]); dO of a token is
    multiplied by 2^g_exp, which is exact in bf16."""
    (q, k, v), out, lse, scale = run_fwd(shape, window, dtype, seed, coords32)
    g = I.gaussian(shape, seed, I.STREAM_DO, dtype)
    if g_exp is not None:
        gf = I.bf16_bits_to_f32(g) * np.exp2(g_exp.astype(np.float32))[..., None]
        g = I.f32_to_bf16_bits(gf.astype(np.float32))
    qd, kd, vd, gd = (dev_tensor(a, dtype) for a in (q, k, v, g))
    cs = gpu_phases(coords32, shape[-1]) if coords32 is not None else None
    desc = B.desc_for(qd, window, scale)
    ws = torch.empty(B.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device="cuda")
    dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
    B.strata_na3d_bwd(desc, qd, kd, vd, cs, out, gd, lse, dq, dk, dv, ws)
    torch.cuda.synchronize()
    return (q, k, v, g), (dq, dk, dv), scale


@pytest.mark.parametrize("shape,window,dtype", [
    ((1, 2, 5, 11, 13, 64), (3, 7, 7), "bf16"),
    ((2, 1, 6, 12, 10, 64), (5, 9, 9), "bf16"),
    ((1, 2, 4, 9, 11, 32), (3, 5, 7), "f32"),
    ((1, 1, 3, 8, 8, 32), (1, 3, 5), "bf16"),
    ((1, 2, 6, 21, 19, 64), (3, 7, 7), "bf16"),
    ((1, 1, 9, 25, 22, 64), (5, 9, 9), "bf16"),
    # the key levels on a ring of waves (5x9x9): as many levels as the window,
    # and a long column in which every wave takes three key levels in turn
    ((1, 2, 5, 12, 12, 64), (5, 9, 9), "bf16"),
    ((1, 1, 13, 13, 9, 64), (5, 9, 9), "bf16"),
    # the balanced dK/dV kernel (two key levels x four 4x4 blocks) and the
    # 12-wave dQ (three query levels): ragged planes whose block counts are odd
    # (a group with one block, square runs of 2, 3 and 4, a 3 x 3 run whose
    # walk ends in a half step), an odd Z (a run with one key level, a last
    # group of one query level)
    ((1, 1, 7, 25, 23, 64), (5, 9, 9), "bf16"),
    ((1, 1, 11, 25, 13, 64), (9, 9, 9), "bf16"),
    # axes of 17-20 positions, where a single block's query box spans five
    # squares: dK/dV on the one-block kernel, dQ on the 12-wave kernel
    ((1, 1, 7, 18, 23, 64), (5, 9, 9), "bf16"),
    ((1, 1, 11, 13, 17, 64), (9, 9, 9), "bf16"),
])
@pytest.mark.parametrize("rope", [True, False])
def test_bwd_full_oracle(shape, window, dtype, rope):
    pl = I.random_placement(shape[0], shape[3], shape[4], 92)
    c32 = oracle_coords(pl, shape[3], shape[4]) if rope else None
    (q, k, v, g), grads, scale = run_bwd(shape, window, dtype, 41, c32)
    refs = oracle.na3d_bwd(*(oracle.widen(a, dtype) for a in (q, k, v, g)), window, scale, coords=c32)
    # f32 inputs: the forward output feeding D is float32, so the f32 bound applies
    for name, got, ref in zip(("dq", "dk", "dv"), grads, refs):
        check_close(host_f64(got), ref, dtype, name)


def test_bwd_full_size_sampled():
    """The 16-tile 5x9x9 backward at full size; sampled rows of dq, dk, dv vs oracle."""
    wl = I.TRAIN_TILE_BWD
    shape = wl.shape()
    window = (wl.kz, wl.ky, wl.kx)
    pl = wl.placement()
    c32 = oracle_coords(pl, wl.H, wl.W)
    (q, k, v, g), (dq, dk, dv), scale = run_bwd(shape, window, "bf16", wl.seed, c32)
    tiles = [0, shape[0] - 1]
    per_tile = shape[1] * wl.N
    sel = sample_queries(shape, 160, wl.seed, tiles)
    local = np.searchsorted(tiles, sel // per_tile) * per_tile + sel % per_tile
    sub = lambda a: oracle.widen(a[tiles], "bf16")
    rq, rk, rv = oracle.na3d_bwd(sub(q), sub(k), sub(v), sub(g), window, scale, coords=c32[tiles],
                                 selq=local, selk=local)
    for name, got, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        check_close(host_rows(got, sel, wl.d), ref, "bf16", name)


@pytest.mark.parametrize("window", [(3, 7, 7), (5, 9, 9)])
@pytest.mark.parametrize("g_shift", [-40, 24])
def test_bwd_dout_magnitude(window, g_shift):
    """dS is carried in float16 with a running power-of-two scale: gradients of
    tiny and huge dO keep the bf16 bound (all grads are linear in dO)."""
    shape = (1, 2, 6, 21, 19, 64)
    pl = I.random_placement(shape[0], shape[3], shape[4], 93)
    c32 = oracle_coords(pl, shape[3], shape[4])
    g_exp = np.full(shape[:-1], g_shift, dtype=np.int32)
    (q, k, v, g), grads, scale = run_bwd(shape, window, "bf16", 43, c32, g_exp=g_exp)
    refs = oracle.na3d_bwd(*(oracle.widen(a, "bf16") for a in (q, k, v, g)), window, scale, coords=c32)
    for name, got, ref in zip(("dq", "dk", "dv"), grads, refs):
        check_close(host_f64(got), ref, "bf16", name)


@pytest.mark.parametrize("window", [(5, 9, 9), (9, 9, 9)])
def test_bwd_dout_scale_per_head(window):
    """The balanced dK/dV kernel scales its float16 copy of dO by a power of two
    per (batch, head): a head whose dO is all zero, one at 2^-30 and one at 2^20
    each keep the bf16 bound against their own RMS (and the zero head gives
    exact zeros)."""
    shape = (1, 3, 9, 21, 23, 64)  # planes the balanced kernel takes
    pl = I.random_placement(shape[0], shape[3], shape[4], 95)
    c32 = oracle_coords(pl, shape[3], shape[4])
    g_exp = np.zeros(shape[:-1], dtype=np.int32)
    g_exp[:, 0], g_exp[:, 1], g_exp[:, 2] = -200, -30, 20  # 2^-200 flushes to zero
    (q, k, v, g), grads, scale = run_bwd(shape, window, "bf16", 45, c32, g_exp=g_exp)
    assert not np.any(I.bf16_bits_to_f32(g)[:, 0])
    refs = oracle.na3d_bwd(*(oracle.widen(a, "bf16") for a in (q, k, v, g)), window, scale, coords=c32)
    for name, got, ref in zip(("dq", "dk", "dv"), grads, refs):
        got = host_f64(got)
        assert not np.any(got[:, 0]), f"{name}: head with zero dO"
        for h in (1, 2):
            check_close(got[:, h], ref[:, h], "bf16", f"{name} head {h}")


def test_bwd_workspace_holds_d_and_dout_exponents():
    """What the MFMA dQ pass leaves in the workspace for the dK/dV pass: D =
    rowsum(dO * O) of every token-head (from the forward's bf16 O), then one
    word per (batch, head) holding the frexp exponent of its largest |dO|
    (-1000 where all of its dO is zero)."""
    shape = (2, 3, 5, 12, 12, 64)
    window = (5, 9, 9)
    (q, k, v), out, lse, scale = run_fwd(shape, window, "bf16", 46)
    g_exp = np.zeros(shape[:-1], dtype=np.int32)
    g_exp[0, 1], g_exp[1, 0], g_exp[1, 2] = -200, -37, 29  # one all-zero head
    g = I.gaussian(shape, 46, I.STREAM_DO, "bf16")
    g = I.f32_to_bf16_bits((I.bf16_bits_to_f32(g) * np.exp2(g_exp.astype(np.float32))[..., None]).astype(np.float32))
    qd, kd, vd, gd = (dev_tensor(a, "bf16") for a in (q, k, v, g))
    desc = B.desc_for(qd, window, scale)
    ws = torch.zeros(B.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device="cuda")
    dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
    B.strata_na3d_bwd(desc, qd, kd, vd, None, out, gd, lse, dq, dk, dv, ws)
    torch.cuda.synchronize()
    n = int(np.prod(shape[:-1]))
    off = (4 * n + 255) // 256 * 256
    w = ws.cpu().numpy()
    d_got = w[:4 * n].view(np.float32).reshape(shape[:-1])
    gf = I.bf16_bits_to_f32(g).astype(np.float64)
    o64 = host_f64(out)
    d_ref = np.sum(gf * o64, axis=-1)
    d_abs = np.sum(np.abs(gf * o64), axis=-1)  # float32 sums of exact products: error <= ~64 ulp of this
    assert np.all(np.abs(d_got - d_ref) <= 2.0 ** -17 * d_abs)
    e_got = w[off:off + 4 * shape[0] * shape[1]].view(np.int32).reshape(shape[:2])
    amax = np.abs(gf).reshape(shape[0], shape[1], -1).max(axis=-1)
    e_ref = np.where(amax > 0, np.frexp(amax)[1], -1000)
    assert np.array_equal(e_got, e_ref), (e_got, e_ref)


@pytest.mark.parametrize("window", [(3, 7, 7), (5, 9, 9)])
def test_bwd_dout_mixed_magnitudes_dq_per_class(window):
    """dO rows scaled by 2^e, e in {-24, -12, 0, 12}: dq of every magnitude class
    meets the bf16 bound relative to that class's own RMS (the dS scale of the
    dq pass is per query)."""
    shape = (1, 2, 6, 21, 19, 64)
    pl = I.random_placement(shape[0], shape[3], shape[4], 94)
    c32 = oracle_coords(pl, shape[3], shape[4])
    cls = I.rng(44, 9).integers(0, 4, size=shape[:-1])
    g_exp = (12 * cls - 24).astype(np.int32)
    (q, k, v, g), (dq, dk, dv), scale = run_bwd(shape, window, "bf16", 44, c32, g_exp=g_exp)
    rq, rk, rv = oracle.na3d_bwd(*(oracle.widen(a, "bf16") for a in (q, k, v, g)), window, scale, coords=c32)
    got = host_f64(dq)
    for c in range(4):
        m = cls == c
        check_close(got[m], rq[m], "bf16", f"dq class 2^{12 * c - 24}")
    check_close(host_f64(dk), rk, "bf16", "dk")
    # dV = sum_q P dO_q with P rounded to bf16 (as in any bf16 P.dO product): with
    # heavy-tailed dO that rounding alone reaches ~2.7% of RMS(dV), so dv also gets
    # its elementwise bound 2^-8 sum_q P |dO_q| (twice bf16's unit roundoff).
    absg = np.abs(oracle.widen(g, "bf16"))
    _, _, a_dv = oracle.na3d_bwd(*(oracle.widen(a, "bf16") for a in (q, k, v)), absg, window, scale,
                                 coords=c32)
    got_v = host_f64(dv)
    excess = np.abs(got_v - rv) - bf16_half_ulp(rv) - np.ldexp(a_dv, -8)
    rms = float(np.sqrt(np.mean(rv * rv)))
    assert float(np.max(excess)) <= 2e-2 * rms, f"dv: {float(np.max(excess)):.3e} > {2e-2 * rms:.3e}"


# ----------------------------------------------------------------------------- input range

def test_fwd_level_sweep_large_keys_stay_finite():
    """Keys of magnitude 61440 (inside float16's range, beyond 65504 / sqrt(2)) through the
    level-sweep kernel (3x7x7, Z = 8): a rotated pair would exceed 65504 at phases near 45
    degrees, so the kernel rotates at half length.  One such key per 8x8 patch of
    positions on one level, so every query window holds at most one.  Every output
    and LSE must be finite.  The float16 copy of such a key carries an absolute
    error of ~2^-11 * 61440 per element, so its logit is only known to within tens
    of units: the oracle is matched (bf16 rule, LSE within 2^-9 relative) where the
    exact logit of the large key is decisive, |s| > 200 (one-hot on it, or no weight),
    and on every query whose window holds no large key."""
    shape, window, scale = (1, 2, 8, 24, 24, 64), (3, 7, 7), 0.125
    q = I.gaussian(shape, 95, 0, "bf16")
    v = I.gaussian(shape, 95, 2, "bf16")
    kf = I.bf16_bits_to_f32(I.gaussian(shape, 95, 1, "bf16"))
    signs = np.where(np.random.default_rng(95).random(shape) < 0.5, -1.0, 1.0).astype(np.float32)
    big = np.zeros(shape[:-1] + (1,), bool)
    big[:, :, 3, 2::8, 3::8] = True
    kf = np.where(big, np.float32(61440.0) * signs, kf).astype(np.float32)
    k = I.f32_to_bf16_bits(kf)
    pl = I.random_placement(1, 24, 24, 95)
    c32 = oracle_coords(pl, 24, 24)
    qd, kd, vd = (dev_tensor(a, "bf16") for a in (q, k, v))
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(B.desc_for(qd, window, scale), qd, kd, vd, gpu_phases(c32, 64), out, lse)
    torch.cuda.synchronize()
    got, gl = host_f64(out), host_f64(lse)
    assert np.all(np.isfinite(got)) and np.all(np.isfinite(gl))
    q64, k64 = (oracle.widen(a, "bf16") for a in (q, k))
    ro, rl = oracle.na3d_fwd(q64, k64, oracle.widen(v, "bf16"), window, scale, coords=c32)
    # exact logit of the large key in each query's window (0 where there is none)
    qr, kr = (oracle.rope_apply(a, c32, base=ROPE_BASE) for a in (q64, k64))
    s_big = np.zeros(shape[:-1])
    s_abs = np.zeros(shape[:-1])  # scale sum |q_i k_i| of the large key: bounds its logit's rounding
    has = np.zeros(shape[:-1], bool)
    for h in range(shape[1]):
        for z in range(8):
            if not (win_lo(z, 8, 3) <= 3 < win_lo(z, 8, 3) + 3):
                continue
            for y in range(24):
                for x in range(24):
                    ys, xs = win_lo(y, 24, 7), win_lo(x, 24, 7)
                    for ky in range(ys, ys + 7):
                        for kx in range(xs, xs + 7):
                            if big[0, h, 3, ky, kx, 0]:
                                has[0, h, z, y, x] = True
                                s_big[0, h, z, y, x] = scale * float(qr[0, h, z, y, x] @ kr[0, h, 3, ky, kx])
                                s_abs[0, h, z, y, x] = scale * float(np.abs(qr[0, h, z, y, x]) @
                                                                     np.abs(kr[0, h, 3, ky, kx]))
    decisive = ~has | (np.abs(s_big) > 200)
    assert np.count_nonzero(has & (s_big > 200)) > 20 and np.count_nonzero(has & (s_big < -200)) > 20
    check_close(got[decisive], ro[decisive], "bf16", "out (large keys, decisive logits)")
    # LSE: the bf16-input rule, plus the float16 rounding of the two operands of the
    # large key's logit (2^-11 relative each) where that logit dominates
    lse_bound = LSE_ABS_BF16 + np.where(has & (s_big > 200), 2.0 ** -9 * s_abs, 0.0)
    assert np.all((np.abs(gl - rl) <= lse_bound)[decisive])


def win_lo(i, L, k):
    """First position of the border-clamped window of position i (the NATTEN rule)."""
    return min(max(i - k // 2, 0), L - k)


def test_stereo_coords_library_length():
    """l_scale == 0 makes the library use Eq. 1's sqrt(4 pi / N_total) for the six faces:
    the same coordinates, bit for bit, as passing that length explicitly."""
    wl = I.SMALL_BF16
    pl = wl.placement()
    f, oy, ox = (torch.from_numpy(a).cuda() for a in pl.as_int32())
    a = torch.empty((wl.B, wl.H, wl.W, 2), dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    B.strata_stereo_coords(f, oy, ox, wl.H, wl.W, 2048, 4, 0.0, a)
    B.strata_stereo_coords(f, oy, ox, wl.H, wl.W, 2048, 4, G.l_scale(2048), b)
    torch.cuda.synchronize()
    assert torch.equal(a, b)

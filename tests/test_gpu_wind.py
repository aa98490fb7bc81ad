"""GPU parity of the wind rotation into the tile-centre frame (Sec. 3.3, Eq. 2)
against the CPU oracle, through the C ABI.  float32: max abs error <= 1e-5;
bf16: within half a bf16 ulp of the exact value plus the float32 arithmetic
bound 2^-20 (|U| + |V|).  Tiles centred exactly on a pole are left out: the
East-North frame is undefined there and the computed longitude depends on the
last bit of the centre."""
import numpy as np
import pytest
import torch

from oracle import geometry as G
from paper_2606_31248_amd import binding as B
from paper_2606_31248_amd import inputs as I
from _util import bf16_half_ulp, dev_tensor, host_f64

pytestmark = pytest.mark.gpu


def check_wind(got, ref, uv, dtype):
    diff = np.abs(got - ref)
    if dtype == "f32":
        assert float(np.max(diff)) <= 1e-5
    else:
        mag = np.abs(uv[..., 0:1]) + np.abs(uv[..., 1:2])
        excess = diff - bf16_half_ulp(ref) - 2.0 ** -20 * mag
        assert float(np.max(excess)) <= 0.0, float(np.max(excess))


def run(field_shape, face, nty, ntx, Ht, Wt, sy, sx, dtype, seed):
    P, n = field_shape[0], field_shape[1]
    f = I.gaussian(field_shape, seed, 0, dtype, 10.0)
    fd = dev_tensor(f, dtype)
    tiles = torch.empty((nty * ntx, P, Ht, Wt, 2), dtype=fd.dtype, device="cuda")
    B.strata_wind_tile_frame(fd, face, nty, ntx, sy, sx, tiles)
    torch.cuda.synchronize()
    fw = I.bf16_bits_to_f32(f).astype(np.float64) if dtype == "bf16" else f.astype(np.float64)
    ref = G.wind_tiles(fw, face, n, nty, ntx, Ht, Wt, sy, sx)
    return host_f64(tiles), ref, fw


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("face", [0, 2, 4, 5])
def test_wind_tiles_match_oracle(dtype, face):
    # 2 x 3 tiles of 16 x 12 cells on a 64-cell face (no tile centred on a pole)
    got, ref, fw = run((3, 64, 64, 2), face, 2, 3, 16, 12, 40, 20, dtype, 90 + face)
    # the (U, V) the oracle saw at every output cell, for the bf16 bound
    uv = np.stack([fw[:, a * 40:a * 40 + 16, b * 20:b * 20 + 12] for a in range(2) for b in range(3)])
    check_wind(got, ref, uv, dtype)


def test_wind_face_rollout_tiling_sampled():
    """The face-rollout tiling in cells (9 x 9 tiles of 256 x 256 cells, stride
    224, on a 2048-cell face), 8 levels, bf16; three tiles checked in full."""
    n, P = 2048, 8
    f = I.gaussian((P, n, n, 2), 91, 0, "bf16", 10.0)
    fd = dev_tensor(f, "bf16")
    tiles = torch.empty((81, P, 256, 256, 2), dtype=fd.dtype, device="cuda")
    B.strata_wind_tile_frame(fd, 0, 9, 9, 224, 224, tiles)
    torch.cuda.synchronize()
    got = host_f64(tiles)
    fw = I.bf16_bits_to_f32(f).astype(np.float64)
    for t in (0, 40, 80):
        a, b = divmod(t, 9)
        sub = fw[:, a * 224:a * 224 + 256, b * 224:b * 224 + 256]
        # the oracle's steps for this tile: its cells' (lat, lon), its centre, Eq. 2
        rows, cols = a * 224 + np.arange(256), b * 224 + np.arange(256)
        beta, alpha = G.cell_angle(rows, n), G.cell_angle(cols, n)
        lat0, lon0 = G.latlon(0, 0.5 * (alpha[0] + alpha[-1]), 0.5 * (beta[0] + beta[-1]))
        A, Bt = np.meshgrid(alpha, beta, indexing="xy")
        lat, lon = G.latlon(np.zeros(A.shape, np.int64), A, Bt)
        u, v = G.wind_to_tile_frame(sub[..., 0], sub[..., 1], lat, lon, lat0, lon0)
        check_wind(got[t], np.stack([u, v], -1), sub, "bf16")


# ----------------------------------------------------------------------------- KBD window

@pytest.mark.parametrize("Ht,Wt,overlap,beta", [(64, 64, 8, 4 * np.pi), (64, 40, 8, 2.0), (16, 16, 8, 10.0),
                                                (256, 256, 32, 4 * np.pi), (5, 7, 3, 0.0)])
def test_kbd_window_matches_oracle(Ht, Wt, overlap, beta):
    w = torch.empty(Ht * Wt, dtype=torch.float32, device="cuda")
    B.strata_kbd_window(Ht, Wt, overlap, beta, w)
    torch.cuda.synchronize()
    ref = G.kbd_window_2d(Ht, Wt, overlap, beta)
    assert float(np.max(np.abs(w.cpu().numpy().astype(np.float64) - ref))) <= 1e-7


def test_kbd_window_blends_a_constant_field_exactly():
    """Any positive window reproduces a constant field through the stitch (D^-1 P^T W)."""
    w = torch.empty(64 * 64, dtype=torch.float32, device="cuda")
    B.strata_kbd_window(64, 64, 8, 4 * np.pi, w)
    tiles = torch.full((9, 2, 64, 64, 4), 0.75, dtype=torch.float32, device="cuda")
    face = torch.empty((2, 176, 176, 4), dtype=torch.float32, device="cuda")
    B.strata_tile_blend(tiles, 3, 3, 56, 56, w, face)
    torch.cuda.synchronize()
    assert torch.all(face == 0.75)


# ----------------------------------------------------------------------------- Duo-grid padding

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,halo,P,C", [(16, 4, 2, 3), (32, 8, 1, 8), (20, 3, 1, 2), (17, 3, 1, 1)])
def test_duo_pad_matches_oracle(dtype, n, halo, P, C):
    f = I.gaussian((6, P, n, n, C), 95 + n, 0, dtype)
    fd = dev_tensor(f, dtype)
    m = n + 2 * halo
    out = torch.empty((6, P, m, m, C), dtype=fd.dtype, device="cuda")
    B.strata_duo_pad(fd, halo, out)
    torch.cuda.synchronize()
    got = host_f64(out)
    fw = I.bf16_bits_to_f32(f).astype(np.float64) if dtype == "bf16" else f.astype(np.float64)
    ref = G.duo_pad(fw, halo)
    # interior: an exact copy
    assert np.array_equal(got[:, :, halo:halo + n, halo:halo + n], fw)
    diff = np.abs(got - ref)
    if dtype == "f32":
        assert float(np.max(diff)) <= 1e-5
    else:  # one rounding of a float32 sum of 4 weighted values
        bound = bf16_half_ulp(ref) + 2.0 ** -20 * 4 * float(np.max(np.abs(fw)))
        assert float(np.max(diff - bound)) <= 0.0


@pytest.mark.parametrize("dtype", ["bf16"])
def test_duo_pad_full_size_sampled(dtype):
    # six 2048-cell faces, 8 levels x 4 channels, halo 16 (the measured
    # workload): interior exact, sampled halo cells (corner diagonals among
    # them) against the oracle's brute-force neighbours over the whole face
    # (about 5 s of CPU per cell)
    n, h, P, C = 2048, 16, 8, 4
    m = n + 2 * h
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1011)
    fd = torch.randn((6, P, n, n, C), generator=gen, device="cuda").to(torch.bfloat16)
    out = torch.empty((6, P, m, m, C), dtype=torch.bfloat16, device="cuda")
    B.strata_duo_pad(fd, h, out)
    torch.cuda.synchronize()
    assert torch.equal(out[:, :, h:h + n, h:h + n], fd)
    rng = np.random.default_rng(7)
    cells = [(0, 0, 0), (1, m - 1, m - 1), (2, h - 1, n + h), (5, m // 3, m - 1)]
    for _ in range(2):
        f = int(rng.integers(6))
        side = int(rng.integers(4))
        t = int(rng.integers(m))
        band = int(rng.integers(h))
        ip, jp = [(band, t), (m - 1 - band, t), (t, band), (t, m - 1 - band)][side]
        cells.append((f, ip, jp))
    for f, ip, jp in cells:
        fp, rows, cols, w = G.duo_halo_neighbours(f, ip - h, jp - h, n)
        vals = fd[fp][:, torch.as_tensor(rows, device="cuda"), torch.as_tensor(cols, device="cuda")]
        vals = vals.float().cpu().numpy().astype(np.float64)  # [P, 4, C]
        ref = np.zeros((P, C))
        for k in range(4):
            ref = ref + w[k] * vals[:, k]
        got = out[f, :, ip, jp].float().cpu().numpy().astype(np.float64)
        bound = bf16_half_ulp(ref) + 2.0 ** -20 * 4 * float(np.max(np.abs(vals)))
        assert float(np.max(np.abs(got - ref) - bound)) <= 0.0, (f, ip, jp)


def _halo_cells(n, halo):
    """Halo cells (ip, jp) of a padded face in plan order: top band, bottom band,
    then the left/right strips row by row."""
    m = n + 2 * halo
    top = [(ip, jp) for ip in range(halo) for jp in range(m)]
    bottom = [(ip, jp) for ip in range(n + halo, m) for jp in range(m)]
    strips = [(ip, jp) for ip in range(halo, n + halo) for jp in list(range(halo)) + list(range(n + halo, m))]
    return top + bottom + strips


@pytest.mark.parametrize("n,halo", [(16, 4), (20, 3), (17, 3)])
def test_duo_plan_entries_match_oracle(n, halo):
    # the plan's leading section, one 64-byte entry per halo cell (float64
    # weights[4], int32 cells[4], int32 face):
    # face and cells exact, weights to float64 rounding
    nb = B.strata_duo_plan_bytes(n, halo)
    plan = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.strata_duo_plan(n, halo, plan)
    torch.cuda.synchronize()
    raw = plan.cpu().numpy()
    ent = np.dtype([("w", "<f8", 4), ("cell", "<i4", 4), ("face", "<i4"), ("unused", "<i4", 3)])
    cells = _halo_cells(n, halo)
    e = raw[:6 * len(cells) * 64].view(ent)  # P's entries lead the plan
    for f in range(6):
        for h, (ip, jp) in enumerate(cells):
            fp, rows, cols, w = G.duo_halo_neighbours(f, ip - halo, jp - halo, n)
            x = e[f * len(cells) + h]
            assert int(x["face"]) == fp, (f, ip, jp)
            assert np.array_equal(x["cell"], rows * n + cols), (f, ip, jp)
            np.testing.assert_allclose(x["w"], w, rtol=0, atol=1e-13)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,halo,P,C", [(16, 4, 2, 3), (32, 8, 1, 8), (17, 3, 3, 1), (20, 3, 2, 2)])
def test_duo_planned_equals_one_shot(dtype, n, halo, P, C):
    # the plan gives the same weights and summation order: identical bits; one
    # plan serves fields of any level and channel count
    nb = B.strata_duo_plan_bytes(n, halo)
    plan = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.strata_duo_plan(n, halo, plan)
    m = n + 2 * halo
    for PP, CC in ((P, C), (1, 2 * C)):
        f = I.gaussian((6, PP, n, n, CC), 131 + n + CC, 0, dtype)
        fd = dev_tensor(f, dtype)
        a = torch.empty((6, PP, m, m, CC), dtype=fd.dtype, device="cuda")
        b = torch.full_like(a, float("nan"))
        B.strata_duo_pad(fd, halo, a)
        B.strata_duo_pad_planned(fd, halo, plan, b)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int16) if dtype == "bf16" else a.view(torch.int32),
                           b.view(torch.int16) if dtype == "bf16" else b.view(torch.int32))


def test_duo_planned_full_size_equals_one_shot():
    n, h, P, C = 2048, 16, 8, 4
    m = n + 2 * h
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1011)
    fd = torch.randn((6, P, n, n, C), generator=gen, device="cuda").to(torch.bfloat16)
    plan = torch.empty(B.strata_duo_plan_bytes(n, h), dtype=torch.uint8, device="cuda")
    B.strata_duo_plan(n, h, plan)
    a = torch.empty((6, P, m, m, C), dtype=torch.bfloat16, device="cuda")
    b = torch.empty_like(a)
    B.strata_duo_pad(fd, h, a)
    B.strata_duo_pad_planned(fd, h, plan, b)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def _vjp_tolerance(ref, abs_sum, dtype):
    if dtype == "f32":  # float64 sums rounded once; weights agree with the oracle's to ~1e-13
        return np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64) + 1e-12 * abs_sum
    # float32 fused multiply-adds over a handful of terms, one bf16 rounding
    return bf16_half_ulp(ref) + 2.0 ** -18 * abs_sum


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,halo,P,C", [(16, 4, 2, 3), (20, 3, 1, 2), (17, 3, 1, 1), (32, 8, 1, 8)])
def test_duo_pad_vjp_matches_oracle(dtype, n, halo, P, C):
    m = n + 2 * halo
    g = I.gaussian((6, P, m, m, C), 171 + n, 0, dtype)
    gd = dev_tensor(g, dtype)
    plan = torch.empty(B.strata_duo_plan_bytes(n, halo), dtype=torch.uint8, device="cuda")
    B.strata_duo_plan(n, halo, plan)
    out = torch.full((6, P, n, n, C), float("nan"), dtype=gd.dtype, device="cuda")
    B.strata_duo_pad_vjp(gd, halo, plan, out)
    torch.cuda.synchronize()
    got = host_f64(out)
    gw = I.bf16_bits_to_f32(g).astype(np.float64) if dtype == "bf16" else g.astype(np.float64)
    ref = G.duo_pad_vjp(gw, halo)
    abs_sum = G.duo_pad_vjp(np.abs(gw), halo)
    assert float(np.max(np.abs(got - ref) - _vjp_tolerance(ref, abs_sum, dtype))) <= 0.0
    # deterministic: a second plan and a second pass give the same bits
    plan2 = torch.empty_like(plan)
    B.strata_duo_plan(n, halo, plan2)
    out2 = torch.empty_like(out)
    B.strata_duo_pad_vjp(gd, halo, plan2, out2)
    torch.cuda.synchronize()
    assert torch.equal(plan, plan2)
    bits = torch.int16 if dtype == "bf16" else torch.int32
    assert torch.equal(out.view(bits), out2.view(bits))


def test_duo_pad_vjp_full_size_adjoint_and_interior():
    # six 2048-cell faces, halo 16, float32: <P x, y> = <x, P^T y>; the total
    # of P^T 1 counts every padded cell once; cells deeper than the halo get
    # their interior gradient bit for bit
    n, h, P, C = 2048, 16, 2, 4
    m = n + 2 * h
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2024)
    x = torch.randn((6, P, n, n, C), generator=gen, device="cuda")
    y = torch.randn((6, P, m, m, C), generator=gen, device="cuda")
    plan = torch.empty(B.strata_duo_plan_bytes(n, h), dtype=torch.uint8, device="cuda")
    B.strata_duo_plan(n, h, plan)
    px = torch.empty_like(y)
    B.strata_duo_pad_planned(x, h, plan, px)
    pty = torch.empty_like(x)
    B.strata_duo_pad_vjp(y, h, plan, pty)
    lhs = float((px.double() * y.double()).sum())
    rhs = float((x.double() * pty.double()).sum())
    scale = float((px.double() * y.double()).abs().sum())
    assert abs(lhs - rhs) <= 1e-6 * scale, (lhs, rhs, scale)
    d = h + 2
    assert torch.equal(pty[:, :, d:n - d, d:n - d], y[:, :, h + d:h + n - d, h + d:h + n - d])
    del x, px
    ones = torch.ones_like(y)
    B.strata_duo_pad_vjp(ones, h, plan, pty)
    total = float(pty.double().sum())
    assert abs(total - 6 * P * C * m * m) <= 1e-6 * 6 * P * C * m * m

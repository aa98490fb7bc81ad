"""GPU parity at the paper's own shapes (App. B.1) against the CPU oracle: the
9x9x9 window at 24 levels, column-wise attention (window (kz, 1, 1), the full
column included, even Z too), head_dim 128; forward and backward, with and
without the attention-block options.  Same rules as the other GPU tests."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_31248_amd import binding as B
from paper_2606_31248_amd import inputs as I
from paper_2606_31248_amd import pipeline
from _util import LSE_ABS_BF16, check_close, dev_tensor, host_f64, host_rows
from oracle import geometry as G
from test_gpu_options import check_bwd_grads, check_out

pytestmark = pytest.mark.gpu


def coords_for(shape, seed):
    pl = I.random_placement(shape[0], shape[3], shape[4], seed)
    return G.tile_coords(pl.face, pl.oy, pl.ox, shape[3], shape[4]).astype(np.float32)


def phases(c32, d):
    c = torch.from_numpy(c32).cuda()
    cs = torch.empty(c32.shape[:3] + (d // 2, 2), dtype=torch.float32, device="cuda")
    B.strata_stereorope_phases(c, d, pipeline.ROPE_BASE, cs)
    return cs


def gate_for(shape, kind, seed, dtype):
    if kind == 0:
        return None
    return I.gaussian(shape[:-1] if kind == 1 else shape, seed, I.STREAM_GATE, dtype, 2.0)


def run(shape, window, dtype, seed, rope=True, qk_norm=False, gkind=0, bwd=False):
    q, k, v = (I.gaussian(shape, seed, s, dtype) for s in (0, 1, 2))
    g = gate_for(shape, gkind, seed, dtype)
    c32 = coords_for(shape, seed + 7) if rope else None
    qd, kd, vd = (dev_tensor(a, dtype) for a in (q, k, v))
    gd = None if g is None else dev_tensor(g, dtype)
    cs = phases(c32, shape[-1]) if rope else None
    scale = 1.0 / np.sqrt(shape[-1])
    desc = B.desc_for(qd, window, scale)
    opts = B.make_opts(qk_norm, 1e-6, gd)
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd_ex(desc, opts, qd, kd, vd, cs, out, lse)
    res = {"inputs": (q, k, v, g), "c32": c32, "scale": scale, "out": out, "lse": lse}
    if bwd:
        dout = I.gaussian(shape, seed, I.STREAM_DO, dtype)
        dod = dev_tensor(dout, dtype)
        ws = torch.empty(B.strata_na3d_bwd_ex_workspace_size(desc, opts), dtype=torch.uint8, device="cuda")
        dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
        dg = None if gd is None else torch.empty_like(gd)
        B.strata_na3d_bwd_ex(desc, opts, qd, kd, vd, cs, out, dod, lse, dq, dk, dv, dg, ws)
        res["dout"] = dout
        res["grads"] = (dq, dk, dv, dg)
    torch.cuda.synchronize()
    return res


def check_fwd(r, window, dtype, qk_norm, sel=None):
    w = lambda a: None if a is None else oracle.widen(a, dtype)
    q, k, v, g = r["inputs"]
    ro, rl = oracle.na3d_fwd(w(q), w(k), w(v), window, r["scale"], coords=r["c32"], qk_norm=qk_norm, gate=w(g),
                             sel=sel)
    d = q.shape[-1]
    got = host_f64(r["out"]) if sel is None else host_f64(r["out"]).reshape(-1, d)[sel]
    gl = host_f64(r["lse"]) if sel is None else host_f64(r["lse"]).reshape(-1)[sel]
    if g is None:
        check_close(got, ro, dtype, "out")
    else:
        check_out(got, r["inputs"], window, r["scale"], dtype, qk_norm, r["c32"], ro, sel=sel)
    tol = LSE_ABS_BF16 if dtype == "bf16" else 1e-5
    assert float(np.max(np.abs(gl - rl))) <= tol


def sample_keys(shape, n, seed):
    """Random flat token indices plus the corners of every tile and head."""
    Bt, h, Z, H, W, _ = shape
    r = np.random.default_rng(seed)
    flat = r.integers(0, Bt * h * Z * H * W, n)
    corners = [((((b * h + hh) * Z + z) * H + y) * W + x) for b in range(Bt) for hh in range(h)
               for z in (0, Z - 1) for y in (0, H - 1) for x in (0, W - 1)]
    return np.unique(np.concatenate([flat, np.array(corners)]))


# ----------------------------------------------------------------------------- 9x9x9 at 24 levels

@pytest.mark.parametrize("shape,rope", [((1, 2, 12, 16, 16, 64), True), ((2, 1, 24, 16, 16, 64), True),
                                        ((1, 1, 10, 21, 19, 64), False), ((1, 1, 9, 9, 9, 64), True)])
def test_w999_fwd_full_oracle(shape, rope):
    r = run(shape, (9, 9, 9), "bf16", 71, rope=rope)
    check_fwd(r, (9, 9, 9), "bf16", False)


@pytest.mark.parametrize("qk_norm,gkind", [(True, "d"), (True, 1), (False, "d")])
def test_w999_fwd_options(qk_norm, gkind):
    shape = (1, 2, 12, 16, 16, 64)
    r = run(shape, (9, 9, 9), "bf16", 72, qk_norm=qk_norm, gkind=gkind)
    check_fwd(r, (9, 9, 9), "bf16", qk_norm)


@pytest.mark.parametrize("shape,qk_norm,gkind", [((1, 2, 12, 16, 16, 64), False, 0),
                                                 ((1, 1, 24, 16, 16, 64), False, 0),
                                                 ((1, 1, 11, 13, 17, 64), False, 0),
                                                 ((1, 2, 12, 16, 16, 64), True, "d")])
def test_w999_bwd_sampled_keys(shape, qk_norm, gkind):
    """dq of every query; dk, dv (and dgate) of sampled keys and queries (the
    oracle's key-side gradient costs O(K^2 d) per key)."""
    window = (9, 9, 9)
    r = run(shape, window, "bf16", 73, qk_norm=qk_norm, gkind=gkind, bwd=True)
    q, k, v, g = r["inputs"]
    sel = sample_keys(shape, 48, 74)
    w = lambda a: None if a is None else oracle.widen(a, "bf16")
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"], selq=sel,
                           selk=sel, qk_norm=qk_norm, gate=w(g))
    got = [None if x is None else host_f64(x) for x in r["grads"]]
    got = [None if x is None else (x.reshape(-1)[sel] if x.ndim == 5 else x.reshape(-1, x.shape[-1])[sel])
           for x in got]
    check_bwd_grads((q, k, v, g, r["dout"]), [None if x is None else torch.from_numpy(x) for x in got], refs,
                    window, r["scale"], "bf16", qk_norm, r["c32"], sel=sel, presliced=True)
    # dq of every query against the oracle (cheap side)
    rq = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"],
                         selk=np.array([0]), qk_norm=qk_norm, gate=w(g))[0]
    check_close(host_f64(r["grads"][0]), rq, "bf16", "dq (all)")


def test_w999_fwd_full_size_sampled():
    """The paper tile (96 tiles x 16 heads x 24 x 16 x 16, 9x9x9) in one launch."""
    wl = I.PAPER_TILE16
    shape = wl.shape()
    tiles = [0, wl.B // 2, wl.B - 1]
    q, k, v = (I.gaussian(shape, wl.seed, s, "bf16") for s in (0, 1, 2))
    pl = wl.placement()
    c32 = G.tile_coords(pl.face, pl.oy, pl.ox, wl.H, wl.W).astype(np.float32)
    qd, kd, vd = (dev_tensor(a, "bf16") for a in (q, k, v))
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(B.desc_for(qd, (9, 9, 9), wl.scale), qd, kd, vd, phases(c32, wl.d), out, lse)
    torch.cuda.synchronize()
    per_tile = wl.heads * wl.N
    r = np.random.default_rng(wl.seed)
    sel = np.unique(np.concatenate([r.integers(0, per_tile, 800) + t * per_tile for t in tiles]))
    local = np.searchsorted(tiles, sel // per_tile) * per_tile + sel % per_tile
    sub = lambda a: oracle.widen(a[tiles], "bf16")
    ro, rl = oracle.na3d_fwd(sub(q), sub(k), sub(v), (9, 9, 9), wl.scale, coords=c32[tiles], sel=local)
    check_close(host_rows(out, sel, wl.d), ro, "bf16", "out")
    assert np.max(np.abs(host_rows(lse, sel) - rl)) <= LSE_ABS_BF16


# ----------------------------------------------------------------------------- column-wise attention

COL_CASES = [((2, 3, 24, 8, 9, 64), (24, 1, 1)),   # the full column, even Z
             ((1, 2, 24, 5, 7, 64), (7, 1, 1)),    # a border-clamped partial column window
             ((1, 2, 8, 6, 6, 64), (8, 1, 1)),     # Z <= 16: one block of levels
             ((1, 1, 13, 4, 4, 64), (5, 1, 1)),
             ((1, 1, 32, 3, 5, 64), (31, 1, 1))]


@pytest.mark.parametrize("shape,window", COL_CASES)
@pytest.mark.parametrize("rope", [True, False])
def test_column_fwd_full_oracle(shape, window, rope):
    """With StereoRoPE on, the oracle rotates q and k; the kernel relies on the
    rotation cancelling inside a column and must still match."""
    r = run(shape, window, "bf16", 75, rope=rope)
    check_fwd(r, window, "bf16", False)


@pytest.mark.parametrize("qk_norm,gkind", [(True, 0), (False, 1), (True, "d")])
@pytest.mark.parametrize("shape,window", [COL_CASES[0], COL_CASES[2]])
def test_column_fwd_options(shape, window, qk_norm, gkind):
    r = run(shape, window, "bf16", 76, qk_norm=qk_norm, gkind=gkind)
    check_fwd(r, window, "bf16", qk_norm)


@pytest.mark.parametrize("shape,window,dtype", [((1, 2, 24, 4, 5, 64), (24, 1, 1), "bf16"),
                                                ((1, 1, 8, 3, 4, 32), (8, 1, 1), "f32"),
                                                ((1, 2, 13, 3, 3, 64), (5, 1, 1), "bf16")])
@pytest.mark.parametrize("qk_norm,gkind", [(False, 0), (True, "d")])
def test_column_bwd_full_oracle(shape, window, dtype, qk_norm, gkind):
    r = run(shape, window, dtype, 77, qk_norm=qk_norm, gkind=gkind, bwd=True)
    q, k, v, g = r["inputs"]
    w = lambda a: None if a is None else oracle.widen(a, dtype)
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"], qk_norm=qk_norm,
                           gate=w(g))
    check_bwd_grads((q, k, v, g, r["dout"]), r["grads"], refs, window, r["scale"], dtype, qk_norm, r["c32"])


def test_column_fwd_full_size_sampled():
    """Column-wise attention over all 24 levels of the paper tile, one launch."""
    wl = I.PAPER_COLUMN
    shape = wl.shape()
    q, k, v = (I.gaussian(shape, wl.seed, s, "bf16") for s in (0, 1, 2))
    qd, kd, vd = (dev_tensor(a, "bf16") for a in (q, k, v))
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(B.desc_for(qd, (24, 1, 1), wl.scale), qd, kd, vd, None, out, lse)
    torch.cuda.synchronize()
    tiles = [0, wl.B - 1]
    per_tile = wl.heads * wl.N
    r = np.random.default_rng(wl.seed)
    sel = np.unique(np.concatenate([r.integers(0, per_tile, 2000) + t * per_tile for t in tiles]))
    local = np.searchsorted(tiles, sel // per_tile) * per_tile + sel % per_tile
    sub = lambda a: oracle.widen(a[tiles], "bf16")
    ro, rl = oracle.na3d_fwd(sub(q), sub(k), sub(v), (24, 1, 1), wl.scale, sel=local)
    check_close(host_rows(out, sel, wl.d), ro, "bf16", "out")
    assert np.max(np.abs(host_rows(lse, sel) - rl)) <= LSE_ABS_BF16


# ----------------------------------------------------------------------------- head_dim 128

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("qk_norm,gkind", [(False, 0), (True, "d")])
def test_d128_fwd_bwd_full_oracle(dtype, qk_norm, gkind):
    shape, window = (1, 1, 5, 9, 8, 128), (3, 5, 5)
    r = run(shape, window, dtype, 78, qk_norm=qk_norm, gkind=gkind, bwd=True)
    check_fwd(r, window, dtype, qk_norm)
    q, k, v, g = r["inputs"]
    w = lambda a: None if a is None else oracle.widen(a, dtype)
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"], qk_norm=qk_norm,
                           gate=w(g))
    check_bwd_grads((q, k, v, g, r["dout"]), r["grads"], refs, window, r["scale"], dtype, qk_norm, r["c32"])


@pytest.mark.parametrize("g_shift", [-40, 24])
def test_column_bwd_dout_magnitude(g_shift):
    """dS enters its float16 product with a per-column power-of-two scale: tiny
    and huge dO keep the bf16 bound (every gradient is linear in dO)."""
    shape, window = (1, 2, 24, 4, 5, 64), (24, 1, 1)
    q, k, v = (I.gaussian(shape, 79, s, "bf16") for s in (0, 1, 2))
    gf = I.bf16_bits_to_f32(I.gaussian(shape, 79, I.STREAM_DO, "bf16")) * np.float32(2.0 ** g_shift)
    dout = I.f32_to_bf16_bits(gf.astype(np.float32))
    qd, kd, vd, gd = (dev_tensor(a, "bf16") for a in (q, k, v, dout))
    scale = 0.125
    desc = B.desc_for(qd, window, scale)
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(desc, qd, kd, vd, None, out, lse)
    ws = torch.empty(B.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device="cuda")
    dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
    B.strata_na3d_bwd(desc, qd, kd, vd, None, out, gd, lse, dq, dk, dv, ws)
    torch.cuda.synchronize()
    w = lambda a: oracle.widen(a, "bf16")
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(dout), window, scale)
    for name, got, ref in zip(("dq", "dk", "dv"), (dq, dk, dv), refs):
        check_close(host_f64(got), ref, "bf16", name)


def test_column_bwd_full_size_sampled():
    """Column-wise backward over all 24 levels of the paper tile, one launch;
    sampled rows of dq, dk, dv vs the oracle on the sampled tiles."""
    wl = I.PAPER_COLUMN
    shape = wl.shape()
    q, k, v, dout = (I.gaussian(shape, wl.seed, s, "bf16") for s in (0, 1, 2, I.STREAM_DO))
    qd, kd, vd, gd = (dev_tensor(a, "bf16") for a in (q, k, v, dout))
    desc = B.desc_for(qd, (24, 1, 1), wl.scale)
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(desc, qd, kd, vd, None, out, lse)
    ws = torch.empty(B.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device="cuda")
    dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
    B.strata_na3d_bwd(desc, qd, kd, vd, None, out, gd, lse, dq, dk, dv, ws)
    torch.cuda.synchronize()
    tiles = [0, wl.B - 1]
    per_tile = wl.heads * wl.N
    r = np.random.default_rng(wl.seed)
    sel = np.unique(np.concatenate([r.integers(0, per_tile, 600) + t * per_tile for t in tiles]))
    local = np.searchsorted(tiles, sel // per_tile) * per_tile + sel % per_tile
    sub = lambda a: oracle.widen(a[tiles], "bf16")
    refs = oracle.na3d_bwd(sub(q), sub(k), sub(v), sub(dout), (24, 1, 1), wl.scale, selq=local, selk=local)
    for name, got, ref in zip(("dq", "dk", "dv"), (dq, dk, dv), refs):
        check_close(host_rows(got, sel, wl.d), ref, "bf16", name)


# ----------------------------------------------------------------------------- head_dim 128, 9x9x9 (MFMA kernel)

@pytest.mark.parametrize("shape,rope", [((1, 1, 12, 16, 16, 128), True), ((1, 2, 10, 21, 19, 128), False),
                                        ((2, 1, 9, 9, 9, 128), True)])
def test_d128_w999_fwd_full_oracle(shape, rope):
    """The head_dim-128 MFMA forward (single-buffered key levels): every output
    and LSE against the oracle, ragged blocks and an odd level count included."""
    r = run(shape, (9, 9, 9), "bf16", 81, rope=rope)
    check_fwd(r, (9, 9, 9), "bf16", False)


def test_d128_w999_fwd_decoder_full_size_sampled():
    """The decoder shape (2 tiles x 1 head x 24 x 64 x 64, head_dim 128) in one
    launch; sampled queries (tile corners included) against the oracle."""
    wl = I.PAPER_DECODER
    shape = wl.shape()
    sel = sample_keys(shape, 1500, 82)
    r = run(shape, (wl.kz, wl.ky, wl.kx), "bf16", wl.seed)
    check_fwd(r, (wl.kz, wl.ky, wl.kx), "bf16", False, sel=sel)


@pytest.mark.parametrize("shape,rope", [((1, 1, 12, 16, 16, 128), True), ((1, 1, 11, 13, 17, 128), False),
                                        ((2, 2, 10, 12, 12, 128), True)])
def test_d128_w999_bwd_sampled_keys(shape, rope):
    """The head_dim-128 MFMA backward: dq of every query, dk and dv of sampled
    keys (corners included) against the oracle."""
    window = (9, 9, 9)
    r = run(shape, window, "bf16", 83, rope=rope, bwd=True)
    q, k, v, _ = r["inputs"]
    sel = sample_keys(shape, 64, 84)
    w = lambda a: oracle.widen(a, "bf16")
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"], selk=sel)
    dq, dk, dv, _ = r["grads"]
    d = shape[-1]
    check_close(host_f64(dq), refs[0], "bf16", "dq")
    check_close(host_rows(dk, sel, d), refs[1], "bf16", "dk")
    check_close(host_rows(dv, sel, d), refs[2], "bf16", "dv")


def test_d128_w999_bwd_decoder_full_size_sampled():
    """The decoder shape's backward in one launch each; sampled queries and keys
    against the oracle on both tiles."""
    wl = I.PAPER_DECODER
    shape = wl.shape()
    window = (wl.kz, wl.ky, wl.kx)
    r = run(shape, window, "bf16", wl.seed, bwd=True)
    q, k, v, _ = r["inputs"]
    sel = sample_keys(shape, 160, 85)
    w = lambda a: oracle.widen(a, "bf16")
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"], selq=sel, selk=sel)
    dq, dk, dv, _ = r["grads"]
    for name, got, ref in zip(("dq", "dk", "dv"), (dq, dk, dv), refs):
        check_close(host_rows(got, sel, wl.d), ref, "bf16", name)


@pytest.mark.parametrize("qk_norm,gkind", [(True, 0), (False, 1), (False, "d"), (True, "d")])
def test_d128_w999_fwd_options_full_oracle(qk_norm, gkind):
    """QK RMSNorm and the output gate (App. B.5: every attention block has them,
    the decoder's included) in the head_dim-128 MFMA forward: full grid."""
    shape = (1, 1, 12, 16, 16, 128)
    r = run(shape, (9, 9, 9), "bf16", 86, qk_norm=qk_norm, gkind=gkind)
    check_fwd(r, (9, 9, 9), "bf16", qk_norm)


def test_d128_w999_fwd_options_decoder_full_size_sampled():
    wl = I.PAPER_DECODER
    shape = wl.shape()
    sel = sample_keys(shape, 1200, 87)
    r = run(shape, (wl.kz, wl.ky, wl.kx), "bf16", wl.seed, qk_norm=True, gkind="d")
    check_fwd(r, (wl.kz, wl.ky, wl.kx), "bf16", True, sel=sel)


@pytest.mark.parametrize("qk_norm,gkind", [(True, 0), (True, "d"), (False, 1), (False, "d")])
def test_d128_w999_bwd_options_sampled_keys(qk_norm, gkind):
    """The head_dim-128 backward with QK RMSNorm and the gate (dQ on the MFMA
    kernel with the two-term dA; dK, dV on it with the norm): dq of every
    query, dk, dv, dgate of sampled keys and queries against the oracle."""
    shape, window = (1, 1, 12, 16, 16, 128), (9, 9, 9)
    r = run(shape, window, "bf16", 88, qk_norm=qk_norm, gkind=gkind, bwd=True)
    q, k, v, g = r["inputs"]
    sel = sample_keys(shape, 40, 89)
    w = lambda a: None if a is None else oracle.widen(a, "bf16")
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"], selq=sel,
                           selk=sel, qk_norm=qk_norm, gate=w(g))
    got = [None if x is None else host_f64(x) for x in r["grads"]]
    got = [None if x is None else (x.reshape(-1)[sel] if x.ndim == 5 else x.reshape(-1, x.shape[-1])[sel])
           for x in got]
    check_bwd_grads((q, k, v, g, r["dout"]), [None if x is None else torch.from_numpy(x) for x in got], refs,
                    window, r["scale"], "bf16", qk_norm, r["c32"], sel=sel, presliced=True)
    rq = oracle.na3d_bwd(w(q), w(k), w(v), w(r["dout"]), window, r["scale"], coords=r["c32"],
                         selk=np.array([0]), qk_norm=qk_norm, gate=w(g))[0]
    check_close(host_f64(r["grads"][0]), rq, "bf16", "dq (all)")


@pytest.mark.parametrize("sign", [-1.0, 1.0])
def test_d128_w999_fwd_uniform_extreme_logits(sign):
    """Every logit equal and 200 (log2 units) from zero at head_dim 128: the lazy
    softmax reference must move (down on the first key level, or up) without
    overflow; the output is the window mean of V, the LSE logit + ln K."""
    shape = (1, 1, 10, 12, 12, 128)
    scale = 1.0 / np.sqrt(128.0)
    logit = sign * 200.0 / 1.4426950408889634
    alpha = logit / (128 * scale)
    q = I.f32_to_bf16_bits(np.full(shape, alpha, np.float32))
    k = I.f32_to_bf16_bits(np.ones(shape, np.float32))
    v = I.gaussian(shape, 90, 2, "bf16")
    qd, kd, vd = (dev_tensor(a, "bf16") for a in (q, k, v))
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    B.strata_na3d_fwd(B.desc_for(qd, (9, 9, 9), scale), qd, kd, vd, None, out, lse)
    torch.cuda.synchronize()
    ro, rl = oracle.na3d_fwd(*(oracle.widen(a, "bf16") for a in (q, k, v)), (9, 9, 9), scale)
    got = host_f64(out)
    assert np.isfinite(got).all()
    check_close(got, ro, "bf16", "out")
    assert np.max(np.abs(host_f64(lse) - rl)) <= LSE_ABS_BF16 + 2.0 ** -10 * float(np.max(np.abs(rl)))

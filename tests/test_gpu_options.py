"""GPU parity of the attention-block options (QK RMSNorm, sigmoid output gate;
App. B.5) against the CPU oracle, through the C ABI.

Same rules as the plain path: bf16 max error beyond storage rounding <= 2e-2 *
RMS of the oracle value, float32 max abs error <= 1e-5; LSE within 2e-2 (bf16)
or 1e-5 (f32) natural-log units."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_31248_amd import binding as B
from paper_2606_31248_amd import inputs as I
from paper_2606_31248_amd import pipeline
from _util import LSE_ABS_BF16, bf16_half_ulp, check_close, dev_tensor, host_bits, host_f64, host_rows
from oracle import geometry as G

pytestmark = pytest.mark.gpu

ROPE_BASE = pipeline.ROPE_BASE


# (qk_norm, gate kind): gate kind 0 = none, 1 = one logit per (token, head), "d" = per channel
OPTIONS = [(True, 0), (False, 1), (False, "d"), (True, "d"), (True, 1)]
OPT_IDS = ["norm", "gate1", "gateD", "norm+gateD", "norm+gate1"]


def coords_for(shape, seed):
    pl = I.random_placement(shape[0], shape[3], shape[4], seed)
    return G.tile_coords(pl.face, pl.oy, pl.ox, shape[3], shape[4]).astype(np.float32)


def gpu_phases(coords32, d):
    c = torch.from_numpy(coords32).cuda()
    cs = torch.empty(coords32.shape[:3] + (d // 2, 2), dtype=torch.float32, device="cuda")
    B.strata_stereorope_phases(c, d, ROPE_BASE, cs)
    return cs


def gate_logits(shape, kind, seed, dtype, mult=2.0):
    if kind == 0:
        return None
    gshape = shape[:-1] if kind == 1 else shape
    return I.gaussian(gshape, seed, I.STREAM_GATE, dtype, mult)


def run_fwd_ex(shape, window, dtype, seed, qk_norm, gkind, coords32=None, scale=None, qk_mult=1.0, eps=1e-6,
               gate_mult=2.0):
    q = I.gaussian(shape, seed, 0, dtype, qk_mult)
    k = I.gaussian(shape, seed, 1, dtype, qk_mult)
    v = I.gaussian(shape, seed, 2, dtype)
    g = gate_logits(shape, gkind, seed, dtype, gate_mult)
    scale = scale or 1.0 / np.sqrt(shape[-1])
    qd, kd, vd = (dev_tensor(a, dtype) for a in (q, k, v))
    gd = None if g is None else dev_tensor(g, dtype)
    cs = gpu_phases(coords32, shape[-1]) if coords32 is not None else None
    out = torch.empty_like(qd)
    lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
    opts = B.make_opts(qk_norm, eps, gd)
    B.strata_na3d_fwd_ex(B.desc_for(qd, window, scale), opts, qd, kd, vd, cs, out, lse)
    torch.cuda.synchronize()
    return (q, k, v, g), (qd, kd, vd, gd, cs, opts), out, lse, scale


def oracle_fwd(inputs, window, scale, dtype, qk_norm, coords32, eps=1e-6, sel=None):
    q, k, v, g = inputs
    w = lambda a: None if a is None else oracle.widen(a, dtype)
    return oracle.na3d_fwd(w(q), w(k), w(v), window, scale, coords=coords32, sel=sel, qk_norm=qk_norm, eps=eps,
                           gate=w(g))


def check_gated(got, ref, ref_attn, sig, dtype, what):
    """The gate multiplies the attention output A and so its error.  The plain
    rule lets A be off by 2e-2 * RMS(A) beyond its bf16 storage rounding; the
    gated output is sigmoid(g) times A's float32 value, rounded once: so bf16
    elements must lie within sigmoid(g) (2e-2 RMS(A) + half an ulp of A) + half
    an ulp of the result of the oracle, never looser than the plain rule (with a
    floor of the smallest normal float, below which results may flush to zero);
    float32 within 1e-5."""
    diff = np.abs(got - ref)
    if dtype == "bf16":
        rms = float(np.sqrt(np.mean(ref_attn * ref_attn)))
        excess = diff - bf16_half_ulp(ref) - sig * (2e-2 * rms + bf16_half_ulp(ref_attn)) - 2.0 ** -126
        assert float(np.max(excess)) <= 0.0, (
            f"{what}: error beyond sigma * 2e-2 RMS(A) + rounding by {float(np.max(excess)):.3e} "
            f"(max abs err {float(np.max(diff)):.3e}, RMS(A) {rms:.3e})")
    else:
        assert float(np.max(diff)) <= 1e-5, f"{what}: max abs err {float(np.max(diff)):.3e}"


def sigmoid_of(g, dtype, shape):
    """sigmoid(g) of stored gate logits, broadcast to the output shape."""
    gl = oracle.widen(g, dtype)
    s = 1.0 / (1.0 + np.exp(-gl))
    return s[..., None] if gl.shape != tuple(shape) else s


def check_out(got, inputs, window, scale, dtype, qk_norm, coords32, ref, eps=1e-6, sel=None):
    """Output check: the plain rule without a gate, the gate-scaled rule with one."""
    g = inputs[3]
    if g is None:
        check_close(got, ref, dtype, "out")
        return
    ra, _ = oracle_fwd(inputs[:3] + (None,), window, scale, dtype, qk_norm, coords32, eps=eps, sel=sel)
    sig = sigmoid_of(g, dtype, inputs[0].shape)
    if sel is not None:
        sig = sig.reshape(-1, sig.shape[-1])[sel]
    check_gated(got, ref, ra, sig, dtype, "out")


def check_lse(got, ref, dtype):
    tol = LSE_ABS_BF16 if dtype == "bf16" else 1e-5
    err = float(np.max(np.abs(host_f64(got) - ref)))
    assert err <= tol, f"lse: {err:.3e} > {tol}"


# ----------------------------------------------------------------------------- forward

FWD_SHAPES = [
    ((2, 3, 8, 19, 21, 64), (3, 7, 7), "bf16"),   # level-sweep kernel, ragged blocks
    ((1, 11, 8, 16, 24, 64), (3, 7, 7), "bf16"),  # level-sweep kernel, ragged head group
    ((2, 3, 5, 19, 21, 64), (3, 7, 7), "bf16"),   # query-stationary MFMA kernel
    ((1, 2, 6, 24, 24, 64), (5, 9, 9), "bf16"),   # query-stationary MFMA kernel, 5x9x9
    ((2, 2, 3, 16, 12, 32), (3, 5, 7), "bf16"),   # plain kernel, bf16
    ((1, 2, 4, 9, 11, 32), (3, 5, 7), "f32"),     # plain kernel, float32
    ((1, 1, 3, 8, 8, 64), (3, 3, 3), "f32"),
]


@pytest.mark.parametrize("shape,window,dtype", FWD_SHAPES)
@pytest.mark.parametrize("qk_norm,gkind", OPTIONS, ids=OPT_IDS)
def test_fwd_options_full_oracle(shape, window, dtype, qk_norm, gkind):
    c32 = coords_for(shape, 95)
    inputs, _, out, lse, scale = run_fwd_ex(shape, window, dtype, 51, qk_norm, gkind, c32)
    ro, rl = oracle_fwd(inputs, window, scale, dtype, qk_norm, c32)
    check_out(host_f64(out), inputs, window, scale, dtype, qk_norm, c32, ro)
    check_lse(lse, rl, dtype)


@pytest.mark.parametrize("shape,window", [((1, 2, 8, 19, 21, 64), (3, 7, 7)), ((1, 2, 6, 24, 24, 64), (5, 9, 9))])
@pytest.mark.parametrize("scale", [0.125, 0.5, 0.7])
def test_fwd_norm_tames_huge_inputs(shape, window, scale):
    """q, k of magnitude ~64 (logits of +-1000s without the norm): with QK RMSNorm
    the logits are bounded by scale * head_dim; larger scales give sharper
    softmax rows, whose maximum the kernels' reference then has to follow."""
    c32 = coords_for(shape, 96)
    inputs, _, out, lse, _ = run_fwd_ex(shape, window, "bf16", 52, True, "d", c32, scale=scale, qk_mult=64.0)
    ro, rl = oracle_fwd(inputs, window, scale, "bf16", True, c32)
    check_out(host_f64(out), inputs, window, scale, "bf16", True, c32, ro)
    check_lse(lse, rl, "bf16")


@pytest.mark.parametrize("shape,window,dtype", [FWD_SHAPES[0], FWD_SHAPES[3], FWD_SHAPES[5]])
def test_fwd_eps_enters_under_the_root(shape, window, dtype):
    """eps = 4 against inputs of mean square ~1: the factor differs visibly from 1/RMS."""
    c32 = coords_for(shape, 97)
    inputs, _, out, lse, scale = run_fwd_ex(shape, window, dtype, 53, True, 0, c32, eps=4.0)
    ro, rl = oracle_fwd(inputs, window, scale, dtype, True, c32, eps=4.0)
    check_close(host_f64(out), ro, dtype, "out")
    check_lse(lse, rl, dtype)


@pytest.mark.parametrize("shape,window,dtype", [FWD_SHAPES[0], FWD_SHAPES[2], FWD_SHAPES[5]])
@pytest.mark.parametrize("gkind", [1, "d"])
def test_fwd_saturated_gates(shape, window, dtype, gkind):
    """Gate logits of +-40: sigmoid is 1 or 0 to float32 precision."""
    c32 = coords_for(shape, 98)
    inputs, _, out, lse, scale = run_fwd_ex(shape, window, dtype, 54, False, gkind, c32, gate_mult=40.0)
    ro, rl = oracle_fwd(inputs, window, scale, dtype, False, c32)
    check_out(host_f64(out), inputs, window, scale, dtype, False, c32, ro)
    check_lse(lse, rl, dtype)


@pytest.mark.parametrize("shape,window,dtype", [FWD_SHAPES[0], FWD_SHAPES[3], FWD_SHAPES[5]])
def test_fwd_ex_without_options_is_the_plain_forward(shape, window, dtype):
    c32 = coords_for(shape, 99)
    _, (qd, kd, vd, _, cs, _), _, _, scale = run_fwd_ex(shape, window, dtype, 55, False, 0, c32)
    desc = B.desc_for(qd, window, scale)
    outs = []
    for opts in (None, B.make_opts(False, 0.0, None), "plain"):
        out = torch.empty_like(qd)
        lse = torch.empty(shape[:-1], dtype=torch.float32, device="cuda")
        if opts == "plain":
            B.strata_na3d_fwd(desc, qd, kd, vd, cs, out, lse)
        else:
            B.strata_na3d_fwd_ex(desc, opts, qd, kd, vd, cs, out, lse)
        torch.cuda.synchronize()
        outs.append((host_bits(out), host_bits(lse)))
    for o, l in outs[1:]:
        assert np.array_equal(o, outs[0][0]) and np.array_equal(l, outs[0][1])


@pytest.mark.parametrize("shape,window,dtype", [FWD_SHAPES[0], FWD_SHAPES[2], FWD_SHAPES[3], FWD_SHAPES[5]])
@pytest.mark.parametrize("gkind", [1, "d"])
def test_fwd_zero_gate_halves_the_output_exactly(shape, window, dtype, gkind):
    """sigmoid(0) = 1/2 exactly and halving is exact in both float formats: the
    gated output is the plain output halved, bit for bit."""
    c32 = coords_for(shape, 102)
    _, (qd, kd, vd, _, cs, _), out, lse, scale = run_fwd_ex(shape, window, dtype, 56, False, 0, c32)
    g0 = torch.zeros(shape[:-1] if gkind == 1 else shape, dtype=qd.dtype, device="cuda")
    out2 = torch.empty_like(out)
    lse2 = torch.empty_like(lse)
    B.strata_na3d_fwd_ex(B.desc_for(qd, window, scale), B.make_opts(False, 1e-6, g0), qd, kd, vd, cs, out2, lse2)
    torch.cuda.synchronize()
    assert torch.equal(out2, out * 0.5)
    assert np.array_equal(host_bits(lse2), host_bits(lse))


def test_fwd_options_full_size_sampled():
    """The face roll-out (81 tiles x 16 heads x 8 x 64 x 64, 3x7x7) with QK RMSNorm
    and a per-channel gate, as one launch; sampled outputs vs the oracle."""
    wl = I.FACE_ROLLOUT
    shape = wl.shape()
    window = (wl.kz, wl.ky, wl.kx)
    pl = wl.placement()
    c32 = G.tile_coords(pl.face, pl.oy, pl.ox, wl.H, wl.W).astype(np.float32)
    inputs, _, out, lse, scale = run_fwd_ex(shape, window, "bf16", wl.seed, True, "d", c32)
    tiles = sorted({0, shape[0] // 2, shape[0] - 1})
    per_tile = shape[1] * wl.N
    r = np.random.default_rng(wl.seed)
    sel = np.unique(np.concatenate([r.integers(0, per_tile, 1500) + t * per_tile for t in tiles]))
    local = np.searchsorted(tiles, sel // per_tile) * per_tile + sel % per_tile
    sub = tuple(None if a is None else a[tiles] for a in inputs)
    ro, rl = oracle_fwd(sub, window, scale, "bf16", True, c32[tiles], sel=local)
    check_out(host_rows(out, sel, wl.d), sub, window, scale, "bf16", True, c32[tiles], ro, sel=local)
    assert np.max(np.abs(host_rows(lse, sel) - rl)) <= LSE_ABS_BF16
    assert torch.isfinite(out.float()).all()


# ----------------------------------------------------------------------------- backward

def run_bwd_ex(shape, window, dtype, seed, qk_norm, gkind, coords32, qk_mult=1.0, eps=1e-6):
    inputs, (qd, kd, vd, gd, cs, opts), out, lse, scale = run_fwd_ex(shape, window, dtype, seed, qk_norm, gkind,
                                                                     coords32, qk_mult=qk_mult, eps=eps)
    dout = I.gaussian(shape, seed, I.STREAM_DO, dtype)
    dod = dev_tensor(dout, dtype)
    desc = B.desc_for(qd, window, scale)
    ws = torch.empty(B.strata_na3d_bwd_ex_workspace_size(desc, opts), dtype=torch.uint8, device="cuda")
    dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
    dg = None if gd is None else torch.empty_like(gd)
    B.strata_na3d_bwd_ex(desc, opts, qd, kd, vd, cs, out, dod, lse, dq, dk, dv, dg, ws)
    torch.cuda.synchronize()
    return inputs + (dout,), (dq, dk, dv, dg), scale


def fwd_bound(ra, ro, sig):
    """Per-element error the forward checks permit for the gated output."""
    rms = float(np.sqrt(np.mean(ra * ra)))
    return sig * (2e-2 * rms + bf16_half_ulp(ra)) + bf16_half_ulp(ro) + 2.0 ** -126


def check_bwd_grads(inputs, grads, refs, window, scale, dtype, qk_norm, coords32, sel=None, presliced=False):
    """dq, dk: the plain rule.  dv, with a gate: also the elementwise bound
    2^-8 sum_q P |dA_q| of the P rounding in the bf16 P.dA product (the gate
    gives dA rows of mixed magnitudes, as in the plain suite's mixed-dO case).
    dgate = (1 - a) dO out is computed from the forward's output: beyond the
    plain rule it may carry that output's permitted error times (1 - a) |dO|
    (summed over the channels for one logit per token and head)."""
    q, k, v, g, dout = inputs
    w = lambda a: None if a is None else oracle.widen(a, dtype)
    rows = (lambda a: a.reshape(-1, a.shape[-1])[sel]) if sel is not None else (lambda a: a)
    got = [None if x is None else host_f64(x) for x in grads]
    if sel is not None and not presliced:
        got = [None if x is None else (x.reshape(-1)[sel] if x.ndim == 5 else x.reshape(-1, x.shape[-1])[sel])
               for x in got]
    check_close(got[0], refs[0], dtype, "dq")
    check_close(got[1], refs[1], dtype, "dk")
    if g is None or dtype != "bf16":
        check_close(got[2], refs[2], dtype, "dv")
        if g is not None:
            check_close(got[3], refs[3], dtype, "dgate")
        return
    kw = dict(coords=coords32, qk_norm=qk_norm, gate=w(g))
    if sel is not None:
        kw.update(selq=sel, selk=sel)
    a_dv = oracle.na3d_bwd(w(q), w(k), w(v), np.abs(w(dout)), window, scale, **kw)[2]
    rms = float(np.sqrt(np.mean(refs[2] ** 2)))
    excess = np.abs(got[2] - refs[2]) - bf16_half_ulp(refs[2]) - np.ldexp(a_dv, -8)
    assert float(np.max(excess)) <= 2e-2 * rms, f"dv: {float(np.max(excess)):.3e} > {2e-2 * rms:.3e}"
    # dgate
    ra, _ = oracle_fwd((q, k, v, None), window, scale, dtype, qk_norm, coords32, sel=sel)
    ro, _ = oracle_fwd((q, k, v, g), window, scale, dtype, qk_norm, coords32, sel=sel)
    gl = w(g)
    head = gl.ndim == 5
    sig = 1.0 / (1.0 + np.exp(-gl))
    rsig = 1.0 / (1.0 + np.exp(gl))
    if head:
        sig, rsig = sig[..., None], rsig[..., None]
    sig, rsig, dof = rows(sig), rows(rsig), rows(w(dout))
    b = rsig * np.abs(dof) * fwd_bound(ra, ro, sig)
    if head:
        b = b.sum(-1)
        if sel is None:
            b = b.reshape(gl.shape)
    ref = refs[3]
    rmsg = float(np.sqrt(np.mean(ref ** 2)))
    excess = np.abs(got[3] - ref) - bf16_half_ulp(ref) - b
    assert float(np.max(excess)) <= 2e-2 * rmsg, f"dgate: {float(np.max(excess)):.3e} > {2e-2 * rmsg:.3e}"


BWD_SHAPES = [
    ((1, 2, 5, 11, 13, 64), (3, 7, 7), "bf16"),
    ((2, 1, 6, 12, 10, 64), (5, 9, 9), "bf16"),
    ((1, 2, 4, 9, 11, 32), (3, 5, 7), "f32"),
    ((1, 1, 3, 8, 8, 32), (1, 3, 5), "bf16"),
]


@pytest.mark.parametrize("shape,window,dtype", BWD_SHAPES)
@pytest.mark.parametrize("qk_norm,gkind", OPTIONS, ids=OPT_IDS)
def test_bwd_options_full_oracle(shape, window, dtype, qk_norm, gkind):
    c32 = coords_for(shape, 100)
    (q, k, v, g, dout), grads, scale = run_bwd_ex(shape, window, dtype, 61, qk_norm, gkind, c32)
    w = lambda a: None if a is None else oracle.widen(a, dtype)
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(dout), window, scale, coords=c32, qk_norm=qk_norm, gate=w(g))
    assert len(refs) == (3 if g is None else 4)
    check_bwd_grads((q, k, v, g, dout), grads, refs, window, scale, dtype, qk_norm, c32)


@pytest.mark.parametrize("shape,window", [((1, 2, 5, 11, 13, 64), (3, 7, 7)), ((2, 1, 6, 12, 10, 64), (5, 9, 9))])
def test_bwd_norm_with_huge_inputs(shape, window):
    c32 = coords_for(shape, 101)
    (q, k, v, g, dout), grads, scale = run_bwd_ex(shape, window, "bf16", 62, True, "d", c32, qk_mult=64.0)
    w = lambda a: oracle.widen(a, "bf16")
    refs = oracle.na3d_bwd(w(q), w(k), w(v), w(dout), window, scale, coords=c32, qk_norm=True, gate=w(g))
    check_bwd_grads((q, k, v, g, dout), grads, refs, window, scale, "bf16", True, c32)


def test_bwd_options_full_size_sampled():
    """The 16-tile 5x9x9 training tile with QK RMSNorm and a per-channel gate;
    sampled rows of dq, dk, dv, dgate vs the oracle."""
    wl = I.TRAIN_TILE_BWD
    shape = wl.shape()
    window = (wl.kz, wl.ky, wl.kx)
    pl = wl.placement()
    c32 = G.tile_coords(pl.face, pl.oy, pl.ox, wl.H, wl.W).astype(np.float32)
    (q, k, v, g, dout), (dq, dk, dv, dg), scale = run_bwd_ex(shape, window, "bf16", wl.seed, True, "d", c32)
    tiles = [0, shape[0] - 1]
    per_tile = shape[1] * wl.N
    r = np.random.default_rng(wl.seed)
    sel = np.unique(np.concatenate([r.integers(0, per_tile, 80) + t * per_tile for t in tiles]))
    local = np.searchsorted(tiles, sel // per_tile) * per_tile + sel % per_tile
    sub = lambda a: oracle.widen(a[tiles], "bf16")
    refs = oracle.na3d_bwd(sub(q), sub(k), sub(v), sub(dout), window, scale, coords=c32[tiles],
                           selq=local, selk=local, qk_norm=True, gate=sub(g))
    # gradients of the sampled rows, the oracle seeing only the sampled tiles
    got = [host_rows(x, sel, wl.d) for x in (dq, dk, dv, dg)]
    st = lambda a: a[tiles]
    check_bwd_grads((st(q), st(k), st(v), st(g), st(dout)), [torch.from_numpy(x) for x in got], refs, window,
                    scale, "bf16", True, c32[tiles], sel=local, presliced=True)

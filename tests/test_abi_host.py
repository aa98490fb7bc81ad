"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every symbol the header declares, and rejects bad arguments before launching."""
import ctypes
import os
import re

import pytest

from paper_2606_31248_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "strata.h")


def header_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(strata_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    syms = header_symbols()
    for name in ("strata_stereorope_apply", "strata_na3d_fwd", "strata_na3d_bwd", "strata_tile_blend"):
        assert name in syms
    assert sorted(B.EXPORTS) == syms


def test_library_exports_every_header_symbol():
    L = B.load()
    for name in header_symbols():
        assert hasattr(L, name), name


def test_status_strings():
    L = B.load()
    assert L.strata_status_string(0) == b"ok"
    assert L.strata_status_string(3) == b"workspace too small"


def fake(addr=0x10000):
    return ctypes.c_void_p(addr)


def call_fwd(desc, q=fake(), k=fake(), v=fake(), out=fake()):
    return B.load().strata_na3d_fwd(ctypes.byref(desc) if desc is not None else None, q, k, v, None,
                                    out, None, None)


GOOD = dict(B=1, heads=2, Z=8, H=16, W=16, head_dim=64, window=(3, 7, 7), scale=0.125, dtype=B.STRATA_BF16)


def desc(**kw):
    a = dict(GOOD)
    a.update(kw)
    return B.make_desc(a["B"], a["heads"], a["Z"], a["H"], a["W"], a["head_dim"], a["window"], a["scale"],
                       a["dtype"])


@pytest.mark.parametrize("kw,status", [
    (dict(window=(2, 7, 7)), B.STRATA_ERR_INVALID_ARG),       # even window
    (dict(window=(3, 17, 7)), B.STRATA_ERR_INVALID_ARG),      # larger than the grid
    (dict(window=(3, 0, 7)), B.STRATA_ERR_INVALID_ARG),
    (dict(H=0), B.STRATA_ERR_INVALID_ARG),
    (dict(scale=0.0), B.STRATA_ERR_INVALID_ARG),
    (dict(scale=float("nan")), B.STRATA_ERR_INVALID_ARG),
    (dict(dtype=7), B.STRATA_ERR_INVALID_ARG),
    (dict(head_dim=48), B.STRATA_ERR_UNSUPPORTED),
])
def test_fwd_rejects_bad_descriptors(kw, status):
    assert call_fwd(desc(**kw)) == status
    assert B.load().strata_last_error() != b""


def test_fwd_rejects_null_and_misaligned_pointers():
    assert call_fwd(None) == B.STRATA_ERR_INVALID_ARG
    assert call_fwd(desc(), q=None) == B.STRATA_ERR_INVALID_ARG
    assert call_fwd(desc(), out=fake(0x10008)) == B.STRATA_ERR_INVALID_ARG
    assert b"aligned" in B.load().strata_last_error()


def test_bwd_workspace_rules():
    L = B.load()
    d = desc()
    need = L.strata_na3d_bwd_workspace_size(ctypes.byref(d))
    assert need >= 1 * 2 * 8 * 16 * 16 * 4 and need % 256 == 0
    p = fake()
    st = L.strata_na3d_bwd(ctypes.byref(d), p, p, p, None, p, p, p, p, p, p, p, need - 1, None)
    assert st == B.STRATA_ERR_WORKSPACE
    st = L.strata_na3d_bwd(ctypes.byref(d), p, p, p, None, p, p, None, p, p, p, p, need, None)
    assert st == B.STRATA_ERR_INVALID_ARG   # lse is required


def test_tiling_rules():
    L = B.load()
    p = fake()
    # tiles reaching past the face
    assert L.strata_tile_blend(p, 9, 9, 4, 64, 64, 64, 56, 56, p, p, 511, 512, B.STRATA_BF16, None) == \
        B.STRATA_ERR_INVALID_ARG
    assert L.strata_tile_extract(p, 2, 2, 1, 8, 8, 8, 0, 8, 16, 16, p, B.STRATA_F32, None) == \
        B.STRATA_ERR_INVALID_ARG


def test_axis_and_rope_rules():
    L = B.load()
    p = fake()
    assert L.strata_na_axis_index(5, 2, p, p, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_na_axis_index(5, 7, p, p, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_stereorope_phases(p, 1, 4, 4, 30, 100.0, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_stereorope_phases(p, 1, 4, 4, 32, -1.0, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_stereorope_apply(p, p, p, 1, 1, 1, 4, 4, 36, 1, 0, None) == B.STRATA_ERR_UNSUPPORTED
    assert L.strata_stereo_coords(p, p, p, 1, 600, 4, 2048, 4, 1e-3, p, None) == B.STRATA_ERR_INVALID_ARG


def opts(qk_norm=0, eps=1e-6, gate=None, gate_dim=0):
    return B.NA3DOpts(qk_norm, eps, gate, gate_dim)


def call_fwd_ex(d, o):
    p = fake()
    return B.load().strata_na3d_fwd_ex(ctypes.byref(d), None if o is None else ctypes.byref(o), p, p, p, None, p,
                                       None, None)


@pytest.mark.parametrize("o", [
    opts(qk_norm=1, eps=float("nan")),
    opts(qk_norm=1, eps=-1e-6),
    opts(qk_norm=1, eps=float("inf")),
    opts(gate=fake(), gate_dim=0),
    opts(gate=fake(), gate_dim=32),           # neither 1 nor head_dim (64)
    opts(gate=fake(0x10002), gate_dim=1),     # misaligned
])
def test_fwd_ex_rejects_bad_options(o):
    assert call_fwd_ex(desc(), o) == B.STRATA_ERR_INVALID_ARG
    assert b"opts" in B.load().strata_last_error()


def test_fwd_ex_checks_the_descriptor_first():
    assert call_fwd_ex(desc(window=(2, 7, 7)), opts(qk_norm=1)) == B.STRATA_ERR_INVALID_ARG


def test_bwd_ex_workspace_layout():
    L = B.load()
    d = desc()
    n = 1 * 2 * 8 * 16 * 16
    row = n * 64 * 2
    base = L.strata_na3d_bwd_workspace_size(ctypes.byref(d))
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), None) == base
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(opts())) == base
    # a gate adds dA as two bf16 terms; the norm needs no workspace
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(opts(gate=fake(), gate_dim=1))) == \
        base + 2 * row
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(opts(qk_norm=1))) == base
    both = opts(qk_norm=1, gate=fake(), gate_dim=64)
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(both)) == base + 2 * row
    f32 = desc(dtype=B.STRATA_F32)
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(f32), ctypes.byref(both)) == \
        L.strata_na3d_bwd_workspace_size(ctypes.byref(f32)) + 2 * row  # one float32 term
    assert L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(opts(gate=fake(), gate_dim=3))) == 0


def test_bwd_ex_requires_dgate_with_a_gate_and_enough_workspace():
    L = B.load()
    d = desc()
    o = opts(gate=fake(), gate_dim=1)
    need = L.strata_na3d_bwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(o))
    p = fake()
    st = L.strata_na3d_bwd_ex(ctypes.byref(d), ctypes.byref(o), p, p, p, None, p, p, p, p, p, p, None, p, need,
                              None)
    assert st == B.STRATA_ERR_INVALID_ARG and b"dgate" in L.strata_last_error()
    st = L.strata_na3d_bwd_ex(ctypes.byref(d), ctypes.byref(o), p, p, p, None, p, p, p, p, p, p, p, p, need - 1,
                              None)
    assert st == B.STRATA_ERR_WORKSPACE


def test_wind_rules():
    L = B.load()
    p = fake()
    assert L.strata_wind_tile_frame(p, 6, 64, 1, 1, 1, 8, 8, 8, 8, p, B.STRATA_F32, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_wind_tile_frame(p, 0, 64, 2, 1, 1, 40, 8, 30, 8, p, B.STRATA_F32, None) == \
        B.STRATA_ERR_INVALID_ARG   # (2-1)*30 + 40 > 64
    assert L.strata_wind_tile_frame(None, 0, 64, 1, 1, 1, 8, 8, 8, 8, p, B.STRATA_F32, None) == \
        B.STRATA_ERR_INVALID_ARG


def test_kbd_rules():
    L = B.load()
    p = fake()
    assert L.strata_kbd_window(8, 8, 0, 4.0, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_kbd_window(8, 8, 9, 4.0, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_kbd_window(8, 8, 4, -1.0, p, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_kbd_window(8, 8, 4, 4.0, None, None) == B.STRATA_ERR_INVALID_ARG


def test_duo_rules():
    L = B.load()
    p = fake()
    assert L.strata_duo_pad(p, 1, 8, 1, 1, p, B.STRATA_F32, None) == B.STRATA_ERR_INVALID_ARG     # n < 16
    assert L.strata_duo_pad(p, 1, 32, 1, 9, p, B.STRATA_F32, None) == B.STRATA_ERR_INVALID_ARG    # halo > n/4
    assert L.strata_duo_pad(p, 1, 32, 1, 0, p, B.STRATA_F32, None) == B.STRATA_ERR_INVALID_ARG
    # within the element limit, but more interior rows than one launch can take
    assert L.strata_duo_pad(p, 1 << 27, 16, 1, 4, p, B.STRATA_F32, None) == B.STRATA_ERR_INVALID_ARG


def test_duo_plan_rules():
    L = B.load()
    p = fake()
    # P (64 bytes per halo cell), its transpose (4 x 16 bytes per halo cell) and
    # one build counter per face cell, at least
    for n, h in ((16, 4), (2048, 16)):
        nh = 6 * ((n + 2 * h) ** 2 - n * n)
        assert B.strata_duo_plan_bytes(n, h) >= nh * 128 + 6 * n * n * 4
        assert B.strata_duo_plan_bytes(n, h) % 16 == 0
    assert B.strata_duo_plan_bytes(8, 1) == 0 and B.strata_duo_plan_bytes(32, 9) == 0
    assert B.strata_duo_plan_bytes(16384, 16) == 0                       # n + 2 halo >= 2^14
    assert B.strata_duo_plan_bytes(16350, 16) > 0
    need = B.strata_duo_plan_bytes(32, 4)
    assert L.strata_duo_plan(32, 4, p, need - 1, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_plan(32, 4, None, need, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_plan(32, 4, fake(0x10008), need, None) == B.STRATA_ERR_INVALID_ARG  # misaligned
    assert L.strata_duo_plan(32, 9, p, need, None) == B.STRATA_ERR_INVALID_ARG
    F = B.STRATA_F32
    assert L.strata_duo_pad_planned(p, 1, 32, 1, 4, p, need - 1, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_planned(p, 1, 32, 1, 4, None, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_planned(p, 1, 32, 1, 4, fake(0x10004), need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_planned(p, 0, 32, 1, 4, p, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_planned(p, 1, 32, 1, 4, p, need, p, 7, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(p, 1, 32, 1, 4, p, need - 1, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(p, 1, 32, 1, 4, None, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(p, 1, 32, 1, 4, fake(0x10004), need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(p, 1, 32, 1, 9, p, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(None, 1, 32, 1, 4, p, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(p, 65536, 32, 1, 4, p, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    # every device buffer must be 16-byte aligned (the narrow copy paths serve odd layouts only)
    odd = fake(0x10002)
    assert L.strata_duo_pad(odd, 1, 32, 1, 4, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad(p, 1, 32, 1, 4, odd, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_planned(odd, 1, 32, 1, 4, p, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_planned(p, 1, 32, 1, 4, p, need, odd, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(odd, 1, 32, 1, 4, p, need, p, F, None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_duo_pad_vjp(p, 1, 32, 1, 4, p, need, odd, F, None) == B.STRATA_ERR_INVALID_ARG


def test_fwd_stitch_rules():
    L = B.load()
    p = fake()
    d = desc(B=4)

    def call(nty=2, ntx=2, sy=8, sx=8, Hf=24, Wf=24, face=p, dd=d):
        return L.strata_na3d_fwd_stitch(ctypes.byref(dd), None, p, p, p, None, p, None, nty, ntx, sy, sx, p,
                                        face, Hf, Wf, None)

    assert call(nty=3, ntx=1) == B.STRATA_ERR_INVALID_ARG          # the batch is not the tiling
    assert call(Hf=20) == B.STRATA_ERR_INVALID_ARG                 # tiles reach past the face
    assert call(sy=0) == B.STRATA_ERR_INVALID_ARG
    assert call(face=None) == B.STRATA_ERR_INVALID_ARG
    assert call(face=fake(0x10008)) == B.STRATA_ERR_INVALID_ARG     # misaligned
    assert call(dd=desc(B=4, window=(2, 7, 7))) == B.STRATA_ERR_INVALID_ARG
    # heads * Z beyond 32 bits (a descriptor the attention calls accept)
    big = desc(B=4, heads=1 << 16, Z=(1 << 16) + 1, H=1, W=1, head_dim=32, window=(1, 1, 1))
    assert call(nty=2, ntx=2, sy=1, sx=1, Hf=2, Wf=2, dd=big) == B.STRATA_ERR_INVALID_ARG
    assert b"32 bits" in B.load().strata_last_error()
    assert L.strata_tile_blend_overlap(p, 9, 9, 4, 64, 64, 64, 56, 56, p, p, 511, 512, B.STRATA_BF16,
                                       None) == B.STRATA_ERR_INVALID_ARG
    assert L.strata_tile_blend_overlap(p, 9, 9, 4, 64, 64, 64, 56, 56, None, p, 512, 512, B.STRATA_BF16,
                                       None) == B.STRATA_ERR_INVALID_ARG


def test_bwd_workspace_layout():
    """D (float32 per token-head) and one int32 word per batch-head, each region
    on a 256-byte boundary; the gate adds its dA terms after them."""
    L = B.load()
    al = lambda x: (x + 255) // 256 * 256
    for kw in (dict(), dict(B=3, heads=5, Z=7, H=9, W=11), dict(B=70, heads=1000, Z=1, H=1, W=1, window=(1, 1, 1))):
        d = desc(**kw)
        bh = d.B * d.heads
        n = bh * d.Z * d.H * d.W
        assert L.strata_na3d_bwd_workspace_size(ctypes.byref(d)) == al(4 * n) + al(4 * bh)


def test_noalloc_rejects_too_many_batch_heads():
    """The allocation-free backward's static array holds one word per batch-head
    up to 2^16 of them: more are rejected on the host, before any launch."""
    L = B.load()
    p = fake()
    ok = desc(B=1 << 8, heads=1 << 8, Z=1, H=1, W=1, window=(1, 1, 1))  # 2^16 batch-heads: the limit
    big = desc(B=(1 << 8) + 1, heads=1 << 8, Z=1, H=1, W=1, window=(1, 1, 1))
    assert L.strata_na3d_bwd_noalloc(ctypes.byref(big), p, p, p, None, p, p, p, p, p, p, None) == \
        B.STRATA_ERR_INVALID_ARG
    assert b"static scratch" in L.strata_last_error()
    assert L.strata_na3d_bwd_workspace_size(ctypes.byref(ok)) <= (1 << 25) + (1 << 18)

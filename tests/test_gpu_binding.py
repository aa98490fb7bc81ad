"""The Python binding rejects, before any launch, device tensors whose shape,
dtype or device disagree with the problem (the C ABI sees only pointers)."""
import pytest
import torch

from paper_2606_31248_amd import binding as B

pytestmark = pytest.mark.gpu

SHAPE = (1, 2, 8, 16, 16, 64)


def dev(shape, dtype=torch.bfloat16):
    return torch.zeros(shape, dtype=dtype, device="cuda")


@pytest.mark.parametrize("bad", ["k_shape", "v_dtype", "out_shape", "cs_shape", "lse_shape", "cpu_out"])
def test_forward_mismatches(bad):
    desc = B.make_desc(*SHAPE, (3, 7, 7), 0.125, B.STRATA_BF16)
    t = {n: dev(SHAPE) for n in ("q", "k", "v", "out")}
    cs = dev((1, 16, 16, 32, 2), torch.float32)
    lse = dev(SHAPE[:-1], torch.float32)
    if bad == "k_shape":
        t["k"] = dev((1, 2, 8, 16, 15, 64))
    elif bad == "v_dtype":
        t["v"] = dev(SHAPE, torch.float32)
    elif bad == "out_shape":
        t["out"] = dev((2, 2, 8, 16, 16, 64))
    elif bad == "cs_shape":
        cs = dev((1, 16, 16, 64), torch.float32)
    elif bad == "lse_shape":
        lse = dev(SHAPE, torch.float32)
    else:
        t["out"] = torch.zeros(SHAPE, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        B.strata_na3d_fwd(desc, t["q"], t["k"], t["v"], cs, t["out"], lse)


def test_backward_and_gate_mismatches():
    desc = B.make_desc(*SHAPE, (3, 7, 7), 0.125, B.STRATA_BF16)
    q = dev(SHAPE)
    lse = dev(SHAPE[:-1], torch.float32)
    ws = dev((B.strata_na3d_bwd_workspace_size(desc),), torch.uint8)
    with pytest.raises(ValueError):  # dq of the wrong shape
        B.strata_na3d_bwd(desc, q, q, q, None, q, q, lse, dev((1, 2, 8, 16, 16, 32)), q, q, ws)
    with pytest.raises(ValueError):  # lse missing
        B.strata_na3d_bwd(desc, q, q, q, None, q, q, None, q, q, q, ws)
    opts = B.make_opts(gate=dev((1, 2, 8, 16, 16, 3)))
    with pytest.raises(ValueError):  # gate neither per token nor per channel
        B.strata_na3d_fwd_ex(desc, opts, q, q, q, None, q)


def test_tiling_mismatches():
    tiles = dev((4, 3, 8, 8, 16))
    win = dev((64,), torch.float32)
    face = dev((3, 12, 12, 16))
    with pytest.raises(ValueError):  # 4 tiles are not a 3 x 2 tiling
        B.strata_tile_blend(tiles, 3, 2, 4, 4, win, face)
    with pytest.raises(ValueError):  # window of the wrong size
        B.strata_tile_blend(tiles, 2, 2, 4, 4, dev((63,), torch.float32), face)
    with pytest.raises(ValueError):  # face of another dtype
        B.strata_tile_blend(tiles, 2, 2, 4, 4, win, dev((3, 12, 12, 16), torch.float32))
    with pytest.raises(ValueError):  # face with other channels
        B.strata_tile_extract(dev((3, 12, 12, 8)), 2, 2, 4, 4, tiles)

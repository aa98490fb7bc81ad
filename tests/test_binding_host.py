"""The Python binding refuses tensors the C ABI cannot check (no GPU needed):
a host tensor never reaches a device pointer argument."""
import pytest
import torch

from paper_2606_31248_amd import binding as B


def cpu(shape, dtype=torch.bfloat16):
    return torch.zeros(shape, dtype=dtype)


SHAPE = (1, 2, 8, 16, 16, 64)


def test_forward_rejects_host_tensors():
    desc = B.make_desc(*SHAPE, (3, 7, 7), 0.125, B.STRATA_BF16)
    q = cpu(SHAPE)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_na3d_fwd(desc, q, q, q, None, q)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_na3d_fwd_ex(desc, None, q, q, q, None, q)


def test_backward_rejects_host_tensors():
    desc = B.make_desc(*SHAPE, (3, 7, 7), 0.125, B.STRATA_BF16)
    q = cpu(SHAPE)
    lse = cpu(SHAPE[:-1], torch.float32)
    ws = cpu((1024,), torch.uint8)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_na3d_bwd(desc, q, q, q, None, q, q, lse, q, q, q, ws)


def test_stitch_rope_geometry_reject_host_tensors():
    tiles = cpu((4, 3, 8, 8, 16))
    win = cpu((64,), torch.float32)
    face = cpu((3, 12, 12, 16))
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_tile_blend(tiles, 2, 2, 4, 4, win, face)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_tile_extract(face, 2, 2, 4, 4, tiles)
    x = cpu(SHAPE)
    cs = cpu((1, 16, 16, 32, 2), torch.float32)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_stereorope_apply(x, x, cs)
    i32 = cpu((1,), torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_stereo_coords(i32, i32, i32, 16, 16, 2048, 4, 0.0, cpu((1, 16, 16, 2), torch.float32))
    with pytest.raises(ValueError, match="GPU tensor"):
        B.strata_na_axis_index(8, 3, *(cpu((8,), torch.int32) for _ in range(3)))


def test_non_tensor_arguments_are_rejected():
    desc = B.make_desc(*SHAPE, (3, 7, 7), 0.125, B.STRATA_BF16)
    with pytest.raises(ValueError, match="torch.Tensor"):
        B.strata_na3d_fwd(desc, 0x1000, 0x1000, 0x1000, None, 0x1000)

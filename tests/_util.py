"""Helpers shared by the GPU tests: moving seeded inputs to the device and the
parity rules (bf16: max |gpu - oracle| <= 2e-2 * RMS(oracle); f32: <= 1e-5)."""
import numpy as np
import torch

BF16_REL_RMS = 2e-2
F32_ABS = 1e-5
LSE_ABS_BF16 = 2e-2


def dev_tensor(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Seeded host array (bf16 bits as uint16, or float32) -> device tensor."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device)


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def host_rows(t: torch.Tensor, sel, width: int = 0) -> np.ndarray:
    """Rows ``sel`` of a device tensor viewed as [-1, width] (its flat elements
    when width is 0), gathered on the device, as float64 on the host: a sampled
    check of a full-size output moves only the samples."""
    flat = t.reshape(-1, width) if width else t.reshape(-1)
    idx = torch.from_numpy(np.asarray(sel, dtype=np.int64)).to(t.device)
    return host_f64(flat.index_select(0, idx))


def host_bits(t: torch.Tensor) -> np.ndarray:
    """Raw storage of a bf16 / f32 device tensor as a numpy array (bit-exact comparisons)."""
    c = t.detach().contiguous().cpu()
    if c.dtype == torch.bfloat16:
        return c.view(torch.int16).numpy().view(np.uint16)
    return c.numpy()


def bf16_half_ulp(ref: np.ndarray) -> np.ndarray:
    """Half a bf16 ulp at each exact value: the error of storing it in bf16 at all."""
    a = np.abs(ref)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8), 0.0)


def check_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str):
    """bf16: |gpu - oracle| <= 2e-2 RMS(oracle) + the bf16 storage rounding of the
    output (half an ulp of the exact value); f32: |gpu - oracle| <= 1e-5."""
    if not got.size:
        return 0.0
    diff = np.abs(got - ref)
    if dtype == "bf16":
        rms = float(np.sqrt(np.mean(ref * ref)))
        excess = diff - bf16_half_ulp(ref)
        worst = float(np.max(excess))
        assert worst <= BF16_REL_RMS * rms, (
            f"{what}: error beyond bf16 storage rounding {worst:.3e} > {BF16_REL_RMS} * RMS = "
            f"{BF16_REL_RMS * rms:.3e} (max abs err {float(np.max(diff)):.3e})")
        return float(np.max(diff))
    err = float(np.max(diff))
    assert err <= F32_ABS, f"{what}: max abs err {err:.3e} > tol {F32_ABS:.1e}"
    return err

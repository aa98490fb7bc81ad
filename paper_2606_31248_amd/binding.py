"""Thin Python binding of libstrata's C ABI (include/strata.h).

Functions carry the C names and only marshal arguments: torch tensors become
device pointers, the current HIP stream of torch becomes the stream argument,
and a non-OK status becomes a ``StrataError``.  Every computation runs in the
HIP kernels of libstrata.so; there is no fallback of any kind -- if the library
is not built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# STRATA_LIB: another build of the same sources (the sanitizer run of the host tests)
LIB_PATH = os.environ.get("STRATA_LIB") or os.path.join(_HERE, "libstrata.so")

STRATA_OK, STRATA_ERR_INVALID_ARG, STRATA_ERR_UNSUPPORTED, STRATA_ERR_WORKSPACE, STRATA_ERR_HIP = range(5)
STRATA_F32, STRATA_BF16 = 0, 1

# Every entry point declared in include/strata.h.
EXPORTS = (
    "strata_stereo_coords", "strata_stereorope_phases", "strata_stereorope_apply",
    "strata_na3d_fwd", "strata_na3d_bwd_workspace_size", "strata_na3d_bwd",
    "strata_na3d_fwd_ex", "strata_na3d_bwd_ex_workspace_size", "strata_na3d_bwd_ex",
    "strata_tile_blend", "strata_tile_extract", "strata_na_axis_index", "strata_wind_tile_frame", "strata_kbd_window",
    "strata_duo_pad", "strata_duo_plan_bytes", "strata_duo_plan", "strata_duo_pad_planned",
    "strata_duo_pad_vjp", "strata_na3d_fwd_stitch", "strata_tile_blend_overlap", "strata_na3d_bwd_noalloc",
    "strata_status_string", "strata_last_error",
)


class StrataError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class NA3DDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("heads", ctypes.c_int32), ("Z", ctypes.c_int32),
                ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("kz", ctypes.c_int32), ("ky", ctypes.c_int32), ("kx", ctypes.c_int32),
                ("scale", ctypes.c_float), ("dtype", ctypes.c_int)]


class NA3DOpts(ctypes.Structure):
    _fields_ = [("qk_norm", ctypes.c_int32), ("eps", ctypes.c_float), ("gate", ctypes.c_void_p),
                ("gate_dim", ctypes.c_int32)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libstrata.so (built by ``python -m paper_2606_31248_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libstrata.so not found at {path}: build it with "
                           "`python -m paper_2606_31248_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(path)
    P, i32, st = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int
    D = ctypes.POINTER(NA3DDesc)
    sig = {
        "strata_stereo_coords": [P, P, P, i32, i32, i32, i32, i32, ctypes.c_double, P, P],
        "strata_stereorope_phases": [P, i32, i32, i32, i32, ctypes.c_double, P, P],
        "strata_stereorope_apply": [P, P, P, i32, i32, i32, i32, i32, i32, st, i32, P],
        "strata_na3d_fwd": [D, P, P, P, P, P, P, P],
        "strata_na3d_bwd": [D, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
        "strata_na3d_bwd_noalloc": [D, P, P, P, P, P, P, P, P, P, P, P],
        "strata_tile_blend": [P, i32, i32, i32, i32, i32, i32, i32, i32, P, P, i32, i32, st, P],
        "strata_tile_blend_overlap": [P, i32, i32, i32, i32, i32, i32, i32, i32, P, P, i32, i32, st, P],
        "strata_tile_extract": [P, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, P, st, P],
        "strata_na_axis_index": [i32, i32, P, P, P, P],
        "strata_wind_tile_frame": [P, i32, i32, i32, i32, i32, i32, i32, i32, i32, P, st, P],
        "strata_kbd_window": [i32, i32, i32, ctypes.c_double, P, P],
        "strata_duo_pad": [P, i32, i32, i32, i32, P, st, P],
        "strata_duo_plan": [i32, i32, P, ctypes.c_size_t, P],
        "strata_duo_pad_planned": [P, i32, i32, i32, i32, P, ctypes.c_size_t, P, st, P],
        "strata_duo_pad_vjp": [P, i32, i32, i32, i32, P, ctypes.c_size_t, P, st, P],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = st
    O = ctypes.POINTER(NA3DOpts)
    for name, args in {
        "strata_na3d_fwd_ex": [D, O, P, P, P, P, P, P, P],
        "strata_na3d_fwd_stitch": [D, O, P, P, P, P, P, P, i32, i32, i32, i32, P, P, i32, i32, P],
        "strata_na3d_bwd_ex": [D, O, P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
    }.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = st
    L.strata_na3d_bwd_workspace_size.argtypes = [D]
    L.strata_na3d_bwd_workspace_size.restype = ctypes.c_size_t
    L.strata_na3d_bwd_ex_workspace_size.argtypes = [D, O]
    L.strata_na3d_bwd_ex_workspace_size.restype = ctypes.c_size_t
    L.strata_duo_plan_bytes.argtypes = [i32, i32]
    L.strata_duo_plan_bytes.restype = ctypes.c_size_t
    L.strata_status_string.argtypes = [st]
    L.strata_status_string.restype = ctypes.c_char_p
    L.strata_last_error.argtypes = []
    L.strata_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libstrata must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _need(name: str, t, shape=None, dtype=None, device=None, numel=None, optional: bool = False):
    """Check one tensor argument before its pointer crosses the ABI (which sees no
    sizes): a contiguous GPU tensor, on `device`, of `dtype`, of exactly `shape`
    (or at least `numel` elements).  Raises ValueError on any mismatch."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name}: a tensor is required")
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a GPU tensor (got device {t.device})")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: on {t.device}, the other arguments are on {device}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(int(x) for x in shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(int(x) for x in shape)}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, at least {numel} needed")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")


def _torch_dtype(code: int):
    if code == STRATA_BF16:
        return torch.bfloat16
    if code == STRATA_F32:
        return torch.float32
    raise ValueError(f"unknown strata dtype {code}")


def _desc_shape(desc: "NA3DDesc"):
    return (desc.B, desc.heads, desc.Z, desc.H, desc.W, desc.head_dim)


def _check_na_tensors(desc: "NA3DDesc", tensors: dict, cs=None, lse=None, lse_required=False, opts=None,
                      dgate=None):
    """q, k, v, out, dout, dq, dk, dv of the problem's shape and dtype on one GPU;
    cs [B, H, W, head_dim/2, 2] and lse [B, heads, Z, H, W] float32; a gate of
    the problem's dtype, [B, heads, Z, H, W] or the full shape, and dgate alike."""
    shape = _desc_shape(desc)
    dt = _torch_dtype(desc.dtype)
    first = next(iter(tensors.values()))
    _need("q", first, shape, dt)
    dev = first.device
    for name, t in tensors.items():
        _need(name, t, shape, dt, dev)
    _need("cs", cs, (desc.B, desc.H, desc.W, desc.head_dim // 2, 2), torch.float32, dev, optional=True)
    _need("lse", lse, shape[:-1], torch.float32, dev, optional=not lse_required)
    gate = getattr(opts, "_keep", None) if opts is not None else None
    if gate is not None:
        if tuple(gate.shape) not in (shape[:-1], shape):
            raise ValueError(f"gate: shape {tuple(gate.shape)}, expected {shape[:-1]} or {shape}")
        _need("gate", gate, tuple(gate.shape), dt, dev)
        if dgate is not None or lse_required:
            _need("dgate", dgate, tuple(gate.shape), dt, dev)
    return dev


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return STRATA_BF16
    if t.dtype == torch.float32:
        return STRATA_F32
    raise ValueError(f"unsupported tensor dtype {t.dtype}")


def _check(status: int):
    if status != STRATA_OK:
        L = load()
        raise StrataError(status, L.strata_last_error().decode())


def make_desc(B, heads, Z, H, W, head_dim, window, scale, dtype: int) -> NA3DDesc:
    kz, ky, kx = window
    return NA3DDesc(B, heads, Z, H, W, head_dim, kz, ky, kx, float(scale), int(dtype))


def desc_for(q: torch.Tensor, window, scale) -> NA3DDesc:
    B, heads, Z, H, W, d = q.shape
    return make_desc(B, heads, Z, H, W, d, window, scale, _dtype(q))


# ---- entry points -------------------------------------------------------------

def strata_stereo_coords(tile_face, tile_oy, tile_ox, H, W, face_cells, patch, l_scale, coords,
                         stream=None):
    B = tile_face.shape[0]
    _need("tile_face", tile_face, (B,), torch.int32)
    dev = tile_face.device
    _need("tile_oy", tile_oy, (B,), torch.int32, dev)
    _need("tile_ox", tile_ox, (B,), torch.int32, dev)
    _need("coords", coords, (B, H, W, 2), torch.float32, dev)
    _check(load().strata_stereo_coords(_ptr(tile_face), _ptr(tile_oy), _ptr(tile_ox), B, H, W,
                                       face_cells, patch, float(l_scale), _ptr(coords),
                                       _stream(stream)))


def strata_stereorope_phases(coords, head_dim, base, cs, stream=None):
    B, H, W, _ = coords.shape
    _need("coords", coords, (B, H, W, 2), torch.float32)
    _need("cs", cs, (B, H, W, head_dim // 2, 2), torch.float32, coords.device)
    _check(load().strata_stereorope_phases(_ptr(coords), B, H, W, head_dim, float(base), _ptr(cs),
                                           _stream(stream)))


def strata_stereorope_apply(x, y, cs, transpose=False, stream=None):
    B, heads, Z, H, W, d = x.shape
    _need("x", x, x.shape)
    _need("y", y, x.shape, x.dtype, x.device)
    _need("cs", cs, (B, H, W, d // 2, 2), torch.float32, x.device)
    _check(load().strata_stereorope_apply(_ptr(x), _ptr(y), _ptr(cs), B, heads, Z, H, W, d,
                                          _dtype(x), int(bool(transpose)), _stream(stream)))


def strata_na3d_fwd(desc: NA3DDesc, q, k, v, cs, out, lse=None, stream=None):
    _check_na_tensors(desc, dict(q=q, k=k, v=v, out=out), cs, lse)
    _check(load().strata_na3d_fwd(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(cs), _ptr(out),
                                  _ptr(lse), _stream(stream)))


def strata_na3d_bwd_workspace_size(desc: NA3DDesc) -> int:
    return int(load().strata_na3d_bwd_workspace_size(ctypes.byref(desc)))


def strata_na3d_bwd(desc: NA3DDesc, q, k, v, cs, out, dout, lse, dq, dk, dv, workspace,
                    stream=None):
    dev = _check_na_tensors(desc, dict(q=q, k=k, v=v, out=out, dout=dout, dq=dq, dk=dk, dv=dv), cs, lse,
                            lse_required=True)
    _need("workspace", workspace, device=dev, optional=True)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().strata_na3d_bwd(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(cs), _ptr(out),
                                  _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
                                  _ptr(workspace), nbytes, _stream(stream)))


def strata_na3d_bwd_noalloc(desc: NA3DDesc, q, k, v, cs, out, dout, lse, dq, dk, dv, stream=None):
    """strata_na3d_bwd without a workspace (D in the library's static device array)."""
    _check_na_tensors(desc, dict(q=q, k=k, v=v, out=out, dout=dout, dq=dq, dk=dk, dv=dv), cs, lse,
                      lse_required=True)
    _check(load().strata_na3d_bwd_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(cs), _ptr(out),
                                          _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv), _stream(stream)))


def make_opts(qk_norm: bool = False, eps: float = 1e-6, gate: Optional[torch.Tensor] = None) -> NA3DOpts:
    """Options of the attention block: QK RMSNorm and the sigmoid output gate.

    gate: logits of the activations' dtype, [B, heads, Z, H, W] (one per token
    and head) or [B, heads, Z, H, W, head_dim] (one per channel)."""
    o = NA3DOpts(int(bool(qk_norm)), float(eps), None, 0)
    if gate is not None:
        o.gate = _ptr(gate)
        o.gate_dim = 1 if gate.dim() == 5 else int(gate.shape[-1])
    o._keep = gate  # the tensor must outlive the call
    return o


def _opts_ref(opts: Optional[NA3DOpts]):
    return None if opts is None else ctypes.byref(opts)


def strata_na3d_fwd_ex(desc: NA3DDesc, opts: Optional[NA3DOpts], q, k, v, cs, out, lse=None, stream=None):
    _check_na_tensors(desc, dict(q=q, k=k, v=v, out=out), cs, lse, opts=opts)
    _check(load().strata_na3d_fwd_ex(ctypes.byref(desc), _opts_ref(opts), _ptr(q), _ptr(k), _ptr(v), _ptr(cs),
                                     _ptr(out), _ptr(lse), _stream(stream)))


def strata_na3d_bwd_ex_workspace_size(desc: NA3DDesc, opts: Optional[NA3DOpts]) -> int:
    return int(load().strata_na3d_bwd_ex_workspace_size(ctypes.byref(desc), _opts_ref(opts)))


def strata_na3d_bwd_ex(desc: NA3DDesc, opts: Optional[NA3DOpts], q, k, v, cs, out, dout, lse, dq, dk, dv,
                       dgate, workspace, stream=None):
    dev = _check_na_tensors(desc, dict(q=q, k=k, v=v, out=out, dout=dout, dq=dq, dk=dk, dv=dv), cs, lse,
                            lse_required=True, opts=opts, dgate=dgate)
    _need("workspace", workspace, device=dev, optional=True)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().strata_na3d_bwd_ex(ctypes.byref(desc), _opts_ref(opts), _ptr(q), _ptr(k), _ptr(v), _ptr(cs),
                                     _ptr(out), _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
                                     _ptr(dgate), _ptr(workspace), nbytes, _stream(stream)))


def _check_tiling(tiles, nty, ntx, window, out):
    """tiles [nty*ntx, P, Ht, Wt, C], window float32 of Ht*Wt, out [P, Hf, Wf, C] of the tiles' dtype."""
    T, P, Ht, Wt, C = tiles.shape
    _need("tiles", tiles, (nty * ntx, P, Ht, Wt, C))
    _need("window", window, (Ht * Wt,), torch.float32, tiles.device)
    _need("out", out, (P, out.shape[1], out.shape[2], C), tiles.dtype, tiles.device)


def strata_tile_blend(tiles, nty, ntx, stride_y, stride_x, window, out, stream=None):
    T, P, Ht, Wt, C = tiles.shape
    _, Hf, Wf, _ = out.shape
    _check_tiling(tiles, nty, ntx, window, out)
    _check(load().strata_tile_blend(_ptr(tiles), nty, ntx, P, Ht, Wt, C, stride_y, stride_x,
                                    _ptr(window), _ptr(out), Hf, Wf, _dtype(tiles), _stream(stream)))


def strata_tile_blend_overlap(tiles, nty, ntx, stride_y, stride_x, window, out, stream=None):
    """Stitch of the face cells that two or more tiles cover (the second call of the fused face step)."""
    T, P, Ht, Wt, C = tiles.shape
    _, Hf, Wf, _ = out.shape
    _check_tiling(tiles, nty, ntx, window, out)
    _check(load().strata_tile_blend_overlap(_ptr(tiles), nty, ntx, P, Ht, Wt, C, stride_y, stride_x,
                                            _ptr(window), _ptr(out), Hf, Wf, _dtype(tiles), _stream(stream)))


def strata_na3d_fwd_stitch(desc: NA3DDesc, opts: Optional[NA3DOpts], q, k, v, cs, tiles, lse, nty, ntx,
                           stride_y, stride_x, window, face, stream=None):
    """Forward of the nty x ntx tiles of one face, cells covered by one tile stored into face [heads*Z, Hf, Wf, d]."""
    _, Hf, Wf, _ = face.shape
    dev = _check_na_tensors(desc, dict(q=q, k=k, v=v, tiles=tiles), cs, lse, opts=opts)
    _need("window", window, (desc.H * desc.W,), torch.float32, dev)
    _need("face", face, (desc.heads * desc.Z, Hf, Wf, desc.head_dim), q.dtype, dev)
    _check(load().strata_na3d_fwd_stitch(ctypes.byref(desc), _opts_ref(opts), _ptr(q), _ptr(k), _ptr(v), _ptr(cs),
                                         _ptr(tiles), _ptr(lse), nty, ntx, stride_y, stride_x, _ptr(window),
                                         _ptr(face), Hf, Wf, _stream(stream)))


def strata_tile_extract(face, nty, ntx, stride_y, stride_x, tiles, stream=None):
    P, Hf, Wf, C = face.shape
    _, _, Ht, Wt, _ = tiles.shape
    _need("face", face, face.shape)
    _need("tiles", tiles, (nty * ntx, P, Ht, Wt, C), face.dtype, face.device)
    _check(load().strata_tile_extract(_ptr(face), nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf,
                                      _ptr(tiles), _dtype(face), _stream(stream)))


def strata_na_axis_index(L, k, starts, qlo, qhi, stream=None):
    _need("starts", starts, (L,), torch.int32)
    _need("qlo", qlo, (L,), torch.int32, starts.device)
    _need("qhi", qhi, (L,), torch.int32, starts.device)
    _check(load().strata_na_axis_index(L, k, _ptr(starts), _ptr(qlo), _ptr(qhi), _stream(stream)))


def strata_wind_tile_frame(field, face, nty, ntx, stride_y, stride_x, tiles, stream=None):
    """field: [P, n, n, 2] (U, V per cell of one face); tiles: [nty*ntx, P, Ht, Wt, 2]."""
    P, n, _, _ = field.shape
    _, _, Ht, Wt, _ = tiles.shape
    _need("field", field, (P, n, n, 2))
    _need("tiles", tiles, (nty * ntx, P, Ht, Wt, 2), field.dtype, field.device)
    _check(load().strata_wind_tile_frame(_ptr(field), int(face), n, nty, ntx, P, Ht, Wt, stride_y, stride_x,
                                         _ptr(tiles), _dtype(field), _stream(stream)))


def strata_kbd_window(Ht, Wt, overlap, beta, window, stream=None):
    """window: float32 [Ht * Wt] on the device."""
    _need("window", window, (Ht * Wt,), torch.float32)
    _check(load().strata_kbd_window(Ht, Wt, overlap, float(beta), _ptr(window), _stream(stream)))


def strata_duo_pad(faces, halo, padded, stream=None):
    """faces: [6, P, n, n, C]; padded: [6, P, n + 2 halo, n + 2 halo, C]."""
    _, P, n, _, C = faces.shape
    _need("faces", faces, (6, P, n, n, C))
    _need("padded", padded, (6, P, n + 2 * halo, n + 2 * halo, C), faces.dtype, faces.device)
    _check(load().strata_duo_pad(_ptr(faces), P, n, C, int(halo), _ptr(padded), _dtype(faces), _stream(stream)))


def strata_duo_plan_bytes(n, halo):
    """Bytes of the padding plan for (n, halo); 0 if the pair is invalid."""
    return int(load().strata_duo_plan_bytes(int(n), int(halo)))


def strata_duo_plan(n, halo, plan, stream=None):
    """plan: a device buffer (e.g. uint8) of at least strata_duo_plan_bytes(n, halo) bytes."""
    _need("plan", plan)
    _check(load().strata_duo_plan(int(n), int(halo), _ptr(plan), plan.numel() * plan.element_size(),
                                  _stream(stream)))


def strata_duo_pad_planned(faces, halo, plan, padded, stream=None):
    """As strata_duo_pad, with the neighbours and weights read from a plan."""
    _, P, n, _, C = faces.shape
    _need("faces", faces, (6, P, n, n, C))
    _need("plan", plan, device=faces.device)
    _need("padded", padded, (6, P, n + 2 * halo, n + 2 * halo, C), faces.dtype, faces.device)
    _check(load().strata_duo_pad_planned(_ptr(faces), P, n, C, int(halo), _ptr(plan),
                                         plan.numel() * plan.element_size(), _ptr(padded), _dtype(faces),
                                         _stream(stream)))


def strata_duo_pad_vjp(grad_padded, halo, plan, grad_faces, stream=None):
    """grad_faces = P^T grad_padded: grad_padded [6, P, n + 2 halo, n + 2 halo, C] ->
    grad_faces [6, P, n, n, C], through a plan built for (n, halo)."""
    _, P, m, _, C = grad_padded.shape
    n = m - 2 * int(halo)
    _need("grad_padded", grad_padded, (6, P, m, m, C))
    _need("plan", plan, device=grad_padded.device)
    _need("grad_faces", grad_faces, (6, P, n, n, C), grad_padded.dtype, grad_padded.device)
    _check(load().strata_duo_pad_vjp(_ptr(grad_padded), P, n, C, int(halo), _ptr(plan),
                                     plan.numel() * plan.element_size(), _ptr(grad_faces), _dtype(grad_padded),
                                     _stream(stream)))

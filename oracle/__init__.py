"""CPU oracle of the STRATA hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never calls it and shares no code with it.

* ``geometry``: Eq. 1 stereographic tile coordinates on the equiangular cubed
  sphere (numpy, float64).
* ``strata_oracle.c`` (built into ``liboracle.so`` with gcc, OpenMP, no
  fast-math, no FP contraction): window indexing, StereoRoPE, neighbourhood
  attention forward/backward (optionally with QK RMSNorm and the sigmoid
  output gate), tile blend and extraction, in float64 (the blend follows its
  fixed operation order).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

from . import geometry  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "strata_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# STRATA_ORACLE_LIB: load another build of the same source instead (the sanitizer
# run of the host tests builds one); build() always writes _LIB
_LOAD = os.environ.get("STRATA_ORACLE_LIB") or _LIB
_lib = None

ROPE_BASE = 100.0


def build(force: bool = False) -> str:
    """Compile the oracle library with gcc (plain C, OpenMP, IEEE semantics)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if _LOAD == _LIB and not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LOAD)
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        P = ctypes.c_void_p
        L.oracle_axis_index.argtypes = [i32, i32, P, P, P]
        L.oracle_rope_phases.argtypes = [P, i32, i32, i32, i32, f64, P]
        L.oracle_rope_apply.argtypes = [P, P, i32, i32, i32, i32, i32, i32, f64, i32, P]
        L.oracle_na3d_fwd.argtypes = [P, P, P, P, f64] + [i32] * 9 + [f64, i64, P, P, P]
        L.oracle_na3d_bwd.argtypes = [P, P, P, P, f64] + [i32] * 9 + [f64, P, i64, P, i64, P, P, P, P]
        L.oracle_na3d_fwd_ex.argtypes = [P, P, P, P, f64] + [i32] * 9 + [f64, i32, f64, P, i32, i64, P, P, P]
        L.oracle_na3d_bwd_ex.argtypes = ([P, P, P, P, f64] + [i32] * 9 + [f64, i32, f64, P, i32, P, i64, P, i64, P]
                                         + [P, P, P, P])
        L.oracle_tile_blend.argtypes = [P, i32, i32, i32, i32, i32, i32, i32, i32, P, P, i32, i32, i32]
        L.oracle_tile_extract.argtypes = [P, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, P, i32]
        L.oracle_set_num_threads.argtypes = [i32]
        L.oracle_set_num_threads.restype = None
        for f in ("oracle_axis_index", "oracle_rope_phases", "oracle_rope_apply", "oracle_na3d_fwd", "oracle_na3d_bwd",
                  "oracle_na3d_fwd_ex", "oracle_na3d_bwd_ex", "oracle_tile_blend", "oracle_tile_extract", "oracle_num_threads"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's OpenMP loops from now on."""
    lib().oracle_set_num_threads(int(n))


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored inputs (bf16 bit patterns or float32)."""
    if dtype == "bf16":
        u = np.ascontiguousarray(a, dtype=np.uint16).astype(np.uint32) << 16
        return u.view(np.float32).astype(np.float64)
    return np.ascontiguousarray(a, dtype=np.float32).astype(np.float64)


def axis_index(L: int, k: int):
    starts = np.zeros(L, np.int32)
    qlo = np.zeros(L, np.int32)
    qhi = np.zeros(L, np.int32)
    rc = lib().oracle_axis_index(L, k, _p(starts), _p(qlo), _p(qhi))
    if rc:
        raise ValueError("invalid axis window (L=%d, k=%d)" % (L, k))
    return starts, qlo, qhi


def rope_phases(coords: np.ndarray, d: int, base: float = ROPE_BASE) -> np.ndarray:
    """(cos, sin) per (b, y, x, pair): float64 [B, H, W, d/2, 2]."""
    c = np.ascontiguousarray(coords, dtype=np.float32)
    B, H, W, _ = c.shape
    out = np.empty((B, H, W, d // 2, 2), np.float64)
    rc = lib().oracle_rope_phases(_p(c), B, H, W, d, base, _p(out))
    if rc:
        raise ValueError("oracle_rope_phases failed (%d)" % rc)
    return out


def rope_apply(x: np.ndarray, coords: np.ndarray, transpose: bool = False,
               base: float = ROPE_BASE) -> np.ndarray:
    """x: [B, heads, Z, H, W, d] float64; coords: [B, H, W, 2] float32."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    c = np.ascontiguousarray(coords, dtype=np.float32)
    B, heads, Z, H, W, d = x.shape
    assert c.shape == (B, H, W, 2)
    y = np.empty_like(x)
    rc = lib().oracle_rope_apply(_p(x), _p(c), B, heads, Z, H, W, d, base, int(transpose), _p(y))
    if rc:
        raise ValueError("oracle_rope_apply failed (%d)" % rc)
    return y


def _gate_arg(gate, shape):
    """gate logits as float64: [B, heads, Z, H, W] (gate_dim 1) or the full shape (gate_dim d)."""
    if gate is None:
        return None, 0
    g = np.ascontiguousarray(gate, dtype=np.float64)
    if g.shape == tuple(shape[:-1]):
        return g, 1
    if g.shape == tuple(shape):
        return g, shape[-1]
    raise ValueError("gate must have shape %s or %s" % (shape[:-1], shape))


def na3d_fwd(q, k, v, window, scale, coords=None, sel=None, base: float = ROPE_BASE,
             qk_norm: bool = False, eps: float = 1e-6, gate=None):
    """Neighbourhood attention forward in float64.

    q, k, v: [B, heads, Z, H, W, d] float64.  window: (kz, ky, kx).
    sel: optional flat query indices into [B, heads, Z, H, W].
    qk_norm: RMS-normalise q and k (no learnable scale) with ``eps``.
    gate: sigmoid-gate logits, [B, heads, Z, H, W] or [B, heads, Z, H, W, d].
    Returns (out, lse): out [n, d] (or full shape when sel is None), lse [n]."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    B, heads, Z, H, W, d = q.shape
    kz, ky, kx = window
    c = None if coords is None else np.ascontiguousarray(coords, dtype=np.float32)
    if sel is None:
        n = B * heads * Z * H * W
        s = None
    else:
        s = np.ascontiguousarray(sel, dtype=np.int64)
        n = s.shape[0]
    out = np.empty((n, d), np.float64)
    lse = np.empty(n, np.float64)
    g, gdim = _gate_arg(gate, q.shape)
    if qk_norm or g is not None:
        rc = lib().oracle_na3d_fwd_ex(_p(q), _p(k), _p(v), _p(c), base, B, heads, Z, H, W, d, kz, ky, kx,
                                      float(scale), int(qk_norm), float(eps), _p(g), gdim, n, _p(s),
                                      _p(out), _p(lse))
    else:
        rc = lib().oracle_na3d_fwd(_p(q), _p(k), _p(v), _p(c), base, B, heads, Z, H, W, d, kz, ky, kx,
                                   float(scale), n, _p(s), _p(out), _p(lse))
    if rc:
        raise ValueError("oracle_na3d_fwd failed (%d)" % rc)
    if sel is None:
        return out.reshape(B, heads, Z, H, W, d), lse.reshape(B, heads, Z, H, W)
    return out, lse


def na3d_bwd(q, k, v, dout, window, scale, coords=None, selq=None, selk=None,
             base: float = ROPE_BASE, qk_norm: bool = False, eps: float = 1e-6, gate=None):
    """Neighbourhood attention backward in float64: (dq, dk, dv), plus dgate when
    ``gate`` is given (options as in ``na3d_fwd``; dout is the gradient of the
    gated output).

    dq and dgate rows follow selq, dk/dv rows follow selk (flat indices; None =
    all, full shape)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    g = np.ascontiguousarray(dout, dtype=np.float64)
    B, heads, Z, H, W, d = q.shape
    kz, ky, kx = window
    c = None if coords is None else np.ascontiguousarray(coords, dtype=np.float32)
    nall = B * heads * Z * H * W
    sq = None if selq is None else np.ascontiguousarray(selq, dtype=np.int64)
    sk = None if selk is None else np.ascontiguousarray(selk, dtype=np.int64)
    nq = nall if sq is None else sq.shape[0]
    nk = nall if sk is None else sk.shape[0]
    dq = np.empty((nq, d), np.float64)
    dk = np.empty((nk, d), np.float64)
    dv = np.empty((nk, d), np.float64)
    gt, gdim = _gate_arg(gate, q.shape)
    dg = None
    if qk_norm or gt is not None:
        if gt is not None:
            dg = np.empty((nq,) if gdim == 1 else (nq, d), np.float64)
        rc = lib().oracle_na3d_bwd_ex(_p(q), _p(k), _p(v), _p(c), base, B, heads, Z, H, W, d, kz, ky, kx,
                                      float(scale), int(qk_norm), float(eps), _p(gt), gdim, _p(g), nq,
                                      _p(sq), nk, _p(sk), _p(dq), _p(dk), _p(dv), _p(dg))
    else:
        rc = lib().oracle_na3d_bwd(_p(q), _p(k), _p(v), _p(c), base, B, heads, Z, H, W, d, kz, ky, kx,
                                   float(scale), _p(g), nq, _p(sq), nk, _p(sk), _p(dq), _p(dk), _p(dv))
    if rc:
        raise ValueError("oracle_na3d_bwd failed (%d)" % rc)
    full = (B, heads, Z, H, W, d)
    if sq is None:
        dq = dq.reshape(full)
        if dg is not None:
            dg = dg.reshape(gt.shape)
    if sk is None:
        dk = dk.reshape(full)
        dv = dv.reshape(full)
    if gt is not None:
        return dq, dk, dv, dg
    return dq, dk, dv


def tile_blend(tiles: np.ndarray, nty: int, ntx: int, stride_y: int, stride_x: int,
               window: np.ndarray, Hf: int, Wf: int, dtype: str) -> np.ndarray:
    """tiles: [nty*ntx, P, Ht, Wt, C] (uint16 bf16 bits or float32); window [Ht*Wt] float32."""
    t = np.ascontiguousarray(tiles)
    T, P, Ht, Wt, C = t.shape
    assert T == nty * ntx
    w = np.ascontiguousarray(window, dtype=np.float32)
    is_bf16 = dtype == "bf16"
    out = np.empty((P, Hf, Wf, C), np.uint16 if is_bf16 else np.float32)
    rc = lib().oracle_tile_blend(_p(t), nty, ntx, P, Ht, Wt, C, stride_y, stride_x, _p(w), _p(out),
                                 Hf, Wf, int(is_bf16))
    if rc:
        raise ValueError("oracle_tile_blend: invalid arguments")
    return out


def tile_extract(face: np.ndarray, nty: int, ntx: int, Ht: int, Wt: int, stride_y: int,
                 stride_x: int) -> np.ndarray:
    """face: [P, Hf, Wf, C] -> tiles [nty*ntx, P, Ht, Wt, C] (exact copy)."""
    f = np.ascontiguousarray(face)
    P, Hf, Wf, C = f.shape
    tiles = np.empty((nty * ntx, P, Ht, Wt, C), f.dtype)
    rc = lib().oracle_tile_extract(_p(f), nty, ntx, P, Ht, Wt, C, stride_y, stride_x, Hf, Wf,
                                   _p(tiles), f.dtype.itemsize)
    if rc:
        raise ValueError("oracle_tile_extract: invalid arguments")
    return tiles

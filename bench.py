"""Throughput of one face rollout step of the STRATA hot path on one MI355X.

Workload (synthetic, seeded): one cube face of 2048^2 cells at 4 x 4 patches =
512^2 horizontal x 8 vertical tokens, cut into 64 x 64-token tiles overlapping
by 8 tokens (stride 56, 9 x 9 = 81 tiles); 16 heads of head_dim 64; Q/K/V iid
N(0,1) in bf16.  One step =
  stereographic coordinates of every tile token (Eq. 1) -> StereoRoPE phases ->
  3x7x7 neighbourhood attention forward with the rotation fused into the Q/K
  loads -> linear-ramp tile stitch of the 81 tile outputs back to the face.
Inputs are resident in HBM before timing starts.

Prints one JSON line.  ``value`` is the neighbourhood-attention forward's
algorithmic TFLOP/s over the whole step (4 B h N K d FLOPs per step divided by
the step time); the dominant kernel's roofline and a timed CPU-oracle sample
are reported beside it.  Two side measurements follow the step (not part of
``value``): the training-tile attention (16 tiles x 16 heads x 8x64x64, 5x9x9,
forward and backward with StereoRoPE) and the standalone StereoRoPE rotation
of its Q and K.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import re
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "NA3D fwd TFLOP/s + tokens/s at 1 MI355X; % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0        # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0            # MI355X HBM3E
PMC_FILE = os.path.join(ROOT, "profiles", "na3d_fwd_face_rollout_pmc.json")
STATS_FILE = os.path.join(ROOT, "profiles", "face_rollout_step_kernel_stats.txt")
SQ_FILE = os.path.join(ROOT, "profiles", "na3d_fwd_face_rollout_sq_counters.json")
# the sources of the kernel that strata_na3d_fwd runs at the face-rollout shape
KERNEL_SOURCES = ["paper_2606_31248_amd/csrc/na3d_fwd_zs.hip", "paper_2606_31248_amd/csrc/mfma_util.h",
                  "paper_2606_31248_amd/csrc/common.h"]
# the sources of the stitch kernels (the overlap stitch of the face step)
BLEND_SOURCES = ["paper_2606_31248_amd/csrc/blend.hip", "paper_2606_31248_amd/csrc/common.h"]
# the face step: the forward with the stitch of single-cover cells fused into its
# store, then the stitch of the overlap cells
FWD_KERNEL = "na3d_fwd_zs_kernel<8, false, false, true>"
BLEND_KERNEL = "tile_blend_overlap_bf16_kernel"
COPY_KERNEL = "copyBuffer"
CALIB_BYTES = 1 << 30


def kernel_source_hash(sources=None) -> str:
    h = hashlib.sha256()
    for p in sources or KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(per_launch_alg_bytes: float):
    """HBM bytes per launch from the committed rocprofv3 counter runs, if they are
    still for the current kernel source; else None."""
    try:
        with open(PMC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None, None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None, None
    return rec.get("hbm_bytes_per_launch"), rec


def _pmc_rows(run_dir: str):
    """(kernel name, counter, value) of every dispatch in a rocprofv3 --pmc csv run."""
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                rows.append((r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"])))
    return rows


def summarize_pmc(fetch_dir: str, write_dir: str, commands) -> dict:
    """HBM traffic per launch of the forward and the blend from a FETCH_SIZE run and
    a WRITE_SIZE run of ``bench.py --calib-copy``: each counter (KiB per dispatch)
    is scaled by the factor that makes the 1 GiB device copy read its true size."""
    def per_kernel(run_dir, counter):
        acc = {}
        for k, c, v in _pmc_rows(run_dir):
            if c.startswith(counter):
                acc.setdefault(k, []).append(v)
        return acc

    fe, wr = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")

    def pick(acc, key, how=np.median):
        vals = [v for k, vs in acc.items() if key in k for v in vs]
        if not vals:
            raise SystemExit(f"no dispatch of {key} in the counter run")
        return float(how(vals))

    # the calibration copy is the largest copy dispatch (the others move a few KiB)
    cf, cw = pick(fe, COPY_KERNEL, np.max), pick(wr, COPY_KERNEL, np.max)
    ff, fw = CALIB_BYTES / (cf * 1024), CALIB_BYTES / (cw * 1024)
    wl_alg = 4.0 * 81 * 16 * 8 * 64 * 64 * 64 * 2
    blend_alg = overlap_stitch_bytes(9, 9, 64, 64, 56, 56, 128, 64)
    fwd_f, fwd_w = pick(fe, FWD_KERNEL), pick(wr, FWD_KERNEL)
    bl_f, bl_w = pick(fe, BLEND_KERNEL), pick(wr, BLEND_KERNEL)
    return {
        "kernel": f"strata_na3d_fwd_stitch ({FWD_KERNEL}: no options)",
        "workload": "face_rollout_81x16x8x64x64_d64_w3x7x7",
        "kernel_source_hash": kernel_source_hash(),
        "fetch_kb_per_launch": fwd_f,
        "write_kb_per_launch": fwd_w,
        "copy_calibration": {"bytes": CALIB_BYTES, "fetch_kb": cf, "write_kb": cw,
                             "fetch_factor": ff, "write_factor": fw},
        "hbm_bytes_per_launch": fwd_f * 1024 * ff + fwd_w * 1024 * fw,
        "alg_bytes_per_launch": wl_alg,
        "blend": {"kernel": f"strata_tile_blend_overlap ({BLEND_KERNEL})",
                  "source_hash": kernel_source_hash(BLEND_SOURCES), "fetch_kb": bl_f, "write_kb": bl_w, "hbm_bytes_per_launch": bl_f * 1024 * ff + bl_w * 1024 * fw,
                  "alg_bytes_per_launch": blend_alg},
        "commands": list(commands),
        "note": "Traffic = FETCH_SIZE * fetch_factor + WRITE_SIZE * write_factor, per dispatch; the factors "
                "make the counters of one 1 GiB device copy read 1 GiB.",
    }


def summarize_sq(run_dir: str, commands) -> dict:
    """Instruction mix of the face forward from one rocprofv3 --pmc run of SQ
    counters (per dispatch, median over dispatches): every MFMA of the kernel is a
    16x16x32 one (2*16*16*32 FLOP), so the MFMA count gives the issued FLOP and,
    against the algorithmic 4*B*h*N*K*d, the useful fraction (window masking
    over the union key box, the last chunk's padding, the row-sum MFMA)."""
    acc = {}
    for k, c, v in _pmc_rows(run_dir):
        if FWD_KERNEL in k:
            acc.setdefault(c, []).append(v)
    if not acc:
        raise SystemExit(f"no dispatch of {FWD_KERNEL} in the counter run")
    med = {c: float(np.median(v)) for c, v in acc.items()}
    flops_alg = 4.0 * 81 * 16 * 8 * 64 * 64 * 147 * 64
    rec = {"kernel": f"strata_na3d_fwd_stitch ({FWD_KERNEL}: no options)",
           "workload": "face_rollout_81x16x8x64x64_d64_w3x7x7",
           "kernel_source_hash": kernel_source_hash(),
           "counters_per_dispatch": med, "commands": list(commands)}
    mf = next((v for c, v in med.items() if c.startswith("SQ_INSTS_MFMA")), None)
    va = next((v for c, v in med.items() if c.startswith("SQ_INSTS_VALU") and "TRANS" not in c), None)
    tr = next((v for c, v in med.items() if c.startswith("SQ_INSTS_VALU_TRANS_F32")), None)
    if mf:
        rec["issued_mfma_flop"] = mf * 2 * 16 * 16 * 32
        rec["algorithmic_flop"] = flops_alg
        rec["useful_fraction"] = flops_alg / rec["issued_mfma_flop"]
        if va:
            rec["valu_per_mfma"] = (va - mf) / mf  # SQ_INSTS_VALU includes the MFMAs
        if tr:
            rec["exp_per_mfma"] = tr / mf
    return rec


def _short_kernel(name: str) -> str:
    """Kernel name with its template arguments, without namespaces and parameter list."""
    name = re.sub(r"\(.*$", "", name.replace("(anonymous namespace)::", ""))
    return re.sub(r"^void |strata::", "", name)


def summarize_counters(label: str, run_dirs, commands) -> str:
    """Text summary of rocprofv3 --pmc runs: per library kernel, the median over its
    dispatches of every counter collected.  FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch) are also given in bytes, scaled by the factor that makes the 1 GiB
    device copy of the same run (--calib-copy) read its size; with SQ_INSTS_VALU
    (which counts the MFMAs too) and SQ_INSTS_MFMA the VALU instructions per MFMA,
    and the MFMA FLOP issued (every MFMA of these kernels is a 16x16x32 one)."""
    acc = {}
    copy = {}
    for d in run_dirs:
        for k, c, v in _pmc_rows(d):
            if COPY_KERNEL in k:
                copy.setdefault(c, []).append(v)
            elif "strata" in k:
                acc.setdefault(_short_kernel(k), {}).setdefault(c, []).append(v)
    fac = {}
    for c, want in (("FETCH_SIZE", CALIB_BYTES), ("WRITE_SIZE", CALIB_BYTES)):
        vals = [x for cc, xs in copy.items() if cc.startswith(c) for x in xs]
        if vals:
            fac[c] = want / (max(vals) * 1024)
    out = [f"# rocprofv3 --pmc counters, {label}, MI355X (median per dispatch over the run's dispatches)"]
    out += [f"# command: {c}" for c in commands]
    if fac:
        out.append("# copy calibration: " + ", ".join(f"{c} x {f:.4f}" for c, f in fac.items()))
    out.append("")
    for kern, cs in sorted(acc.items()):
        med = {c: float(np.median(v)) for c, v in cs.items()}
        out.append(f"{kern}   ({max(len(v) for v in cs.values())} dispatches)")
        for c in sorted(med):
            out.append(f"    {c:32s} {med[c]:16.6g}")
        mf = next((v for c, v in med.items() if c.startswith("SQ_INSTS_MFMA")), None)
        va = next((v for c, v in med.items() if c.startswith("SQ_INSTS_VALU") and c.split("[")[0] == "SQ_INSTS_VALU"), None)
        if mf:
            out.append(f"    {'= MFMA FLOP issued':32s} {mf * 2 * 16 * 16 * 32:16.6g}")
            if va:
                out.append(f"    {'= VALU per MFMA':32s} {(va - mf) / mf:16.3f}")
        for c, f in fac.items():
            x = next((v for cc, v in med.items() if cc.startswith(c)), None)
            if x is not None:
                out.append(f"    {'= ' + c + ' bytes':32s} {x * 1024 * f:16.6g}")
        out.append("")
    return "\n".join(out)


def overlap_stitch_bytes(nty, ntx, Ht, Wt, sy, sx, P, C, elem=2) -> float:
    """Algorithmic bytes of the overlap-only stitch: every tile value of a cell
    covered by two or more tiles read once, every such face cell written once."""
    Hf, Wf = (nty - 1) * sy + Ht, (ntx - 1) * sx + Wt
    ny = np.array([sum(a * sy <= y < a * sy + Ht for a in range(nty)) for y in range(Hf)])
    nx = np.array([sum(b * sx <= x < b * sx + Wt for b in range(ntx)) for x in range(Wf)])
    cover = ny[:, None] * nx[None, :]
    multi = (ny[:, None] > 1) | (nx[None, :] > 1)
    return float((cover[multi].sum() + multi.sum()) * P * C * elem)


def summarize_stats(stats_csv: str, command: str) -> str:
    """Text summary of a rocprofv3 --kernel-trace --stats run (kernel_stats.csv)."""
    import csv
    with open(stats_csv) as fh:
        rows = list(csv.DictReader(fh))
    out = ["# rocprofv3 kernel trace of bench.py (face rollout step, training-tile side measurement), MI355X",
           f"# command: {command}",
           f"# forward kernel source hash: {kernel_source_hash()}", "",
           f"{'kernel':72s} {'calls':>6s} {'avg_us':>10s} {'min_us':>10s} {'max_us':>10s} {'pct':>6s}"]
    for r in rows:
        # kernel name with its template arguments, without namespaces and parameter list
        name = re.sub(r"\(.*$", "", r["Name"].replace("(anonymous namespace)::", ""))
        name = re.sub(r"^void |strata::", "", name)
        name = name if len(name) <= 72 else name[:69] + "..."
        out.append(f"{name:72s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:10.1f} "
                   f"{float(r['MinNs']) / 1e3:10.1f} {float(r['MaxNs']) / 1e3:10.1f} {float(r['Percentage']):6.2f}")
    return "\n".join(out) + "\n"


def cpu_baseline(wl, tiles_sample: int):
    """Time the CPU oracle on a bounded sample of the same workload: the
    coordinates and neighbourhood-attention forward of ``tiles_sample`` tiles
    (all heads and levels); reported in the metric's unit (algorithmic TFLOP/s)."""
    import oracle
    from oracle import geometry as G
    from paper_2606_31248_amd import inputs as I

    pl = wl.placement()
    sel = np.arange(tiles_sample)
    shape = (tiles_sample,) + wl.shape()[1:]
    q, k, v = (I.gaussian(shape, wl.seed + 100, s, "bf16") for s in (0, 1, 2))
    q, k, v = (oracle.widen(a, "bf16") for a in (q, k, v))
    t0 = time.perf_counter()
    c = G.tile_coords(pl.face[sel], pl.oy[sel], pl.ox[sel], wl.H, wl.W).astype(np.float32)
    oracle.na3d_fwd(q, k, v, (wl.kz, wl.ky, wl.kx), wl.scale, coords=c)
    dt = time.perf_counter() - t0
    flops = 4.0 * tiles_sample * wl.heads * wl.N * wl.K * wl.d
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(dt, 3),
            "sample": f"coordinates + float64 NA3D forward with StereoRoPE of {tiles_sample} of the "
                      f"{wl.B} tiles (all {wl.heads} heads x {wl.N} tokens; blend not included)"}


def cpu_one_thread() -> dict:
    """The oracle on one thread: the whole tiny float32 forward (C1) and one of the
    eight tiles of the bf16 forward with StereoRoPE (C2, scaled to all eight)."""
    import oracle
    from oracle import geometry as G
    from paper_2606_31248_amd import inputs as I
    res = {}
    n0 = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        for key, wl, tiles in (("C1", I.TINY_F32, 1), ("C2", I.SMALL_BF16, 1)):
            pl = wl.placement()
            qkv = tuple(oracle.widen(x[:tiles], wl.dtype) for x in wl.qkv())
            t0 = time.perf_counter()
            c = G.tile_coords(pl.face[:tiles], pl.oy[:tiles], pl.ox[:tiles], wl.H, wl.W).astype(np.float32)
            oracle.na3d_fwd(*qkv, (wl.kz, wl.ky, wl.kx), wl.scale, coords=c)
            dt = (time.perf_counter() - t0) * wl.B / tiles
            flops = 4.0 * wl.B * wl.heads * wl.N * wl.K * wl.d
            res[key] = {"seconds": round(dt, 4), "tflops": flops / dt / 1e12, "cores": 1,
                        "sample": f"{tiles} of {wl.B} tiles, scaled to all" if tiles < wl.B else "whole workload"}
    finally:
        oracle.set_num_threads(n0)
    return res


def train_tile(steps: int):
    """Forward and backward of the 16-tile 5x9x9 training tile (StereoRoPE on), and
    the standalone rotation of its Q and K; HIP-event times on the current stream."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    from paper_2606_31248_amd import pipeline as Pp

    wl = I.TRAIN_TILE_BWD
    dev = torch.device("cuda:0")

    def to_dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v = (to_dev(x) for x in wl.qkv())
    g = to_dev(wl.dout())
    geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in wl.placement().as_int32()))
    _, cs = Pp.stereo_phases(geom, wl.H, wl.W, wl.d)
    window = (wl.kz, wl.ky, wl.kx)
    desc = Bd.desc_for(q, window, wl.scale)
    out = torch.empty_like(q)
    lse = torch.empty(wl.shape()[:-1], dtype=torch.float32, device=dev)
    ws = torch.empty(Bd.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device=dev)
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    qr = torch.empty_like(q)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        st = torch.cuda.current_stream()
        ts = []
        for _ in range(steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            fn()
            e1.record(st)
            ts.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in ts]))

    fwd_ms = timed(lambda: Bd.strata_na3d_fwd(desc, q, k, v, cs, out, lse))
    bwd_ms = timed(lambda: Bd.strata_na3d_bwd(desc, q, k, v, cs, out, g, lse, dq, dk, dv, ws))

    def rope_qk():
        Bd.strata_stereorope_apply(q, qr, cs)
        Bd.strata_stereorope_apply(k, qr, cs)
    rope_ms = timed(rope_qk)
    n = wl.B * wl.heads * wl.N
    fwd_fl, bwd_fl = 4.0 * n * wl.K * wl.d, 10.0 * n * wl.K * wl.d
    rope_bytes = 2 * 2 * n * wl.d * 2 + 2 * wl.B * wl.H * wl.W * wl.d * 4   # Q, K read+write; phases
    # algorithmic bytes per token-head: forward reads Q, K, V and writes O (bf16) and
    # LSE (fp32); backward reads Q, K, V, O, dO (bf16) and LSE, writes dQ, dK, dV
    fwd_bytes, bwd_bytes = n * (4 * wl.d * 2 + 4), n * (8 * wl.d * 2 + 4)
    out = {
        "workload": f"{wl.name}: {wl.B} tiles x {wl.heads} heads x {wl.Z}x{wl.H}x{wl.W}, window "
                    f"{wl.kz}x{wl.ky}x{wl.kx}, StereoRoPE on",
        "fwd_ms": round(fwd_ms, 4), "fwd_tflops": round(fwd_fl / fwd_ms / 1e9, 2),
        "bwd_ms": round(bwd_ms, 4), "bwd_tflops": round(bwd_fl / bwd_ms / 1e9, 2),
        "bwd_pct_bf16_peak": round(100 * bwd_fl / bwd_ms / 1e9 / PEAK_BF16_TFLOPS, 2),
        "bwd_flops_model": "10 B h N K d (QK^T twice, dO.V^T, P^T.dO, dS.K, dS^T.Q)",
        "rope_apply_qk": {"ms": round(rope_ms, 4), "gbs": round(rope_bytes / rope_ms / 1e6, 1),
                          "frac_hbm": round(rope_bytes / rope_ms / 1e6 / PEAK_HBM_GBS, 4)},
    }
    out["_fwd"] = (fwd_fl, fwd_bytes, fwd_ms)
    out["_bwd"] = (bwd_fl, bwd_bytes, bwd_ms)
    return out


def _timed(fn, steps: int) -> float:
    """Mean HIP-event time (ms) of fn on the current stream over `steps` passes."""
    import torch
    fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    ts = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        fn()
        e1.record(st)
        ts.append((e0, e1))
    torch.cuda.synchronize()
    return float(np.mean([a.elapsed_time(b) for a, b in ts]))


def options_face_fwd(wl, desc, q, k, v, cs, out, steps: int) -> dict:
    """The face forward with the attention-block options (QK RMSNorm, sigmoid
    output gate per channel or per token-head) against the plain forward."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    dev = q.device
    gd = torch.from_numpy(I.gaussian(wl.shape(), wl.seed, I.STREAM_GATE, "bf16", 2.0).view(np.int16)).view(
        torch.bfloat16).to(dev)
    g1 = gd[..., 0].contiguous()
    n = wl.B * wl.heads * wl.N
    flops = 4.0 * n * wl.K * wl.d
    variants = {"plain": (None, 0), "norm": (Bd.make_opts(True, 1e-6, None), 0),
                "gate_d": (Bd.make_opts(False, 1e-6, gd), n * wl.d * 2),
                "norm_gate_1": (Bd.make_opts(True, 1e-6, g1), n * 2),
                "norm_gate_d": (Bd.make_opts(True, 1e-6, gd), n * wl.d * 2)}
    res = {}
    for name, (opts, extra) in variants.items():
        ms = _timed(lambda: Bd.strata_na3d_fwd_ex(desc, opts, q, k, v, cs, out, None), steps)
        nbytes = 4.0 * n * wl.d * 2 + extra
        res[name] = dict(roofline_row(flops, nbytes, ms), ms=round(ms, 4),
                         achieved_gbs=round(nbytes / ms / 1e6, 1), frac_hbm=round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4))
    del gd, g1
    return res


def options_train_bwd(steps: int) -> dict:
    """The 16-tile 5x9x9 training-tile backward with QK RMSNorm and a per-channel
    gate (gate row pass included) against the plain backward."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    from paper_2606_31248_amd import pipeline as Pp
    wl = I.TRAIN_TILE_BWD
    dev = torch.device("cuda:0")
    to_dev = lambda bits: torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)
    q, k, v = (to_dev(x) for x in wl.qkv())
    g = to_dev(wl.dout())
    gd = to_dev(I.gaussian(wl.shape(), wl.seed, I.STREAM_GATE, "bf16", 2.0))
    geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in wl.placement().as_int32()))
    _, cs = Pp.stereo_phases(geom, wl.H, wl.W, wl.d)
    desc = Bd.desc_for(q, (wl.kz, wl.ky, wl.kx), wl.scale)
    out = torch.empty_like(q)
    lse = torch.empty(wl.shape()[:-1], dtype=torch.float32, device=dev)
    dq, dk, dv, dgt = (torch.empty_like(q) for _ in range(4))
    n = wl.B * wl.heads * wl.N
    flops = 10.0 * n * wl.K * wl.d
    res = {}
    for name, opts in (("plain", None), ("norm", Bd.make_opts(True, 1e-6, None)),
                       ("norm_gate_d", Bd.make_opts(True, 1e-6, gd))):
        ws = torch.empty(Bd.strata_na3d_bwd_ex_workspace_size(desc, opts), dtype=torch.uint8, device=dev)
        Bd.strata_na3d_fwd_ex(desc, opts, q, k, v, cs, out, lse)
        dgate = dgt if opts is not None and opts.gate else None
        ms = _timed(lambda: Bd.strata_na3d_bwd_ex(desc, opts, q, k, v, cs, out, g, lse, dq, dk, dv, dgate, ws),
                    steps)
        res[name] = {"ms": round(ms, 4), "tflops": round(flops / ms / 1e9, 2)}
        del ws
    return res


def paper_shapes(steps: int) -> dict:
    """The paper's own attention shapes (24 levels): NA3D 9x9x9 on 16x16- and
    32x32-token tiles, 3x7x7 over 24 levels (forward), column-wise attention over
    all 24 levels, the decoder's head_dim-128 NA3D; forward (and backward) against
    their rooflines.  Inputs
    are seeded N(0,1) drawn on the device (their values do not change the time)."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    from paper_2606_31248_amd import pipeline as Pp
    dev = torch.device("cuda:0")
    res = {}
    for wl, bwd in ((I.PAPER_TILE16, True), (I.PAPER_TILE32, True), (I.Z24_TILE, False), (I.PAPER_COLUMN, True),
                    (I.PAPER_DECODER, True)):
        gen = torch.Generator(device=dev)
        gen.manual_seed(wl.seed)
        q, k, v, g = (torch.randn(wl.shape(), generator=gen, device=dev).to(torch.bfloat16) for _ in range(4))
        cs = None
        if wl.ky > 1 or wl.kx > 1:  # the rotation cancels inside a column
            geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in wl.placement().as_int32()))
            _, cs = Pp.stereo_phases(geom, wl.H, wl.W, wl.d)
        desc = Bd.desc_for(q, (wl.kz, wl.ky, wl.kx), wl.scale)
        out = torch.empty_like(q)
        lse = torch.empty(wl.shape()[:-1], dtype=torch.float32, device=dev)
        n = wl.B * wl.heads * wl.N
        fl, nb = 4.0 * n * wl.K * wl.d, n * (4 * wl.d * 2 + 4)
        ms = _timed(lambda: Bd.strata_na3d_fwd(desc, q, k, v, cs, out, lse), steps)
        row = dict(roofline_row(fl, nb, ms), ms=round(ms, 4), pct_bf16_peak=round(100 * fl / ms / 1e9 / PEAK_BF16_TFLOPS, 2))
        entry = {"shape": list(wl.shape()), "window": [wl.kz, wl.ky, wl.kx], "fwd": row}
        if bwd:
            ws = torch.empty(Bd.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device=dev)
            dq, dk, dv = (torch.empty_like(q) for _ in range(3))
            ms = _timed(lambda: Bd.strata_na3d_bwd(desc, q, k, v, cs, out, g, lse, dq, dk, dv, ws), steps)
            fl, nb = 10.0 * n * wl.K * wl.d, n * (8 * wl.d * 2 + 4)
            entry["bwd"] = dict(roofline_row(fl, nb, ms), ms=round(ms, 4),
                                pct_bf16_peak=round(100 * fl / ms / 1e9 / PEAK_BF16_TFLOPS, 2))
            del ws, dq, dk, dv
        if wl is I.PAPER_DECODER:
            # the production attention block (App. B.5): QK RMSNorm and a per-channel gate
            gt = torch.randn(wl.shape(), generator=gen, device=dev).to(torch.bfloat16)
            opts = Bd.make_opts(True, 1e-6, gt)
            ms = _timed(lambda: Bd.strata_na3d_fwd_ex(desc, opts, q, k, v, cs, out, lse), steps)
            entry["fwd_norm_gate_d"] = dict(roofline_row(4.0 * n * wl.K * wl.d, n * (5 * wl.d * 2 + 4), ms),
                                            ms=round(ms, 4))
            ws = torch.empty(Bd.strata_na3d_bwd_ex_workspace_size(desc, opts), dtype=torch.uint8, device=dev)
            dq, dk, dv, dg = (torch.empty_like(q) for _ in range(4))
            ms = _timed(lambda: Bd.strata_na3d_bwd_ex(desc, opts, q, k, v, cs, out, g, lse, dq, dk, dv, dg, ws), steps)
            entry["bwd_norm_gate_d"] = dict(roofline_row(10.0 * n * wl.K * wl.d, n * (10 * wl.d * 2 + 4), ms),
                                            ms=round(ms, 4))
            del gt, ws, dq, dk, dv, dg
        res[wl.name] = entry
        del q, k, v, g, out, lse, cs
        torch.cuda.empty_cache()
    return res


def wind_frame(steps: int) -> dict:
    """Wind vectors of the face-rollout tiling, in cells (9 x 9 tiles of 256 x 256
    cells, stride 224, 8 levels, bf16), rotated into each tile's centre frame
    while being cut from the face: HBM-bound (one read, one write per value)."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(1010)
    n, P = 2048, 8
    field = torch.randn((P, n, n, 2), generator=gen, device=dev).to(torch.bfloat16)
    tiles = torch.empty((81, P, 256, 256, 2), dtype=torch.bfloat16, device=dev)
    ms = _timed(lambda: Bd.strata_wind_tile_frame(field, 0, 9, 9, 224, 224, tiles), steps)
    nbytes = 2 * tiles.numel() * 2
    del field, tiles
    return {"workload": "face_rollout_cells_81x8x256x256x2_bf16", "ms": round(ms, 4), "bound": "hbm",
            "achieved_gbs": round(nbytes / ms / 1e6, 1), "frac_hbm": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4)}


def duo_padding(steps: int) -> dict:
    """Duo-grid halo padding of all six 2048-cell faces by 16 cells (8 levels x 4
    channels, bf16): the padding operator built once as a plan, then applied
    (interior copy plus the 4-neighbour halo gather, HBM-bound); the one-shot
    entry point (geometry recomputed in the same launch) beside it."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(1011)
    n, h, P, C = 2048, 16, 8, 4
    faces = torch.randn((6, P, n, n, C), generator=gen, device=dev).to(torch.bfloat16)
    padded = torch.empty((6, P, n + 2 * h, n + 2 * h, C), dtype=torch.bfloat16, device=dev)
    plan = torch.empty(Bd.strata_duo_plan_bytes(n, h), dtype=torch.uint8, device=dev)
    plan_ms = _timed(lambda: Bd.strata_duo_plan(n, h, plan), max(steps, 3))
    ms = _timed(lambda: Bd.strata_duo_pad_planned(faces, h, plan, padded), steps)
    one_shot_ms = _timed(lambda: Bd.strata_duo_pad(faces, h, padded), steps)
    # the adjoint: padded-shape gradient in, face-shape gradient out (same bytes)
    vjp_ms = _timed(lambda: Bd.strata_duo_pad_vjp(padded, h, plan, faces), steps)
    nbytes = (faces.numel() + padded.numel()) * 2
    del faces, padded, plan
    return {"workload": "duo_pad_6x8x2048x2048x4_halo16_bf16", "ms": round(ms, 4), "bound": "hbm",
            "achieved_gbs": round(nbytes / ms / 1e6, 1), "frac_hbm": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4),
            "plan_build_ms": round(plan_ms, 4), "one_shot_ms": round(one_shot_ms, 4),
            "vjp_ms": round(vjp_ms, 4), "vjp_frac_hbm": round(nbytes / vjp_ms / 1e6 / PEAK_HBM_GBS, 4),
            "alg_bytes": nbytes}


def _seeded_device(wl, dev, gen_seed=None):
    """q, k, v (and dO) of a workload on the device: N(0,1) bf16 drawn on the device
    from a seeded generator (the time does not depend on the values)."""
    import torch
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed if gen_seed is None else gen_seed)
    dt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    return tuple(torch.randn(wl.shape(), generator=gen, device=dev).to(dt) for _ in range(4))


def profile_workload(name: str, steps: int, warmup: int, calib_copy: bool = False) -> dict:
    """Run one kernel call of one workload `warmup + steps` times and nothing else
    (no oracle, no side measurements): the target of rocprofv3 counter runs.

    Names: face_step (the timed step of the default run), c1 .. c3 (forwards of
    the tiny, 8-tile and training-tile workloads), c4 (the training-tile
    backward), paper16_fwd / paper16_bwd (9x9x9 at 24 levels on 16x16-token
    tiles), paper32_fwd / paper32_bwd, z24_fwd (3x7x7 at 24 levels),
    column_fwd / column_bwd (window 24x1x1 over all 24 levels), decoder_fwd /
    decoder_bwd (head_dim 128, 9x9x9),
    rope (the standalone rotation of the training tile's Q), blend (the whole
    stitch of the face tiling), wind (the wind rotation cut from one face into
    the face tiling), duo (the planned Duo padding)."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    from paper_2606_31248_amd import pipeline as Pp
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    Bd.load()
    if calib_copy:  # one 1 GiB device copy: the HBM counter calibration of the same run
        src = torch.empty(CALIB_BYTES // 2, dtype=torch.int16, device=dev).fill_(1)
        torch.empty_like(src).copy_(src)
        torch.cuda.synchronize()
        del src
    fwd_wl = {"c1": I.TINY_F32, "c2": I.SMALL_BF16, "c3": I.TRAIN_TILE, "paper16_fwd": I.PAPER_TILE16,
              "paper32_fwd": I.PAPER_TILE32, "z24_fwd": I.Z24_TILE, "column_fwd": I.PAPER_COLUMN,
              "decoder_fwd": I.PAPER_DECODER}
    bwd_wl = {"c4": I.TRAIN_TILE_BWD, "paper16_bwd": I.PAPER_TILE16, "paper32_bwd": I.PAPER_TILE32,
              "column_bwd": I.PAPER_COLUMN, "decoder_bwd": I.PAPER_DECODER}
    if name in fwd_wl or name in bwd_wl or name == "rope":
        wl = fwd_wl.get(name) or bwd_wl.get(name) or I.TRAIN_TILE
        q, k, v, g = _seeded_device(wl, dev)
        geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in wl.placement().as_int32()))
        _, cs = Pp.stereo_phases(geom, wl.H, wl.W, wl.d)
        desc = Bd.desc_for(q, (wl.kz, wl.ky, wl.kx), wl.scale)
        out = torch.empty_like(q)
        lse = torch.empty(wl.shape()[:-1], dtype=torch.float32, device=dev)
        if name == "rope":
            fn = lambda: Bd.strata_stereorope_apply(q, out, cs)
        elif name in fwd_wl:
            fn = lambda: Bd.strata_na3d_fwd(desc, q, k, v, cs, out, lse)
        else:
            Bd.strata_na3d_fwd(desc, q, k, v, cs, out, lse)
            ws = torch.empty(Bd.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device=dev)
            dq, dk, dv = (torch.empty_like(q) for _ in range(3))
            fn = lambda: Bd.strata_na3d_bwd(desc, q, k, v, cs, out, g, lse, dq, dk, dv, ws)
    elif name in ("face_step", "blend"):
        wl = I.FACE_ROLLOUT
        nty, ntx, sy, sx = wl.tiling
        Hf, Wf = (nty - 1) * sy + wl.H, (ntx - 1) * sx + wl.W
        q, k, v, _ = _seeded_device(wl, dev)
        geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in wl.placement().as_int32()))
        win = torch.from_numpy(I.ramp_window_2d(wl.H, wl.W, I.FACE_OVERLAP)).to(dev)
        face = torch.empty((wl.heads * wl.Z, Hf, Wf, wl.d), dtype=torch.bfloat16, device=dev)
        out = torch.empty_like(q)
        coords = torch.empty((wl.B, wl.H, wl.W, 2), dtype=torch.float32, device=dev)
        cs = torch.empty((wl.B, wl.H, wl.W, wl.d // 2, 2), dtype=torch.float32, device=dev)
        if name == "blend":
            planes = q.view(wl.B, wl.heads * wl.Z, wl.H, wl.W, wl.d)
            fn = lambda: Bd.strata_tile_blend(planes, nty, ntx, sy, sx, win, face)
        else:
            fn = lambda: Pp.face_step(q, k, v, geom, (wl.kz, wl.ky, wl.kx), wl.scale, wl.tiling, win, face,
                                      coords=coords, cs=cs, out=out, fused=True)
    elif name == "wind":
        gen = torch.Generator(device=dev)
        gen.manual_seed(1010)
        field = torch.randn((8, 2048, 2048, 2), generator=gen, device=dev).to(torch.bfloat16)
        tiles = torch.empty((81, 8, 256, 256, 2), dtype=torch.bfloat16, device=dev)
        fn = lambda: Bd.strata_wind_tile_frame(field, 0, 9, 9, 224, 224, tiles)
    elif name == "duo":
        n, h, P, C = 2048, 16, 8, 4
        gen = torch.Generator(device=dev)
        gen.manual_seed(1011)
        faces = torch.randn((6, P, n, n, C), generator=gen, device=dev).to(torch.bfloat16)
        padded = torch.empty((6, P, n + 2 * h, n + 2 * h, C), dtype=torch.bfloat16, device=dev)
        plan = torch.empty(Bd.strata_duo_plan_bytes(n, h), dtype=torch.uint8, device=dev)
        Bd.strata_duo_plan(n, h, plan)
        fn = lambda: Bd.strata_duo_pad_planned(faces, h, plan, padded)
    else:
        raise SystemExit(f"unknown profile workload {name!r}")
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ms = _timed(fn, steps)
    return {"profile_workload": name, "steps": steps, "warmup": warmup, "ms_mean": round(ms, 4)}


# ---- the workloads C1-C4 on the GPU, and the parity of every timed output -------
# The GPU half (config_runs) times each workload and keeps a seeded sample of its
# outputs on the host; the CPU leg (cpu_leg) evaluates the oracle on those same
# samples and on the sampled face cells of the timed step, and times the oracle.

BF16_RULE = 2e-2      # max |gpu - oracle| <= 2e-2 RMS(oracle) for bf16 results
F32_RULE = 1e-5       # max |gpu - oracle| for float32 results


def _half_ulp_bf16(a: np.ndarray) -> np.ndarray:
    """Half a bf16 ulp of every exact value: the error of storing it in bf16 at all."""
    a = np.abs(a)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8), 0.0)


def parity_bf16(got: np.ndarray, ref: np.ndarray, carried=None) -> dict:
    """The bf16 rule as written (max |err| / RMS(ref) <= 2e-2) and as applied by the
    tests: beyond half a bf16 ulp of the exact value (the rounding of storing it at
    all) plus `carried` (rounding the value inherits, e.g. the tiles' own storage
    rounding carried through the stitch)."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    diff = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref)))
    excess = diff - _half_ulp_bf16(ref) - (0.0 if carried is None else carried)
    lit, r11 = float(diff.max()) / rms, float(excess.max()) / rms
    return {"n_values": int(ref.size), "max_abs_err": float(diff.max()), "rms_ref": rms,
            "err_over_rms_literal": round(lit, 6), "r11_excess_over_rms": round(r11, 6), "bound": BF16_RULE,
            "pass_literal": bool(lit <= BF16_RULE), "pass_r11": bool(r11 <= BF16_RULE)}


def face_sample_cells(wl, per_plane: int = 16, seed: int = 1105):
    """Face cells of the face-rollout step to check: on every plane, the face
    corners, single-cover cells of the corner tile and of an interior tile, and
    cells of the y-overlap strip, the x-overlap strip and the four-tile corner
    where the interior tile row/column meets the next one.  Returns (plane, y, x)
    arrays; every covering tile lies in a small set (corner tiles and the 2 x 2
    junction), which keeps the oracle's work bounded."""
    nty, ntx, sy, sx = wl.tiling
    Hf, Wf = (nty - 1) * sy + wl.H, (ntx - 1) * sx + wl.W
    ov_y, ov_x = wl.H - sy, wl.W - sx
    a0, b0 = nty // 2 - 1, ntx // 2 - 1
    ys1, xs1 = (a0 * sy + ov_y, (a0 + 1) * sy), (b0 * sx + ov_x, (b0 + 1) * sx)   # interior single cover
    ysov, xsov = ((a0 + 1) * sy, a0 * sy + wl.H), ((b0 + 1) * sx, b0 * sx + wl.W)  # overlap strips
    regions = [((0, sy), (0, sx), 2), (ys1, xs1, 3), (ysov, xs1, 3), (ys1, xsov, 3), (ysov, xsov, 3)]
    corners = [(0, 0), (0, Wf - 1), (Hf - 1, 0), (Hf - 1, Wf - 1)]
    rng = np.random.default_rng(seed)
    cells = []
    for p in range(wl.heads * wl.Z):
        for j in range(per_plane - sum(r[2] for r in regions)):
            cells.append((p,) + corners[(p * 2 + j) % 4])
        for (y0, y1), (x0, x1), n in regions:
            for _ in range(n):
                cells.append((p, int(rng.integers(y0, y1)), int(rng.integers(x0, x1))))
    c = np.array(cells, np.int64)
    return c[:, 0], c[:, 1], c[:, 2]


def _covering(y, L, s, n):
    """Tiles along one axis covering face position y, with the local position."""
    return [(a, y - a * s) for a in range(n) if 0 <= y - a * s < L]


def oracle_rows(oracle, G, qkv_bits, pl, wl, groups, coords_cache=None):
    """Oracle forward rows for {(tile, head): [flat query index in [Z, H, W]]}: each
    (tile, head) slice widened on its own, so the full tensors never go to float64."""
    out = {}
    cc = {} if coords_cache is None else coords_cache
    for (t, h), sel in groups.items():
        if t not in cc:
            cc[t] = G.tile_coords(pl.face[t:t + 1], pl.oy[t:t + 1], pl.ox[t:t + 1], wl.H, wl.W).astype(np.float32)
        q, k, v = (oracle.widen(a[t:t + 1, h:h + 1], wl.dtype) for a in qkv_bits)
        o, lse = oracle.na3d_fwd(q, k, v, (wl.kz, wl.ky, wl.kx), wl.scale, coords=cc[t] if wl.rope else None,
                                 sel=np.asarray(sel, np.int64))
        out[(t, h)] = (o, lse)
    return out


def face_parity(wl, qkv_bits, face_rows, cells, win) -> dict:
    """Parity of the timed step's own face against the oracle: the oracle forward of
    every covering tile's query of each sampled cell, stitched in float64 with the
    same weights (ref = sum w o / sum w).  The face stores the stitch of bf16 tile
    values, so the applied rule also carries the tiles' own storage rounding
    through the weights."""
    ref, carried, meta = face_reference(wl, qkv_bits, cells, win)
    rec = parity_bf16(face_rows, ref, carried)
    rec.update(meta)
    return rec


def face_reference(wl, qkv_bits, cells, win):
    """(ref, carried, meta) of face_parity: the oracle's stitched value of every
    sampled cell [n, d], the tiles' bf16 storage rounding carried through the
    stitch weights [n, d], and a description of the sample."""
    import oracle
    from oracle import geometry as G
    nty, ntx, sy, sx = wl.tiling
    pl = wl.placement()
    P_, Y, X = cells
    groups, plan = {}, []
    for p, y, x in zip(P_, Y, X):
        h, z = divmod(int(p), wl.Z)
        cov = [(a * ntx + b, ly, lx) for a, ly in _covering(int(y), wl.H, sy, nty)
               for b, lx in _covering(int(x), wl.W, sx, ntx)]
        ent = []
        for t, ly, lx in cov:
            sel = groups.setdefault((t, h), [])
            ent.append((t, h, len(sel), float(win[ly * wl.W + lx])))
            sel.append((z * wl.H + ly) * wl.W + lx)
        plan.append(ent)
    rows = oracle_rows(oracle, G, qkv_bits, pl, wl, groups)
    ref = np.zeros((len(plan), wl.d))
    carried = np.zeros((len(plan), wl.d))
    for i, ent in enumerate(plan):
        wsum = sum(w for *_, w in ent)
        for t, h, j, w in ent:
            o = rows[(t, h)][0][j]
            ref[i] += w * o
            carried[i] += w * _half_ulp_bf16(o)
        ref[i] /= wsum
        carried[i] /= wsum
    meta = {"n_cells": len(plan), "n_tiles": len({t for t, _ in groups}), "planes": int(len(np.unique(P_))),
            "cells": "every plane: face corners, single-cover cells of a corner and an interior tile, the "
                     "y- and x-overlap strips and the 4-tile corner of an interior junction"}
    return ref, carried, meta


def _flush_mall(buf):
    """Overwrite a 1 GiB buffer: evicts the 256 MB last-level cache (MALL) between timed launches."""
    buf.fill_(1)


def config_runs(steps: int) -> dict:
    """C1-C4 of the workload list on the GPU, with seeded host inputs: times per
    launch (HIP events on the launch stream) and, for the CPU leg, the outputs
    to check (C1, C2 whole; C3, C4 sampled rows)."""
    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    from paper_2606_31248_amd import pipeline as Pp
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(2024)
    runs = {}

    def to_dev(bits, dtype):
        if dtype == "bf16":
            return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(bits).to(dev)

    def fwd_setup(wl, mult=1.0):
        qkv = tuple(I.gaussian(wl.shape(), wl.seed, s, wl.dtype, mult) for s in (I.STREAM_Q, I.STREAM_K, I.STREAM_V))
        q, k, v = (to_dev(x, wl.dtype) for x in qkv)
        geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in wl.placement().as_int32()))
        _, cs = Pp.stereo_phases(geom, wl.H, wl.W, wl.d)
        out = torch.empty_like(q)
        lse = torch.empty(wl.shape()[:-1], dtype=torch.float32, device=dev)
        return qkv, (q, k, v), cs, out, lse

    def sample(wl, n_groups, per_group):
        """(tile, head) groups and flat query indices inside [Z, H, W]."""
        N = wl.Z * wl.H * wl.W
        th = rng.choice(wl.B * wl.heads, size=min(n_groups, wl.B * wl.heads), replace=False)
        return {(int(x) // wl.heads, int(x) % wl.heads): np.sort(rng.choice(N, per_group, replace=False))
                for x in th}

    def rows_of(t, groups, wl):
        idx = np.concatenate([(t_ * wl.heads + h) * wl.Z * wl.H * wl.W + sel for (t_, h), sel in groups.items()])
        flat = t.reshape(-1, wl.d)
        return flat.index_select(0, torch.from_numpy(idx).to(dev)).float().cpu().numpy().astype(np.float64)

    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    for key, wl, mult, scale in (("C1", I.TINY_F32, 1.0, None), ("C2", I.SMALL_BF16, 1.0, None),
                                 ("C2_literal", I.SMALL_BF16, 1.0 / 8.0, None), ("C3", I.TRAIN_TILE, 1.0, None)):
        qkv, (q, k, v), cs, out, lse = fwd_setup(wl, mult)
        desc = Bd.desc_for(q, (wl.kz, wl.ky, wl.kx), wl.scale if scale is None else scale)
        fn = lambda: Bd.strata_na3d_fwd(desc, q, k, v, cs, out, lse)
        warm = _timed(fn, steps)
        st = torch.cuda.current_stream()
        ts = []
        for _ in range(max(steps, 5)):  # each launch after a cache flush
            _flush_mall(flush)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            fn()
            e1.record(st)
            ts.append((e0, e1))
        torch.cuda.synchronize()
        cold = float(np.mean([a.elapsed_time(b) for a, b in ts]))
        n = wl.B * wl.heads * wl.N
        flops = 4.0 * n * wl.K * wl.d
        nbytes = n * (4 * wl.d * (4 if wl.dtype == "f32" else 2) + 4)
        r = {"workload": wl.name + (" (inputs x 1/8 as well: the literal reading of 'scaled by 1/sqrt(64)')"
                                    if key == "C2_literal" else ""),
             "ms": round(cold, 4), "ms_cache_warm": round(warm, 4), "timing": "mean of HIP-event times, each "
             "launch after a 1 GiB write that evicts the 256 MB MALL; ms_cache_warm: back-to-back launches",
             "tflops": round(flops / cold / 1e9, 2), "tokens_per_s": round(wl.B * wl.N / (cold * 1e-3), 1),
             "pct_bf16_peak": round(100 * flops / cold / 1e9 / PEAK_BF16_TFLOPS, 3),
             "roofline": roofline_row(flops, nbytes, cold), "dtype": wl.dtype}
        if key in ("C1", "C2", "C2_literal"):   # checked whole
            r["_got"] = (out.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64))
        else:
            groups = sample(wl, 32, 32)
            r["_groups"] = groups
            r["_got"] = (rows_of(out, groups, wl), None)
        r["_qkv"], r["_wl"] = qkv, wl
        r["_scale"] = wl.scale if scale is None else scale
        runs[key] = r
        del q, k, v, out, lse, cs
        torch.cuda.empty_cache()
    del flush
    # C4: the training-tile backward (forward first for out and lse)
    wl = I.TRAIN_TILE_BWD
    qkv, (q, k, v), cs, out, lse = fwd_setup(wl)
    dob = wl.dout()
    g = to_dev(dob, wl.dtype)
    desc = Bd.desc_for(q, (wl.kz, wl.ky, wl.kx), wl.scale)
    Bd.strata_na3d_fwd(desc, q, k, v, cs, out, lse)
    ws = torch.empty(Bd.strata_na3d_bwd_workspace_size(desc), dtype=torch.uint8, device=dev)
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    ms = _timed(lambda: Bd.strata_na3d_bwd(desc, q, k, v, cs, out, g, lse, dq, dk, dv, ws), steps)
    n = wl.B * wl.heads * wl.N
    flops, nbytes = 10.0 * n * wl.K * wl.d, n * (8 * wl.d * 2 + 4)
    gq, gk = sample(wl, 16, 16), sample(wl, 16, 16)
    runs["C4"] = {"workload": wl.name, "ms": round(ms, 4), "tflops": round(flops / ms / 1e9, 2),
                  "pct_bf16_peak": round(100 * flops / ms / 1e9 / PEAK_BF16_TFLOPS, 3),
                  "roofline": roofline_row(flops, nbytes, ms), "dtype": wl.dtype,
                  "flops_model": "10 B h N K d (QK^T twice, dO.V^T, P^T.dO, dS.K, dS^T.Q)",
                  "_groups": (gq, gk), "_got": (rows_of(dq, gq, wl), rows_of(dk, gk, wl), rows_of(dv, gk, wl)),
                  "_qkv": qkv, "_dout": dob, "_wl": wl, "_scale": wl.scale}
    del q, k, v, out, lse, cs, g, ws, dq, dk, dv
    torch.cuda.empty_cache()
    return runs


def config_parity(runs: dict) -> dict:
    """The oracle on every config's checked outputs (CPU leg)."""
    import oracle
    from oracle import geometry as G
    res = {}
    for key, r in runs.items():
        wl, qkv = r["_wl"], r["_qkv"]
        pl = wl.placement()
        window = (wl.kz, wl.ky, wl.kx)
        if key in ("C1", "C2", "C2_literal"):
            c32 = G.tile_coords(pl.face, pl.oy, pl.ox, wl.H, wl.W).astype(np.float32)
            ro, rl = oracle.na3d_fwd(*(oracle.widen(a, wl.dtype) for a in qkv), window, r["_scale"], coords=c32)
            got, gl = r["_got"]
            if wl.dtype == "f32":
                err = float(np.max(np.abs(got - ro)))
                par = {"n_values": int(ro.size), "max_abs_err": err, "bound": F32_RULE, "pass": bool(err <= F32_RULE)}
            else:
                par = parity_bf16(got, ro)
            par["lse_max_abs_err"] = float(np.max(np.abs(gl - rl)))
            par["checked"] = "every output of the launch"
        elif key == "C3":
            rows = oracle_rows(oracle, G, qkv, pl, wl, r["_groups"])
            ref = np.concatenate([rows[g][0] for g in r["_groups"]])
            par = parity_bf16(r["_got"][0], ref)
            par["checked"] = f"{ref.shape[0]} query rows of {len(r['_groups'])} (tile, head) pairs"
        else:  # C4
            gq, gk = r["_groups"]
            refs = {"dq": [], "dk": [], "dv": []}
            cc = {}
            for (t, h), sel in gq.items():
                s = slice(t, t + 1), slice(h, h + 1)
                if t not in cc:
                    cc[t] = G.tile_coords(pl.face[t:t + 1], pl.oy[t:t + 1], pl.ox[t:t + 1], wl.H,
                                          wl.W).astype(np.float32)
                dq, _, _ = oracle.na3d_bwd(*(oracle.widen(a[s], wl.dtype) for a in qkv + (r["_dout"],)), window,
                                           wl.scale, coords=cc[t], selq=sel, selk=sel[:1])
                refs["dq"].append(dq)
            for (t, h), sel in gk.items():
                s = slice(t, t + 1), slice(h, h + 1)
                if t not in cc:
                    cc[t] = G.tile_coords(pl.face[t:t + 1], pl.oy[t:t + 1], pl.ox[t:t + 1], wl.H,
                                          wl.W).astype(np.float32)
                _, dk, dv = oracle.na3d_bwd(*(oracle.widen(a[s], wl.dtype) for a in qkv + (r["_dout"],)), window,
                                            wl.scale, coords=cc[t], selq=sel[:1], selk=sel)
                refs["dk"].append(dk)
                refs["dv"].append(dv)
            par = {name: parity_bf16(got, np.concatenate(refs[name]))
                   for name, got in zip(("dq", "dk", "dv"), r["_got"])}
            par["checked"] = (f"{sum(len(x) for x in gq.values())} dq rows of {len(gq)} and "
                              f"{sum(len(x) for x in gk.values())} dk, dv rows of {len(gk)} (tile, head) pairs")
        res[key] = par
    return res


def _done(what: str, t_start: float) -> None:
    """One progress line on stderr per finished measurement (stdout carries only the result)."""
    print(f"bench: {what} done at {time.perf_counter() - t_start:.1f} s", file=sys.stderr, flush=True)


def roofline_row(flops: float, nbytes: float, ms: float) -> dict:
    """Achieved rate of a kernel against min(MFMA peak, intensity x HBM peak)."""
    ai = flops / nbytes
    cap = min(PEAK_BF16_TFLOPS, ai * PEAK_HBM_GBS / 1e3)
    tf = flops / ms / 1e9
    return {"bound": "hbm" if cap < PEAK_BF16_TFLOPS else "mfma", "flop_per_byte": round(ai, 1),
            "cap_tflops": round(cap, 1), "achieved_tflops": round(tf, 2), "frac_of_cap": round(tf / cap, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-tiles", type=int, default=32, help="tiles in the CPU-oracle sample (0: skip)")
    ap.add_argument("--train-steps", type=int, default=5,
                    help="timed passes of the training-tile forward/backward side measurement (0: skip)")
    ap.add_argument("--config-steps", type=int, default=5,
                    help="timed launches of each of the workloads C1-C4 (0: skip them)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the HBM-traffic summary of two rocprofv3 --pmc runs to profiles/ and exit")
    ap.add_argument("--summarize-sq", metavar="SQ_DIR",
                    help="write the instruction-mix summary of a rocprofv3 --pmc run of SQ counters to profiles/ and exit")
    ap.add_argument("--summarize-stats", metavar="KERNEL_STATS_CSV",
                    help="write the kernel-trace summary of a rocprofv3 --stats run to profiles/ and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar=("NAME", "DIR"),
                    help="write profiles/NAME.txt, the per-kernel summary of rocprofv3 --pmc runs in DIR..., and exit")
    ap.add_argument("--label", default="", help="what the summarized counter runs measured")
    ap.add_argument("--command", action="append", default=[],
                    help="the profiler command(s) the summary records")
    ap.add_argument("--profile", metavar="WORKLOAD",
                    help="run only one kernel call of one workload (see profile_workload) and exit")
    a = ap.parse_args()
    if a.profile:
        print(json.dumps(profile_workload(a.profile, a.steps, a.warmup, a.calib_copy)), flush=True)
        return
    if a.summarize_counters:
        name, dirs = a.summarize_counters[0], a.summarize_counters[1:]
        txt = summarize_counters(a.label or name, dirs, a.command)
        with open(os.path.join(ROOT, "profiles", name + ".txt"), "w") as f:
            f.write(txt)
        print(txt)
        return
    if a.summarize_pmc:
        rec = summarize_pmc(a.summarize_pmc[0], a.summarize_pmc[1], a.command)
        with open(PMC_FILE, "w") as f:
            json.dump(rec, f, indent=1)
        print(json.dumps(rec))
        return
    if a.summarize_sq:
        rec = summarize_sq(a.summarize_sq, a.command)
        with open(SQ_FILE, "w") as f:
            json.dump(rec, f, indent=1)
        print(json.dumps(rec))
        return
    if a.summarize_stats:
        txt = summarize_stats(a.summarize_stats, a.command[0] if a.command else "")
        with open(STATS_FILE, "w") as f:
            f.write(txt)
        print(txt)
        return
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures one GPU only (no multi-GPU path); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_31248_amd import binding as Bd
    from paper_2606_31248_amd import inputs as I
    from paper_2606_31248_amd import pipeline as Pp

    Bd.load()
    t_start = time.perf_counter()
    _done("library load", t_start)
    wl = I.FACE_ROLLOUT
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    nty, ntx, sy, sx = wl.tiling
    Hf = (nty - 1) * sy + wl.H
    Wf = (ntx - 1) * sx + wl.W
    window = (wl.kz, wl.ky, wl.kx)

    def to_dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)

    qkv_host = wl.qkv()
    q, k, v = (to_dev(x) for x in qkv_host)
    pl = wl.placement()
    geom = Pp.TileGeometry(*(torch.from_numpy(x).to(dev) for x in pl.as_int32()))
    win = torch.from_numpy(I.ramp_window_2d(wl.H, wl.W, I.FACE_OVERLAP)).to(dev)
    coords = torch.empty((wl.B, wl.H, wl.W, 2), dtype=torch.float32, device=dev)
    cs = torch.empty((wl.B, wl.H, wl.W, wl.d // 2, 2), dtype=torch.float32, device=dev)
    out = torch.empty_like(q)
    face = torch.empty((wl.heads * wl.Z, Hf, Wf, wl.d), dtype=torch.bfloat16, device=dev)
    desc = Bd.desc_for(q, window, wl.scale)

    if a.calib_copy:
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev).fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    ev = {n: [] for n in ("coords", "na", "blend")}
    planes = out.view(wl.B, wl.heads * wl.Z, wl.H, wl.W, wl.d)

    def step(record: bool):
        st = torch.cuda.current_stream()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)] if record else None
        if record:
            e[0].record(st)
        Bd.strata_stereo_coords(geom.face, geom.oy, geom.ox, wl.H, wl.W, geom.face_cells, geom.patch,
                                0.0, coords)
        Bd.strata_stereorope_phases(coords, wl.d, Pp.ROPE_BASE, cs)
        if record:
            e[1].record(st)
        Bd.strata_na3d_fwd_stitch(desc, None, q, k, v, cs, out, None, nty, ntx, sy, sx, win, face)
        if record:
            e[2].record(st)
        Bd.strata_tile_blend_overlap(planes, nty, ntx, sy, sx, win, face)
        if record:
            e[3].record(st)
            ev["coords"].append((e[0], e[1]))
            ev["na"].append((e[1], e[2]))
            ev["blend"].append((e[2], e[3]))

    for _ in range(a.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        step(True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / a.steps
    avg = {n: float(np.mean([s.elapsed_time(e) for s, e in lst])) for n, lst in ev.items()}
    _done("face-rollout step", t_start)
    # the timed step's own output at the sampled cells (checked against the oracle in the CPU leg)
    cells = face_sample_cells(wl)
    cidx = torch.from_numpy((cells[0] * Hf + cells[1]) * Wf + cells[2]).to(dev)
    face_rows = face.view(-1, wl.d).index_select(0, cidx).float().cpu().numpy().astype(np.float64)

    flops = 4.0 * wl.B * wl.heads * wl.N * wl.K * wl.d
    tflops_step = flops / (ms_step * 1e-3) / 1e12
    tflops_na = flops / (avg["na"] * 1e-3) / 1e12
    alg_bytes = 4.0 * wl.B * wl.heads * wl.N * wl.d * 2        # Q, K, V read + O write, bf16
    gbs_na = alg_bytes / (avg["na"] * 1e-3) / 1e9
    blend_bytes = overlap_stitch_bytes(nty, ntx, wl.H, wl.W, sy, sx, wl.heads * wl.Z, wl.d)
    traffic, pmc = stored_traffic(alg_bytes)
    tokens = wl.B * wl.N

    res = {
        "metric": METRIC,
        "value": round(tflops_step, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded iid N(0,1) Q/K/V; analytic equiangular cubed-sphere tile geometry)",
        "config": {"workload": wl.name, "tiles": wl.B, "heads": wl.heads, "Z": wl.Z, "H": wl.H,
                   "W": wl.W, "head_dim": wl.d, "window": list(window), "face_tokens": [Hf, Wf],
                   "tile_stride": [sy, sx], "overlap": I.FACE_OVERLAP, "blend_window": "linear ramp",
                   "stitch": "fused: the forward stores the cells one tile covers, then the overlap-only stitch"},
        "tokens_per_s": round(tokens / (ms_step * 1e-3), 1),
        "face_tokens_per_s": round(wl.Z * Hf * Wf / (ms_step * 1e-3), 1),
        "pct_bf16_peak": round(100.0 * tflops_step / PEAK_BF16_TFLOPS, 2),
        "kernels_ms": {k2: round(v2, 4) for k2, v2 in avg.items()},
        "na3d_fwd": {"tflops": round(tflops_na, 2), "pct_bf16_peak": round(100 * tflops_na / PEAK_BF16_TFLOPS, 2),
                     "hbm_gbs_algorithmic": round(gbs_na, 1)},
        "blend": {"gbs_algorithmic": round(blend_bytes / (avg["blend"] * 1e-3) / 1e9, 1)},
        "roofline": {"bound": "hbm", "achieved": round(gbs_na, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs_na / PEAK_HBM_GBS, 4),
                     "traffic": None if traffic is None else float(traffic),
                     "kernel": f"strata_na3d_fwd_stitch ({FWD_KERNEL})", "alg_bytes_per_launch": alg_bytes},
    }
    # every row of the hot path against the roofline that bounds it
    res["rows"] = {
        "a1_a2_coords_phases": {"ms": round(avg["coords"], 4), "bound": "alu (fp64 geometry)"},
        "a3_a6_na3d_fwd_face": dict(roofline_row(flops, alg_bytes, avg["na"]), achieved_gbs=round(gbs_na, 1),
                                    frac_hbm=round(gbs_na / PEAK_HBM_GBS, 4)),
        "a8_tile_blend_face": {"bound": "hbm", "achieved_gbs": round(blend_bytes / (avg["blend"] * 1e-3) / 1e9, 1),
                               "frac_hbm": round(blend_bytes / (avg["blend"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
    }
    if a.train_steps > 0:
        # the same step without the fusion: every tile output written, then the whole stitch
        full_bytes = (wl.B * wl.heads * wl.Z * wl.H * wl.W * wl.d + wl.heads * wl.Z * Hf * Wf * wl.d) * 2
        na_plain = _timed(lambda: Bd.strata_na3d_fwd(desc, q, k, v, cs, out, None), a.train_steps)
        bl_full = _timed(lambda: Bd.strata_tile_blend(planes, nty, ntx, sy, sx, win, face), a.train_steps)
        res["face_step_unfused"] = {
            "na3d_fwd_ms": round(na_plain, 4), "tile_blend_ms": round(bl_full, 4),
            "tile_blend_gbs": round(full_bytes / (bl_full * 1e-3) / 1e9, 1),
            "step_ms": round(avg["coords"] + na_plain + bl_full, 4)}
        _done("unfused face step", t_start)
        # the attention-block options (App. B.5) on the same face forward
        opt = options_face_fwd(wl, desc, q, k, v, cs, out, a.train_steps)
        res["options"] = {"face_fwd": opt}
        res["rows"]["f1_qk_norm_gate_fwd_face"] = opt["norm_gate_d"]
        _done("options face forward", t_start)
        del q, k, v, out, face, coords, cs
        torch.cuda.empty_cache()
        tt = train_tile(a.train_steps)
        res["rows"]["a3_a6_na3d_fwd_train_tile"] = roofline_row(*tt.pop("_fwd"))
        res["rows"]["a7_na3d_bwd_train_tile"] = roofline_row(*tt.pop("_bwd"))
        res["rows"]["a2_rope_apply_train_tile"] = {"bound": "hbm", "achieved_gbs": tt["rope_apply_qk"]["gbs"],
                                                   "frac_hbm": tt["rope_apply_qk"]["frac_hbm"]}
        res["train_tile"] = tt
        _done("training tile", t_start)
        torch.cuda.empty_cache()
        res["options"]["train_tile_bwd"] = options_train_bwd(a.train_steps)
        res["rows"]["f1_qk_norm_gate_bwd_train_tile"] = res["options"]["train_tile_bwd"]["norm_gate_d"]
        _done("options backward", t_start)
        torch.cuda.empty_cache()
        ps = paper_shapes(a.train_steps)
        res["paper_shapes"] = ps
        res["rows"]["f2_na3d_fwd_w999_paper_tile16"] = ps[I.PAPER_TILE16.name]["fwd"]
        res["rows"]["f2_na3d_bwd_w999_paper_tile16"] = ps[I.PAPER_TILE16.name]["bwd"]
        res["rows"]["f2_na3d_fwd_w377_z24"] = ps[I.Z24_TILE.name]["fwd"]
        res["rows"]["f2_column_fwd_paper"] = ps[I.PAPER_COLUMN.name]["fwd"]
        res["rows"]["f2_na3d_fwd_d128_decoder"] = ps[I.PAPER_DECODER.name]["fwd"]
        res["rows"]["f2_na3d_bwd_d128_decoder"] = ps[I.PAPER_DECODER.name]["bwd"]
        res["rows"]["f1_f2_decoder_norm_gate_fwd"] = ps[I.PAPER_DECODER.name]["fwd_norm_gate_d"]
        res["rows"]["f1_f2_decoder_norm_gate_bwd"] = ps[I.PAPER_DECODER.name]["bwd_norm_gate_d"]
        _done("paper shapes", t_start)
        torch.cuda.empty_cache()
        res["rows"]["f4_wind_tile_frame_face"] = wind_frame(a.train_steps)
        _done("wind frame", t_start)
        torch.cuda.empty_cache()
        res["rows"]["f3_duo_pad_faces"] = duo_padding(a.train_steps)
        _done("duo padding", t_start)
    if a.train_steps <= 0:
        del q, k, v, out, face, coords, cs
        torch.cuda.empty_cache()
    runs = None
    if a.config_steps > 0:
        runs = config_runs(a.config_steps)
        _done("configs C1-C4", t_start)
    if a.cpu_tiles > 0:
        # CPU leg: the oracle timed on a sample, and evaluated on the outputs sampled above
        import oracle
        res["parity"] = face_parity(wl, qkv_host, face_rows, cells, I.ramp_window_2d(wl.H, wl.W, I.FACE_OVERLAP))
        _done("face parity", t_start)
        res["cpu_baseline"] = cpu_baseline(wl, a.cpu_tiles)
        res["cpu_baseline"]["host_cpus"] = os.cpu_count()
        res["cpu_baseline"]["one_thread"] = cpu_one_thread()
        _done("cpu baseline", t_start)
        if runs is not None:
            par = config_parity(runs)
            _done("config parity", t_start)
    if runs is not None:
        res["configs"] = {}
        for key, r in runs.items():
            ent = {k2: v2 for k2, v2 in r.items() if not k2.startswith("_")}
            if a.cpu_tiles > 0:
                ent["parity"] = par[key]
            res["configs"][key] = ent
        c5 = {"workload": wl.name, "ms": round(ms_step, 4), "tflops": round(tflops_step, 2),
              "tokens_per_s": round(tokens / (ms_step * 1e-3), 1), "roofline": res["roofline"],
              "note": "the timed face step of this line (value)"}
        if "parity" in res:
            c5["parity"] = res["parity"]
        res["configs"]["C5"] = c5
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

"""Build libstrata.so (HIP, gfx950) in-tree with hipcc.

Usage: python -m paper_2606_31248_amd.build [--force] [-j N]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libstrata.so")

SOURCES = ["api.hip", "geometry.hip", "rope.hip", "blend.hip", "na3d_ref.hip", "na3d_opts.hip", "na3d_col.hip", "duo.hip", "na3d_mfma_q.hip",
           "na3d_mfma_kv.hip", "na3d_mfma_kvp.hip", "na3d_fwd_zs.hip", "na3d_fwd_lsg.hip", "na3d_mfma_d128.hip",
           "na3d_bwd_d128.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-FP32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
    "-I", INCLUDE, "-I", CSRC,
]


# Per-file extra flags.  The attention kernel never sees NaN inputs by contract
# (masked logits are -inf, not NaN), so max() needs no NaN canonicalisation.
EXTRA = {"na3d_mfma_q.hip": ["-fno-honor-nans"], "na3d_mfma_d128.hip": ["-fno-honor-nans"], "na3d_bwd_d128.hip": ["-fno-honor-nans"], "na3d_col.hip": ["-fno-honor-nans"], "na3d_mfma_kv.hip": ["-fno-honor-nans"], "na3d_mfma_kvp.hip": ["-fno-honor-nans"],
         # the level-sweep forward: MFMA accumulators in VGPRs, so that the logits the
         # softmax reads are not routed through AGPRs
         "na3d_fwd_zs.hip": ["-fno-honor-nans", "-mllvm", "-amdgpu-mfma-vgpr-form=1"],
         "na3d_fwd_lsg.hip": ["-fno-honor-nans", "-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + FLAGS + EXTRA.get(src, []) + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    # the host pass does not know the packed-fp32 feature and says so; keep other warnings
    noise = "'-packed-fp32-ops' is not a recognized feature"
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if noise not in ln and ln.strip()]
    if msgs:
        print("\n".join(msgs), file=sys.stderr)
    return obj


def build(jobs: int = 8) -> str:
    """Compile every HIP source and link libstrata.so next to this file."""
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(SOURCES)))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=8)
    a = ap.parse_args()
    print(build(a.j))

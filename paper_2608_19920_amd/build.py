"""Build libh2o.so (HIP, gfx950) in-tree.

    python -m paper_2608_19920_amd.build

Every call recompiles all sources (one hipcc process per source, in
parallel) into ``_build/`` and links ``libh2o.so`` next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libh2o.so")
BUILD = os.path.join(os.path.dirname(HERE), "_build")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # packed FP32 VALU ops are left out of the device code on purpose
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
# Per-source additions. The MFMA kernels keep their accumulators in VGPRs:
# the scores are read by VALU code every tile, and AGPR accumulators would be
# copied back and forth. The prefill kernels never see a NaN (masked scores
# are -inf), so max() needs no NaN quieting.
FILE_FLAGS = {
    "decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "sdpa_mfma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans"],
    "backward_mfma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def flags_for(src: str):
    return FLAGS + FILE_FLAGS.get(os.path.basename(src), [])


def _quiet(text: str) -> str:
    keep = [ln for ln in text.splitlines()
            if "not a recognized feature for this target" not in ln]
    return "\n".join(keep)


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *flags_for(src), "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = _quiet(r.stdout + r.stderr).strip()
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msg}")
    if msg:
        print(msg, file=sys.stderr)
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + _quiet(r.stdout + r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()

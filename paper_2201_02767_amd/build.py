"""Build the HIP library ``libqta.so`` for gfx950 (in-tree, next to this file).

Every kernel source is compiled with hipcc for gfx950 only; the host C ABI is compiled in the same
invocation style and linked into one shared library. Packed-fp32 instruction selection is turned
off for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "libqta.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(HERE, '..', 'include')}",
]


# The attention kernels (forward and backward) never see a NaN (finite inputs; masked logits are
# -inf and are selected away before use), so their max reductions may skip the NaN-quieting the
# IEEE mode asks for, which lets each butterfly step fuse into one DPP max.
NO_NAN_SOURCES = {"fine.hip", "coarse.hip", "backward.hip", "coarse_bwd.hip"}

# The fine kernels and the backward query pass keep one accumulator per 16-slot tile; with the MFMA
# results in VGPRs instead of AGPRs (the compiler's default) they hold the same values in fewer
# registers in total, which keeps 8 waves per SIMD for 64 slots in the forward and raises the
# 128- and 256-slot instantiations, and the 64-slot backward query passes, by one or two.
MFMA_VGPR_SOURCES = {"fine.hip", "backward.hip"}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    extra = ["-fno-honor-nans"] if os.path.basename(src) in NO_NAN_SOURCES else []
    if os.path.basename(src) in MFMA_VGPR_SOURCES:
        extra += ["-mllvm", "-amdgpu-mfma-vgpr-form"]
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(sources))) as ex:
        objs = list(ex.map(_compile, sources))
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print("built", LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)

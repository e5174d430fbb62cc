"""Build libdeer.so (HIP, gfx950) in-tree: one hipcc job per translation unit, then link.

    python -m paper_2605_12683_amd.build [--force]
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdeer.so")
SOURCES = ["deer_api.hip", "k_plrnn.hip", "k_diag.hip", "k_dense.hip", "k_shallow.hip", "k_readout.hip", "k_seq.hip", "k_quasi.hip", "k_small.hip", "k_train.hip", "deer_noalloc.hip", "k_obs.hip", "k_big.hip", "k_shfused.hip"]
HEADERS = ["common.h", "launch.h", "newton_ctl.h", "row16.h", os.path.join("..", "..", "include", "deer.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # every multiply-add in the kernels is either an explicit fmaf or deliberately unfused
    "-ffp-contract=off",
    # no packed-fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the chunk kernels apply VALU operations to
    # them every step, which would otherwise cost two accumulator moves per element
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wno-unused-result",
]


def _newest_header() -> float:
    return max(os.path.getmtime(os.path.join(CSRC, h)) for h in HEADERS)


def _compile(src: str, force: bool) -> str:
    out = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    path = os.path.join(CSRC, src)
    if not force and os.path.exists(out) and os.path.getmtime(out) >= max(os.path.getmtime(path), _newest_header()):
        return out
    cmd = [HIPCC, *FLAGS, "-c", path, "-o", out + ".tmp"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def build(force: bool = True, verbose: bool = False) -> str:
    """Compile every translation unit for gfx950 and link libdeer.so; returns its path."""
    os.makedirs(OBJ, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda s: _compile(s, force), SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], check=True)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(force="--force" in sys.argv, verbose=True)

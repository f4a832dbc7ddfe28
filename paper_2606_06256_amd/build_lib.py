"""Build libsegpa.so (HIP kernels + C-ABI host code) for gfx950 with hipcc.

Usage: python -m paper_2606_06256_amd.build_lib   (or build() from Python).
Objects go to paper_2606_06256_amd/_build/, the library next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsegpa.so")

SOURCES = ["api.cpp", "append.hip", "decode.hip", "mass.hip", "prefill.hip", "rope.hip", "select.hip", "summary.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def common_flags() -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
            # packed FP32 instructions stay disabled in device code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC]


# per-source extra flags: matrix-core accumulators in ordinary VGPRs (the
# decode kernel rescales them every tile; AGPR accumulators cost a copy each way)
EXTRA = {"decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
         # no NaN operands reach the prefill arithmetic (masked keys are -inf
         # by selection, stale slots are zeroed), so max needs no quieting
         "prefill.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans"]}


def _compile(src: str, flags: list[str] = ()) -> str:
    sub = "poison" if flags else ""
    out = os.path.join(BUILD, sub, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *common_flags(), *EXTRA.get(src, []), *flags, "-c", os.path.join(CSRC, src),
           "-o", out]
    if src.endswith(".cpp"):
        cmd.insert(1, "-xhip")
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return out


# Debug build of the same sources: key and value slots in LDS are filled with
# NaN before their copies (the kernels that stage tiles through LDS), so a
# read that is not ordered after its copy corrupts the result visibly.
POISON_LIB = os.path.join(HERE, "libsegpa_poison.so")
POISON_FLAGS = ["-DSEGPA_LDS_POISON"]


def _link(objs: list[str], lib: str) -> None:
    tmp = lib + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False, poison: bool = True) -> str:
    """Builds libsegpa.so and (poison=True) the LDS-poison debug library."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = [(s, []) for s in SOURCES]
    if poison:
        os.makedirs(os.path.join(BUILD, "poison"), exist_ok=True)
        jobs += [(s, POISON_FLAGS) for s in SOURCES]
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(lambda j: _compile(*j), jobs))
    _link(objs[:len(SOURCES)], LIB)
    if verbose:
        print("built", LIB)
    if poison:
        _link(objs[len(SOURCES):], POISON_LIB)
        if verbose:
            print("built", POISON_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

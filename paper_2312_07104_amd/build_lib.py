"""Builds the native library of this package in-tree.

``libradixattn.so``: the host radix cache (C++) and the gfx950 HIP kernels
behind the C ABI in ``include/radixattn.h``.  All HIP code is compiled with
packed fp32 instructions disabled.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build", "radixattn")
LIB = os.path.join(HERE, "libradixattn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function", f"-I{ROOT}/include", f"-I{CSRC}"]
# -mno-amdgpu-ieee with -fno-honor-nans: the kernels never produce or test
# NaNs (masked scores are -inf), so max/min need no operand canonicalisation.
HIP_ONLY = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-mno-amdgpu-ieee", "-fno-honor-nans"]


# Per-source extra flags.  extend.hip keeps the compiler's own MFMAs in VGPR
# form (the prologue's S^T, read by the VALU) although the kernel holds Q^T
# and the O^T accumulators in AGPRs through inline assembly.
EXTRA = {"extend.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r


def sources():
    out = []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".cpp")):
            out.append(os.path.join(CSRC, f))
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs, cmds = [], []
    for src in sources():
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        objs.append(obj)
        if src.endswith(".hip"):
            cmds.append([HIPCC, *COMMON, *HIP_ONLY, *EXTRA.get(os.path.basename(src), []), "-c", src, "-o", obj])
        else:
            # Host sources still go through hipcc for the HIP runtime headers;
            # name the target so no default-architecture code object is made.
            cmds.append([HIPCC, *COMMON, f"--offload-arch={ARCH}", "-c", src, "-o", obj])
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        for r in ex.map(_run, cmds):
            if verbose and (r.stdout or r.stderr):
                print(r.stdout + r.stderr, file=sys.stderr)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

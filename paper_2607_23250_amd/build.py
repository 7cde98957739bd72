"""Build the C-ABI library ``liblibra.so`` in-tree for gfx950.

``python -m paper_2607_23250_amd.build`` (or ``build()``) compiles the host
planner with g++ and the HIP sources with hipcc, then links one shared
library next to this file.  Objects go to ``_build/``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "liblibra.so")

HIP_SOURCES = ["attn_fwd.hip", "attn_bwd.hip", "attn_bwd_dq.hip", "attn_api.hip", "mfma_loop.hip"]
CXX_SOURCES = ["plan.cpp", "vrsp.cpp"]
ARCH = os.environ.get("LIBRA_OFFLOAD_ARCH", "gfx950")


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# Per-source extra flags.  The forward and dK / dV kernels take the MFMA
# results that the VALU reads (S, dP) in VGPRs; the default heuristic lands
# them in AGPRs and copies every element out before use.  The compiler still
# keeps the long-lived dK / dV accumulators in AGPRs.  The dQ kernel stays in
# the default form: in VGPR form it runs out of registers for its LDS reads.
_VGPR_FORM = ["-mllvm", "--amdgpu-mfma-vgpr-form=1"]
EXTRA_FLAGS = {
    "attn_fwd.hip": _VGPR_FORM,
    "attn_api.hip": _VGPR_FORM,
    "attn_bwd.hip": _VGPR_FORM,
}


def hip_flags(src: str = ""):
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-munsafe-fp-atomics",
            # no packed-fp32 instructions anywhere in the device code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            f"-I{INCLUDE}", f"-I{CSRC}"] + EXTRA_FLAGS.get(src, [])


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n"
                           f"{res.stdout}\n{res.stderr}")
    return res


def build(verbose: bool = False, jobs: int = 4) -> str:
    """Compile every source and link ``liblibra.so``; returns its path."""
    os.makedirs(OUT_DIR, exist_ok=True)
    hipcc = _hipcc()
    cmds, objs = [], []
    for src in CXX_SOURCES:
        obj = os.path.join(OUT_DIR, src + ".o")
        cmds.append(["g++", "-O2", "-std=c++17", "-fPIC", "-Wall", f"-I{INCLUDE}", f"-I{CSRC}",
                     "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HIP_SOURCES:
        obj = os.path.join(OUT_DIR, src + ".o")
        cmds.append([hipcc] + hip_flags(src) + ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    procs = []
    for cmd in cmds:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                            text=True)))
        while sum(p.poll() is None for _, p in procs) >= jobs:
            procs[0][1].wait(timeout=600)
    errors = []
    for cmd, p in procs:
        out, err = p.communicate(timeout=900)
        if p.returncode != 0:
            errors.append(f"{' '.join(cmd)}\n{out}\n{err}")
    if errors:
        raise RuntimeError("build failed:\n" + "\n".join(errors))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs, verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

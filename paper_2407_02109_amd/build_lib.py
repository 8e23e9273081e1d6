"""Build libfla_swin.so in-tree with hipcc for gfx950.

Run as ``python -m paper_2407_02109_amd.build_lib``; ``__graft_entry__.build()`` calls
``build()``.  Always recompiles: the output replaces the library atomically."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
SOURCES = ["fla_swin_api.cpp", "fla_swin_bf16.hip", "fla_swin_f32.hip", "fla_swin_bwd_bf16_window.hip",
           "fla_swin_bwd_bf16_blocks.hip", "fla_swin_bwd_f32.hip", "fla_swin_scratch.hip", "fla_cycle_scan.hip"]
LIB = os.path.join(PKG, "libfla_swin.so")

# -packed-fp32-ops: keep the compiler from forming packed fp32 ALU instructions.
# -fno-honor-nans: inputs are finite; lets max reductions skip NaN canonicalisation
# (infinities, which the masking relies on, stay honoured).
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-fno-honor-nans",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, extra_flags=()) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIP_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (res.stdout + res.stderr).splitlines()
            if "packed-fp32-ops" not in l or "error" in l]
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

"""Builds libmbe.so (the C-ABI HIP library) in-tree for gfx950 with hipcc.

    python -m paper_2607_22663_amd.build              # libmbe.so
    python -m paper_2607_22663_amd.build --timeline   # also libmbe_timeline.so

libmbe_timeline.so is a profiling build of the same sources with
-DMBE_TIMELINE: the attention kernel records a per-workgroup phase timeline
(read with mbe_timeline_read; bench.py --timeline).  Nothing else loads it.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmbe.so")
TIMELINE_LIB = os.path.join(PKG, "libmbe_timeline.so")
SOURCES = ["abi.cpp", "edit_select.hip", "attn_window.hip", "block_select.hip", "kv_write.hip", "noalloc.hip"]

# Packed fp32 VALU ops are disabled for every HIP source: ordinary float code
# is compiled to scalar-per-lane v_*_f32 instructions only.  MFMA results are
# allocated in ordinary VGPRs where possible (the softmax reads the score
# accumulators with VALU instructions every tile; AGPR results would need a
# copy each time).
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-result",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, timeline: bool = False) -> str:
    """Builds libmbe.so, or with timeline=True the profiling build
    libmbe_timeline.so; returns the path."""
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    lib = TIMELINE_LIB if timeline else LIB
    tmp = lib + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *(["-DMBE_TIMELINE"] if timeline else []), "-I", os.path.join(ROOT, "include"),
           "-o", tmp, *srcs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "is not a recognized feature for this target" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{out}")
    if verbose and out.strip():
        print(out)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    if "--timeline" in sys.argv:
        print(build(verbose="-v" in sys.argv, timeline=True))

"""Build the HIP library in-tree with hipcc for gfx950.

    python -m paper_2510_12633_amd.build

produces paper_2510_12633_amd/liblaminar_decode_attn.so next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "liblaminar_decode_attn.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)

SOURCES = [os.path.join(CSRC, "decode_attn.hip"),
           os.path.join(CSRC, "attn_entry.hip"), os.path.join(CSRC, "calibrate.hip"),
           os.path.join(CSRC, "kv_append.hip"), os.path.join(CSRC, "kv_pack.hip"), os.path.join(CSRC, "migrate.hip"),
           os.path.join(CSRC, "linear.hip"), os.path.join(CSRC, "decode_step.hip"),
           os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "repack.cpp")]

# Packed fp32 VALU forms are switched off for all device code.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-function"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"),
                 "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile the shared library (always recompiles); return its path."""
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC,
           *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature: drop that note.
    err = "\n".join(l for l in res.stderr.splitlines()
                    if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))

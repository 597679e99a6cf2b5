"""Build libdiffopt.so (the HIP library behind include/diffopt.h) for gfx950.

    python paper_2211_06934_amd/build.py          # compile in-tree

Run it as a file (or through __graft_entry__.build()): importing the package
loads the library, so the build must not go through the package.

The shared library lands next to this file so that it travels with the
source tree.  Extra preprocessor definitions (tile sizes, streaming loads)
can be passed as ``defines`` for tuning builds written elsewhere.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdiffopt.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -packed-fp32-ops: keep the compiler from forming packed fp32 VALU ops.
HIPFLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(out: str = LIB, defines=(), verbose: bool = False) -> str:
    """Compile every csrc/*.hip into one shared library; returns its path."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *HIPFLAGS, "-I", INCLUDE, "-I", CSRC,
           *["-D%s" % d for d in defines], *sources(), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building %s" % out)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

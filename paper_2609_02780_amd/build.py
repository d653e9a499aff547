"""Build ``libshallowstream.so`` for gfx950 with hipcc, in-tree.

    python -m paper_2609_02780_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB_NAME = "libshallowstream.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
SOURCES = [os.path.join(CSRC, "ss_kernels.hip"), os.path.join(CSRC, "ss_api.cpp")]
ARCH = "gfx950"

# Packed fp32 VALU ops are kept out of every kernel (hipcc would otherwise form
# them from ordinary float code).
HIPCC_FLAGS = ["-O3", "-fPIC", "-shared", "-std=c++17", f"--offload-arch={ARCH}",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the library)")


def build_library(verbose: bool = False) -> str:
    """Compile the HIP sources into ``LIB_PATH`` (always recompiles)."""
    fd, tmp = tempfile.mkstemp(prefix=".libshallowstream.", suffix=".so.tmp", dir=HERE)
    os.close(fd)
    cmd = [hipcc(), *HIPCC_FLAGS, *SOURCES, "-o", tmp]
    try:
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + res.stdout + res.stderr)
        if verbose:
            print(" ".join(cmd))
        os.replace(tmp, LIB_PATH)
    finally:
        if os.path.exists(tmp):
            os.unlink(tmp)
    return LIB_PATH


if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv))

"""Build libpic_attn.so in-tree with hipcc for gfx950.

    python -m paper_2606_13126_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpic_attn.so")
SOURCES = [os.path.join(CSRC, "pic_kernels.hip"), os.path.join(CSRC, "pic_host.cpp"),
           os.path.join(CSRC, "pic_cache.cpp")]

# -packed-fp32-ops is a device feature: hipcc's host pass warns that it does not
# know it, which is harmless.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, extra: list | None = None) -> str:
    """Compile every source into libpic_attn.so (always recompiles)."""
    fd, tmp = tempfile.mkstemp(prefix="libpic_attn.", suffix=".so.tmp", dir=PKG)
    os.close(fd)
    cmd = [hipcc()] + FLAGS + (extra or []) + SOURCES + ["-o", tmp]
    try:
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + res.stdout + res.stderr)
        if verbose:
            print(" ".join(cmd))
        os.replace(tmp, LIB)
    finally:
        if os.path.exists(tmp):
            os.remove(tmp)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

"""Build libevisel.so for gfx950 with hipcc (in-tree, next to this file).

Usage: ``python -m paper_2608_05780_amd.build`` or ``build()`` from Python.
Always recompiles. The host plan builder is part of the same library; CPU-only
tests load it and call only the host entry points.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libevisel.so")
SOURCES = ["api.hip", "attn.hip", "attn_pipe.hip", "evidence.hip", "select.hip",
           "plan.cpp"]
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 VALU instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc",
              shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    cmd = [hipcc(), *HIP_FLAGS, "-shared", "-o", LIB + ".tmp",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    for s in SOURCES:
        p = os.path.join(CSRC, s)
        if s.endswith(".cpp"):
            cmd += ["-x", "hip", p]      # compiled by the same driver
        else:
            cmd += [p]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + out)
    if verbose and out.strip():
        print(out)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

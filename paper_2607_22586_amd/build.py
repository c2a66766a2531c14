"""Builds libmmshiftkv.so (gfx950) in-tree with hipcc.

    python -m paper_2607_22586_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmmshiftkv.so")
SOURCES = ["api.hip", "proxies.hip", "score.hip", "select.hip", "gather.hip", "hidden.hip", "decode.hip", "baselines.hip"]
HEADERS = ["common.hpp", "kernels.hpp", "normal.hpp"]
ARCH = "gfx950"

# Packed fp32 VALU instructions are disabled for every device compilation.
HIPCC_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", "--offload-arch=" + ARCH,
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-mllvm", "-amdgpu-mfma-vgpr-form",
               "-fno-fast-math", "-Wall", "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    """Compile every HIP source into the shared library (always recompiles)."""
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + ["-I" + os.path.join(os.path.dirname(HERE), "include"),
                                     "-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + msgs)
    if verbose and msgs.strip():
        print(msgs, flush=True)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    deps = SOURCES + HEADERS
    inc = os.path.join(os.path.dirname(HERE), "include", "mmshiftkv.h")
    return any(os.path.getmtime(os.path.join(CSRC, s)) > t for s in deps) or os.path.getmtime(inc) > t


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

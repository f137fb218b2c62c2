"""Build the gfx950 HIP library in-tree: ``python -m paper_2607_17979_amd.build``.

Produces ``paper_2607_17979_amd/libgdn_mi355x.so`` from ``csrc/`` with hipcc.
All device code is compiled with packed-fp32 instruction generation disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_NAME = "libgdn_mi355x.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
SOURCES = ["csrc/gdn_api.cpp", "csrc/gdn_decode.hip", "csrc/gdn_prefill.hip", "csrc/gdn_prefill_pipe.hip",
           "csrc/gdn_recur.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def compile_flags():
    return [
        f"--offload-arch={ARCH}",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-fvisibility=hidden",
        "-Wall",
        "-Wno-unused-function",
        "-Wshadow",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"),
    ]


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link the shared library.  Always
    recompiles.  Returns the library path; raises CalledProcessError on error."""
    srcs = [os.path.join(HERE, s) for s in SOURCES]
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), *compile_flags(), "-shared", "-x", "hip", *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(line for line in (res.stdout + res.stderr).splitlines()
                    if "packed-fp32-ops" not in line)
    if res.returncode != 0:
        sys.stderr.write(out + "\n")
        raise subprocess.CalledProcessError(res.returncode, cmd, output=out)
    if verbose and out.strip():
        print(out)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))

"""Build libstepq.so in-tree with hipcc for gfx950."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libstepq.so")
SOURCES = ["stepq_host.hip", "stepq_kernels.hip", "stepq_setup.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 VALU forms stay off: scalar fp32 only on the device
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def build(extra_flags: list[str] | None = None, out: str = LIB, verbose: bool = False) -> str:
    hip = [os.path.join(CSRC, s) for s in SOURCES if s.endswith(".hip")]
    cpp = [os.path.join(CSRC, s) for s in SOURCES if s.endswith(".cpp")]
    srcs = hip + ["-x", "c++"] + cpp      # plain host C++ last
    tmp = out + ".tmp"
    cmd = [HIPCC] + FLAGS + (extra_flags or []) + ["-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd, cwd=CSRC)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

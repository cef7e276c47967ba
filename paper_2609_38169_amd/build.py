"""Build libstepq.so in-tree for gfx950.

Each source is compiled on its own (the .hip files with hipcc for gfx950,
the host-only setup code with g++) and the objects are linked by hipcc.
Mixing a `-x c++` source into one hipcc command makes hipcc drop
--offload-arch and fall back to its default target, so the link step is
followed by a check that the library's device bundle is gfx950 and only
gfx950.
"""
from __future__ import annotations

import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libstepq.so")
HIP_SOURCES = ["stepq_host.hip", "stepq_kernels.hip", "stepq_refit.hip", "stepq_rowmax.hip"]
CXX_SOURCES = ["stepq_setup.cpp", "stepq_plan.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU forms stay off: scalar fp32 only on the device
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the decode bodies then fit
    # 64 registers (8 waves per SIMD) without a separate AGPR block
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-pthread"]


def device_targets(path: str) -> list[str]:
    """Offload targets named in a built library's device bundle."""
    data = open(path, "rb").read()
    return sorted(set(t.decode() for t in re.findall(rb"hipv4-amdgcn-amd-amdhsa--(gfx[0-9a-f]+)", data)))


def build(extra_flags: list[str] | None = None, out: str = LIB, verbose: bool = False, csrc: str = CSRC,
          build_dir: str = BUILD_DIR) -> str:
    os.makedirs(build_dir, exist_ok=True)
    objs = []

    def run(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, cwd=csrc, stderr=subprocess.PIPE, text=True)
        # hipcc's host pass does not know the device-only feature flag; drop that note
        for line in r.stderr.splitlines():
            if "packed-fp32-ops' is not a recognized feature" not in line:
                print(line, file=sys.stderr)
        if r.returncode != 0:
            raise subprocess.CalledProcessError(r.returncode, cmd)

    inc = ["-I", os.path.join(ROOT, "include"), "-I", csrc]
    cmds = []
    for s in HIP_SOURCES:
        o = os.path.join(build_dir, s + ".o")
        cmds.append([HIPCC] + HIP_FLAGS + (extra_flags or []) + inc + ["-c", os.path.join(csrc, s), "-o", o])
        objs.append(o)
    for s in CXX_SOURCES:
        o = os.path.join(build_dir, s + ".o")
        cmds.append(["g++"] + CXX_FLAGS + inc + ["-c", os.path.join(csrc, s), "-o", o])
        objs.append(o)
    # the translation units are independent: compile them side by side
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        for f in [ex.submit(run, c) for c in cmds]:
            f.result()
    out = os.path.abspath(out)
    tmp = out + ".tmp"
    run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-pthread", "-o", tmp] + objs)
    targets = device_targets(tmp)
    if targets != [ARCH]:
        os.remove(tmp)
        raise RuntimeError(f"libstepq device bundle targets {targets}, expected only {ARCH}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

"""Build libgefen.so (HIP, gfx950) in-tree.

Every kernel's register and scratch use is taken from the compiler's
kernel-resource-usage remarks and written next to the library
(``libgefen.resources.txt``); a kernel that spills to scratch fails the build, since a
spill turns the HBM-bound step into a scratch-memory-bound one.
"""
from __future__ import annotations

import glob
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libgefen.so")
RES = os.path.join(HERE, "libgefen.resources.txt")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Rpass-analysis=kernel-resource-usage",
    "-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib",
]


def _parse_resources(log: str):
    """Per-kernel (name, vgpr, agpr, sgpr, scratch, occupancy) from the remarks."""
    kernels = {}
    cur = None
    for line in log.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            kernels[cur] = {}
            continue
        if cur is None:
            continue
        for key, pat in (("vgpr", r"VGPRs: (\d+)"), ("agpr", r"AGPRs: (\d+)"),
                         ("sgpr", r"SGPRs: (\d+)"),
                         ("scratch", r"ScratchSize \[bytes/lane\]: (\d+)"),
                         ("occupancy", r"Occupancy \[waves/SIMD\]: (\d+)"),
                         ("lds", r"LDS Size \[bytes/block\]: (\d+)")):
            m = re.search(pat, line)
            if m:
                kernels[cur][key] = int(m.group(1))
    return kernels


def build(verbose: bool = False) -> str:
    srcs = sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))
    tmp = LIB + ".tmp"
    cmd = [HIPCC] + FLAGS + ["-I", os.path.join(ROOT, "include"),
                             "-I", os.path.join(HERE, "csrc")] + srcs + ["-o", tmp]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    log = proc.stdout + proc.stderr
    if proc.returncode != 0:
        sys.stderr.write(log)
        raise RuntimeError("hipcc failed building libgefen.so")
    kernels = _parse_resources(log)
    lines = ["# kernel  vgpr  agpr  sgpr  scratch_bytes_per_lane  lds_bytes  occupancy_waves_per_simd"]
    spills = []
    for name in sorted(kernels):
        k = kernels[name]
        lines.append(f"{name} {k.get('vgpr', -1)} {k.get('agpr', -1)} {k.get('sgpr', -1)} "
                     f"{k.get('scratch', -1)} {k.get('lds', -1)} {k.get('occupancy', -1)}")
        if k.get("scratch", 0) > 0 and "k_step" in name:
            spills.append(name)
    with open(RES, "w") as f:
        f.write("\n".join(lines) + "\n")
    if spills:
        raise RuntimeError("step kernels spill to scratch: " + ", ".join(spills))
    os.replace(tmp, LIB)
    if verbose:
        print("\n".join(lines))
    return LIB


if __name__ == "__main__":
    build(verbose=True)

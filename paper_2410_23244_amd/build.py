"""Build libbart.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "bart.hip")
LIB = os.path.join(HERE, "libbart.so")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    # packed fp32 instructions are disabled for all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


CLOCKS_LIB = os.path.join(HERE, "libbart_clocks.so")


def build(verbose: bool = False, extra: list[str] | None = None, clocks: bool = False) -> str:
    """libbart.so; with clocks=True the diagnostic variant libbart_clocks.so
    (phase clocks of the register sweep kernel, see phase_budget.py)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    out = CLOCKS_LIB if clocks else LIB
    tmp = out + ".tmp"
    cmd = [hipcc, *FLAGS, *(["-DBART_PHASE_CLOCKS"] if clocks else []), *(extra or []), SRC,
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed to build {os.path.basename(out)}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

"""Build libpulse.so (the codec) and libpulse_ceiling.so (the benchmark's
bandwidth probes, probe/ceiling.hip) in-tree with hipcc for gfx950.

    python -m paper_2602_03839_amd.build          # build (always recompiles)

Flags: -ffp-contract=off (no FMA contraction anywhere on the path) and the
packed-FP32 instruction feature switched off for device code.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libpulse.so")
CEILING_SRC = os.path.join(HERE, "probe", "ceiling.hip")
CEILING_LIB = os.path.join(HERE, "libpulse_ceiling.so")
ARCH = os.environ.get("PULSE_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-ffp-contract=off",
    "-Wall",
    "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _hipcc(out: str, srcs: list[str], verbose: bool) -> str:
    tmp = out + f".tmp{os.getpid()}"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *srcs]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with exit code {res.returncode}")
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile both libraries; returns the path of libpulse.so."""
    _hipcc(CEILING_LIB, [CEILING_SRC], verbose)
    return _hipcc(LIB, sources(), verbose)


if __name__ == "__main__":
    print(build(verbose=True))

"""Build libfathom.so for gfx950 with hipcc (in-tree, no JIT cache).

Flags: -O3; -ffp-contract=off so no multiply-add is fused unless a kernel
asks for one explicitly (the documented score order depends on it); packed
fp32 instructions disabled; correctly rounded fp32 division and sqrt (hipcc's
default, no fast-math).
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
LIB = os.path.join(OUT_DIR, "libfathom.so")
PROBE_LIB = os.path.join(OUT_DIR, "libfathom_probe.so")  # the bench's streaming-read reference
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _hipcc(out: str, srcs, verbose: bool) -> None:
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *srcs]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (res.stderr or "").splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if err.strip() and verbose:
        print(err, file=sys.stderr)
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    _hipcc(LIB, sources(), verbose)
    _hipcc(PROBE_LIB, sorted(glob.glob(os.path.join(HERE, "probe", "*.hip"))), verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

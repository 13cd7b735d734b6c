"""Build step for libuq: hipcc for gfx950, in-tree shared library.

Run as `python -m paper_2109_12497_amd.build` or through __graft_entry__.build().
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("uq_kernels.hip", "uq_randk.hip", "uq_abi.hip")]
LIB_PATH = os.path.join(HERE, "libuq.so")
# achievable-bandwidth references used by the benchmark (not part of libuq)
PROBE_SOURCES = [os.path.join(CSRC, "uq_probe.hip")]
PROBE_LIB_PATH = os.path.join(HERE, "libuq_probe.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # bit-exact binary32 arithmetic: no contraction into fused multiply-adds,
    # denormals kept
    "-ffp-contract=off",
    "-fno-gpu-flush-denormals-to-zero",
    # no packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
    "-I" + CSRC,
]


def _hipcc(sources, out, verbose):
    hipcc = os.environ.get("HIPCC", "hipcc")
    tmp = out + ".tmp"
    cmd = [hipcc, *HIPCC_FLAGS, *sources, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    log = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{' '.join(cmd)}\n{log}")
    if verbose and log.strip():
        print(log, file=sys.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Builds libuq.so (the product library) and libuq_probe.so."""
    _hipcc(PROBE_SOURCES, PROBE_LIB_PATH, verbose)
    return _hipcc(SOURCES, LIB_PATH, verbose)


if __name__ == "__main__":
    print(build(verbose=True))

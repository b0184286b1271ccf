"""Build the HIP library libmbscan.so in-tree (gfx950 only), and the issue-rate
micro-benchmark behind the instruction cost model (csrc/issue_rates.hip).

    python -m paper_2401_13660_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmbscan.so")
SOURCES = ["mbscan.hip"]
ISSUE_RATES = os.path.join(PKG, "issue_rates")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # Packed-fp32 instructions stay off: every fp32 operation is a plain VALU op.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    # A name that shadows another (a lambda local over a captured variable among
    # them) is an error: one such shadow once sent LDS writes to a private array.
    "-Werror=shadow-all",
]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed to build libmbscan.so")
    os.replace(tmp, LIB)
    build_issue_rates(verbose)
    return LIB


def build_issue_rates(verbose: bool = False) -> str:
    """The stand-alone issue-rate program (run it on the GPU: ./issue_rates)."""
    tmp = ISSUE_RATES + ".tmp"
    flags = [f for f in FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [HIPCC, *flags, os.path.join(CSRC, "issue_rates.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed to build issue_rates")
    os.replace(tmp, ISSUE_RATES)
    return ISSUE_RATES


if __name__ == "__main__":
    print(build(verbose=True))

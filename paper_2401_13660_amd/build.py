"""Build the HIP library libmbscan.so in-tree (gfx950 only), the issue-rate
micro-benchmark behind the instruction cost model (csrc/issue_rates.hip), the
LDS bank probe behind the time-split kernel's tables (csrc/lds_banks.hip), and
the exhaustive check of the bf16 pair conversion (csrc/bf16_pack_check.hip).

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
    build_lds_banks(verbose)
    build_bf16_pack_check(verbose)
    return LIB


def build_tool(name: str, verbose: bool = False) -> str:
    """A stand-alone GPU program from csrc/<name>.hip, as paper_2401_13660_amd/<name>."""
    out = os.path.join(PKG, name)
    tmp = out + ".tmp"
    flags = [f for f in FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [HIPCC, *flags, "-I", CSRC, os.path.join(CSRC, name + ".hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed to build {name}")
    os.replace(tmp, out)
    return out


def build_issue_rates(verbose: bool = False) -> str:
    """The stand-alone issue-rate program (run it on the GPU: ./issue_rates)."""
    return build_tool("issue_rates", verbose)


def build_lds_banks(verbose: bool = False) -> str:
    """The LDS bank probe behind the time-split kernel's table layout (./lds_banks)."""
    return build_tool("lds_banks", verbose)


def build_bf16_pack_check(verbose: bool = False) -> str:
    """The exhaustive check of the bf16 pair conversion (run by a GPU test)."""
    return build_tool("bf16_pack_check", verbose)

if __name__ == "__main__":
    print(build(verbose=True))

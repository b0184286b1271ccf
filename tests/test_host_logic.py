"""Host-side launch logic of the library, run on the CPU.

The forward cuts the sequence into time segments when the (batch, channel)
rows are too few to fill the chip: the count is the largest that fills the
resident waves at most twice over, for fewer than 3/8 of them per segment;
segments are at least 256 bytes and a multiple of 32.  A small host program
built from the library's own header prints its choice; the expectations come
from that rule, written out here, and from a few cases worked by hand.
"""
import math
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2401_13660_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None,
                                reason="needs hipcc")


@pytest.fixture(scope="module")
def segments_exe(tmp_path_factory):
    exe = tmp_path_factory.mktemp("host") / "segments"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-I", CSRC,
                    os.path.join(ROOT, "tests", "host", "segments_main.cpp"), "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    return str(exe)


def _rule(wb: int, L: int, resident: int):
    n = 2 * resident // wb if wb * 8 < resident * 3 else 1
    n = max(1, min(n, L // 256))
    seg = -(-L // n)
    seg = -(-seg // 32) * 32
    return -(-L // seg), seg


def _run(exe, cases):
    out = subprocess.run([exe], input="".join(f"{w} {L} {r}\n" for w, L, r in cases), check=True,
                         capture_output=True, text=True).stdout.split("\n")
    return [tuple(int(v) for v in line.split()) for line in out if line.strip()]


# (waves_base, L, resident) -> (segments, segment length), worked by hand
HAND = [
    ((576, 65536, 2048), (7, 9376)),     # 1.6B layer, batch 1: ceil(65536/7) = 9363 -> 9376
    ((1792, 8192, 2048), (1, 8192)),     # 972M layer: enough rows
    ((1024, 8192, 2048), (1, 8192)),     # 353M layer: at the threshold's far side
    ((448, 8192, 2048), (9, 928)),       # 972M shape at batch 1: 4096 // 448 = 9; ceil(8192/9) = 911 -> 928
    ((8, 4096, 2048), (16, 256)),        # few rows: capped at 256-byte segments
    ((1, 4112, 2048), (15, 288)),        # ceil(4112/16) = 257 -> 288 bytes, so 15 segments
    ((1, 640, 2048), (2, 320)),
    ((767, 8192, 2048), (5, 1664)),      # just below 3/8 of the resident waves
    ((768, 8192, 2048), (1, 8192)),      # at 3/8: no segments
    ((576, 65536, 512), (1, 65536)),     # a device with 64 CUs: 576 waves fill it
    ((1, 16, 2048), (1, 32)),            # one segment, its length rounded up to 32 (the launcher
                                         # does not cut sequences below 512 bytes at all)
]


def test_segment_counts_worked_by_hand(segments_exe):
    got = _run(segments_exe, [c for c, _ in HAND])
    assert got == [e for _, e in HAND]


def test_segment_counts_follow_the_rule(segments_exe):
    cases = [(wb, L, r) for r in (512, 2048, 4096) for wb in (1, 3, 8, 100, 255, 256, 448, 576, 700, 1000, 1535,
                                                               1536, 5000)
             for L in (16, 256, 512, 528, 1008, 4096, 8192, 65536)]
    got = _run(segments_exe, cases)
    for (wb, L, r), g in zip(cases, got):
        assert g == _rule(wb, L, r), (wb, L, r, g)
        n, seg = g
        assert seg % 32 == 0 or n == 1
        assert (n - 1) * seg < L <= n * seg
        assert n == 1 or seg >= 256

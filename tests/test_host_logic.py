"""Host-side launch logic of the library, run on the CPU.

The forward cuts the sequence into time segments when the (batch, channel)
rows are too few to fill the chip: the count is the largest that fills the
resident waves at most twice over, for fewer than 3/8 of them per segment;
segments are at least 256 bytes and a multiple of 32.  The segment pre-pass
cuts each segment into 2 pieces (then segments are a multiple of 64) where
that shortens its busiest SIMD's work: ceil(2 w / simds) / 2 below
ceil(w / simds) for its w one-piece waves.  A small host program
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


def _rule(wb: int, L: int, resident: int, simds: int):
    n = 2 * resident // wb if wb * 8 < resident * 3 else 1
    n = max(1, min(n, L // 256))
    m = 1
    if n > 1:
        w = wb * (n - 1)
        if -(-2 * w // simds) < 2 * -(-w // simds):
            m = 2
    seg = -(-L // n)
    seg = -(-seg // (32 * m)) * (32 * m)
    return -(-L // seg), seg, m


def _run(exe, cases):
    out = subprocess.run([exe], input="".join(f"{w} {L} {r} {s}\n" for w, L, r, s in cases), check=True,
                         capture_output=True, text=True).stdout.split("\n")
    return [tuple(int(v) for v in line.split()) for line in out if line.strip()]


# (waves_base, L, resident, simds) -> (segments, segment length, pre-pass pieces), worked by hand
HAND = [
    ((576, 65536, 2048, 1024), (7, 9408, 2)),   # 1.6B layer, batch 1: 3456 pre-pass waves are 3.375
                                                # per SIMD (4 on some), 6912 are 6.75 (7): 7/2 < 4, so
                                                # 2 pieces; ceil(65536/7) = 9363 -> 9408 (64 | 9408)
    ((1792, 8192, 2048, 1024), (1, 8192, 1)),   # 972M layer: enough rows
    ((1024, 8192, 2048, 1024), (1, 8192, 1)),   # 353M layer: at the threshold's far side
    ((448, 8192, 2048, 1024), (9, 960, 2)),     # 972M shape at batch 1: 4096 // 448 = 9; 3584 waves:
                                                # ceil(7)/2 < ceil(3.5); ceil(8192/9) = 911 -> 960
    ((8, 4096, 2048, 1024), (16, 256, 2)),      # few rows: capped at 256-byte segments, 120 waves
    ((1, 4112, 2048, 1024), (13, 320, 2)),      # ceil(4112/16) = 257 -> 320 bytes, so 13 segments
    ((1, 640, 2048, 1024), (2, 320, 2)),
    ((767, 8192, 2048, 1024), (5, 1664, 1)),    # just below 3/8 of the resident waves; 3068 waves:
                                                # ceil(5.99) = 6 = 2 ceil(2.996), so one piece
    ((768, 8192, 2048, 1024), (1, 8192, 1)),    # at 3/8: no segments
    ((750, 1296, 2048, 1024), (5, 288, 1)),     # 4096 // 750 = 5 = 1296 // 256; 3000 waves: ceil(5.86)
                                                # = 6 = 2 ceil(2.93), one piece; ceil(1296/5) = 260 -> 288
    ((576, 65536, 512, 256), (1, 65536, 1)),    # a device with 64 CUs: 576 waves fill it
    ((1, 16, 2048, 1024), (1, 32, 1)),          # one segment, its length rounded up to 32 (the launcher
                                                # does not cut sequences below 512 bytes at all)
]


def test_segment_counts_worked_by_hand(segments_exe):
    got = _run(segments_exe, [c for c, _ in HAND])
    assert got == [e for _, e in HAND]


def test_segment_counts_follow_the_rule(segments_exe):
    cases = [(wb, L, r, r // 2) for r in (512, 2048, 4096)
             for wb in (1, 3, 8, 100, 255, 256, 448, 576, 700, 1000, 1535, 1536, 5000)
             for L in (16, 256, 512, 528, 1008, 4096, 8192, 65536)]
    got = _run(segments_exe, cases)
    for (wb, L, r, s), g in zip(cases, got):
        assert g == _rule(wb, L, r, s), (wb, L, r, s, g)
        n, seg, m = g
        assert seg % (32 * m) == 0 or n == 1
        assert (n - 1) * seg < L <= n * seg
        assert n == 1 or seg >= 256
        assert m in (1, 2) and (n > 1 or m == 1)

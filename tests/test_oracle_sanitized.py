"""The oracle's C code built with AddressSanitizer and UndefinedBehaviorSanitizer
(host code only, gcc), running every pin in a child process that preloads the
sanitizer runtime: an out-of-bounds index, a use of freed memory, a signed
overflow or a misaligned access in the oracle ends that process with a report.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

_CHILD = r"""
import sys
sys.path[:0] = [{root!r}, {here!r}]
import oracle
import oracle_pins as P
orc = oracle.Oracle({lib!r})
for pin in P.ALL_PINS:
    pin(orc)
    print("ok", pin.__name__, flush=True)
print("ALL-PINS-DONE", flush=True)
"""


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_pins_clean_under_asan_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    import oracle
    lib = str(tmp_path / "liboracle_san.so")
    oracle.build(out=lib, extra_flags=["-O1", "-g", "-fno-omit-frame-pointer",
                                       "-fsanitize=address,undefined", "-fno-sanitize-recover=all"])
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan
    # Python's own allocations are not the subject here (and look like leaks at exit).
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "2"
    code = _CHILD.format(root=ROOT, here=HERE, lib=lib)
    res = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout + res.stderr
    assert "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert "runtime error:" not in out, out[-4000:]
    assert res.returncode == 0 and "ALL-PINS-DONE" in res.stdout, out[-4000:]

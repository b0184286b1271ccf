"""A plain C program calls the library through include/mbscan.h alone (device
memory from the HIP runtime's C API, no Python or torch in the path) and checks
mb_scan_fwd against the fp64 oracle; __graft_entry__.build() compiles it."""
import os
import subprocess

import pytest

from gpu_util import announce, has_gpu

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "host", "c_caller")


def test_c_caller_matches_oracle():
    assert os.path.exists(EXE), f"{EXE} is not built; run __graft_entry__.build()"
    announce("plain C caller: mb_scan_fwd (2, 40, 528) fp32 against the oracle")
    res = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(res.stdout, res.stderr, flush=True)
    assert res.returncode == 0, f"c_caller exited with {res.returncode}: {res.stdout} {res.stderr}"

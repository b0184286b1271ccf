"""The bf16 outputs are rounded by the hardware pair conversion (v_cvt_pk_bf16_f32);
the stand-alone check compares it with the bit-level round-to-nearest-even over
every fp32 pattern, in both halves of the pair, on the GPU."""
import os
import subprocess

import pytest

from gpu_util import announce, has_gpu

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]

PROG = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2401_13660_amd", "bf16_pack_check")


def test_pair_conversion_matches_bit_rounding_on_every_pattern():
    if not os.path.exists(PROG):
        pytest.fail(f"{PROG} is not built (python -m paper_2401_13660_amd.build)")
    announce("bf16 pair conversion, all 2^32 patterns")
    res = subprocess.run([PROG], capture_output=True, text=True, timeout=100)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "0 of 8589934592 results differ" in res.stdout, res.stdout

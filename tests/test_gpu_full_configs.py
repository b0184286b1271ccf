"""The three layer-shaped workloads at full size, in the configuration the
benchmark times, checked on sampled (batch, channel) rows over their whole
length (the oracle computes each row independently)."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, gpu_fwd, has_gpu
from paper_2401_13660_amd.inputs import workload

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]


def sample_rows(nb, dim, k=48, seed=0):
    rng = np.random.default_rng(seed)
    rows = {0, dim - 1, nb * dim - 1, (nb - 1) * dim, dim // 2}
    rows |= set(rng.integers(0, nb * dim, k).tolist())
    return np.array(sorted(rows), dtype=np.int64)


@pytest.mark.parametrize("name", ["mambabyte353m_L8192", "mambabyte972m_L8192", "mambabyte1p6b_L65536"])
def test_full_size_sampled_rows(name):
    inp = workload(name)
    announce(f"{name} full size {inp.u.shape}, sampled rows")
    y, h = gpu_fwd(inp)
    rows = sample_rows(inp.batch, inp.dim)
    check_against_oracle(inp, y, h, rows=rows)
    assert np.isfinite(y[0].float().cpu().numpy()).all()

"""The differentiable scan (``selective_scan``): torch autograd through the
forward with checkpoints and the backward from them gives the oracle's
gradients of the same loss."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, has_gpu, to_device
from parity import rel_err
from paper_2401_13660_amd.inputs import make_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_autograd_matches_oracle(dtype):
    import paper_2401_13660_amd as mb
    inp = make_inputs(2, 72, 256, 16, dtype=dtype, seed=101, with_h0=True)
    announce(f"autograd selective_scan (2, 72, 256) {dtype}")
    t = {k: (v.clone().requires_grad_() if v.is_floating_point() else v) for k, v in to_device(inp).items()}
    y, h_last = mb.selective_scan(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t["Dskip"], dt_bias=t["dt_bias"],
                                  z=t["z"], h0=t["h0"])
    assert y.dtype == t["u"].dtype
    rng = np.random.default_rng(102)
    wy = torch.from_numpy(rng.standard_normal(inp.u.shape).astype(np.float32)).to("cuda:0")
    wh = torch.from_numpy(rng.standard_normal(inp.h0.shape).astype(np.float32)).to("cuda:0")
    loss = (y.float() * wy).sum() + (h_last * wh).sum()
    loss.backward()
    torch.cuda.synchronize()
    dy = wy.to(y.dtype).float().cpu().numpy()            # the incoming gradient as autograd hands it over
    ref = oracle.default().scan_bwd(inp.u, inp.delta, inp.A, inp.B, inp.C, dy, z=inp.z, Dskip=inp.Dskip,
                                    dt_bias=inp.dt_bias, h0=inp.h0, dh_last=wh.cpu().numpy(), dtype=inp.dtype)
    bf = dtype == "bf16"
    for name, rname, tol in (("u", "du", 1e-4), ("delta", "ddelta", 1e-4), ("z", "dz", 1e-4), ("A", "dA", 2e-4),
                             ("B", "dB", 1e-4), ("C", "dC", 1e-4), ("Dskip", "dD", 2e-4),
                             ("dt_bias", "dbias", 2e-4), ("h0", "dh0", 1e-4)):
        g = t[name].grad
        assert g is not None and g.dtype == t[name].dtype, name
        # gradients of bf16 tensors are bf16: one more rounding
        bar = tol + (2.0 ** -8 if g.dtype == torch.bfloat16 else 0.0)
        e = rel_err(g.float().cpu().numpy().astype(np.float64), ref[rname])
        assert e <= bar, f"grad {name}: {e:.3e} > {bar:.1e}"

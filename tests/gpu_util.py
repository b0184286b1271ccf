"""Helpers for the GPU tests: move seeded inputs to the device, run both sides."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from parity import rel_err


def has_gpu() -> bool:
    return torch.cuda.is_available()


def dev_tensor(a, device="cuda:0"):
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:                    # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


def to_device(inp, device="cuda:0"):
    return {k: dev_tensor(v, device) for k, v in inp.arrays().items()}


def announce(msg: str):
    print(f"\n[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def gpu_fwd(inp, *, out_dtype=torch.float32, return_last_state=True, delta_softplus=True, **over):
    import paper_2401_13660_amd as mb
    t = to_device(inp)
    t.update(over)
    res = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t.get("Dskip"),
                      dt_bias=t.get("dt_bias"), z=t.get("z"), h0=t.get("h0"),
                      delta_softplus=delta_softplus, out_dtype=out_dtype,
                      return_last_state=return_last_state)
    torch.cuda.synchronize()
    return res


def check_against_oracle(inp, y_gpu, h_gpu, rows=None, tol_y=2e-3, tol_h=1e-4, delta_softplus=True):
    """Compare (sampled rows of) the GPU result with the fp64 oracle; returns the errors."""
    y_ref, h_ref = oracle.scan_inputs(inp, rows=rows, delta_softplus=delta_softplus)
    yg = y_gpu.float().cpu().numpy().astype(np.float64)
    hg = None if h_gpu is None else h_gpu.cpu().numpy().astype(np.float64)
    nb, dim, L = inp.u.shape
    if rows is not None:
        yg = yg.reshape(nb * dim, L)[rows]
        hg = None if hg is None else hg.reshape(nb * dim, -1)[rows]
    ey = rel_err(yg, y_ref)
    eh = rel_err(hg, h_ref) if hg is not None else 0.0
    assert ey <= tol_y, f"y relative error {ey:.3e} > {tol_y:.1e}"
    assert eh <= tol_h, f"h_last relative error {eh:.3e} > {tol_h:.1e}"
    return ey, eh

"""The selective scan as a differentiable torch operation, for training.

The forward runs ``mb_scan_fwd_ckpt`` (y in u's dtype, h_last, and the state
every 16 bytes); the backward runs ``mb_scan_bwd`` from those checkpoints.  All
arithmetic happens in the HIP library: this module only holds tensors between
the two calls.  dB and dC come back in fp32 and are handed to autograd in B's
and C's dtype.  Supported as the library's backward is: dstate 16 and L a
multiple of 16 (the library raises otherwise).
"""
from __future__ import annotations

import torch

from . import _binding as _b


class _SelectiveScan(torch.autograd.Function):
    @staticmethod
    def forward(ctx, u, delta, A, B, C, D, dt_bias, z, h0, delta_softplus):
        y, h_last, ck = _b.scan_fwd(u, delta, A, B, C, D=D, dt_bias=dt_bias, z=z, h0=h0,
                                    delta_softplus=delta_softplus, out_dtype=u.dtype, return_last_state=True,
                                    return_ckpt=True)
        ctx.delta_softplus = delta_softplus
        ctx.save_for_backward(u, delta, A, B, C, D, dt_bias, z, h0, ck)
        return y, h_last

    @staticmethod
    def backward(ctx, dy, dh_last):
        u, delta, A, B, C, D, dt_bias, z, h0, ck = ctx.saved_tensors
        g = _b.scan_bwd(u, delta, A, B, C, dy.contiguous(), D=D, dt_bias=dt_bias, z=z, h0=h0,
                        dh_last=None if dh_last is None else dh_last.contiguous(),
                        delta_softplus=ctx.delta_softplus, ck=ck)
        dB = g["dB"] if B.dtype == torch.float32 else g["dB"].to(B.dtype)
        dC = g["dC"] if C.dtype == torch.float32 else g["dC"].to(C.dtype)
        return (g["du"], g["ddelta"], g["dA"], dB, dC, g["dD"], g["ddt_bias"], g["dz"],
                g["dh0"] if h0 is not None else None, None)


def selective_scan(u, delta, A, B, C, D=None, dt_bias=None, z=None, h0=None, *, delta_softplus=True):
    """Differentiable scan: returns (y, h_last), y in u's dtype.  Shapes and dtypes
    as for ``scan_fwd``; gradients flow to every tensor argument."""
    return _SelectiveScan.apply(u, delta, A, B, C, D, dt_bias, z, h0, delta_softplus)

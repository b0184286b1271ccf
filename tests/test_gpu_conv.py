"""GPU parity of mb_conv1d_fwd / mb_conv1d_step against the fp64 oracle.

The convolution is 4 fp32 FMAs and a Swish per output, so an fp32 output is
held to 1e-5 under the metric of tests/parity.py, and a bf16 output to
1e-5 + 2^-8 (one bf16 rounding).  The carried state holds raw inputs, so it
must match exactly.  Splitting a sequence and chaining the state, or running
byte by byte, must reproduce one call bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, dev_tensor, has_gpu
from parity import rel_err
from paper_2401_13660_amd.inputs import conv_workload, make_conv_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]

TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-5 + 2.0 ** -8}


def run_conv(c, out_dtype=None, apply_silu=True, rows=None, **kw):
    import paper_2401_13660_amd as mb
    x = dev_tensor(c.x)
    out_dtype = out_dtype or x.dtype
    y, st = mb.conv1d(x, dev_tensor(c.w), bias=dev_tensor(c.bias), state=dev_tensor(c.state),
                      apply_silu=apply_silu, out_dtype=out_dtype, return_state=True, **kw)
    torch.cuda.synchronize()
    y_ref, st_ref = oracle.default().conv1d(c.x, c.w, bias=c.bias, state=c.state, apply_silu=apply_silu,
                                            dtype=c.dtype)
    yg = y.float().cpu().numpy().astype(np.float64)
    if rows is not None:
        nb, dim, L = c.x.shape
        yg, y_ref = yg.reshape(nb * dim, L)[rows], y_ref.reshape(nb * dim, L)[rows]
    e = rel_err(yg, y_ref)
    assert e <= TOL[out_dtype], f"conv y relative error {e:.3e}"
    if c.w.shape[1] > 1:
        assert np.array_equal(st.cpu().numpy().astype(np.float64), st_ref), "conv state differs"
    return y, st


# (batch, dim, L): vector path (L % 8 == 0) with a ragged channel count; element
# path (L % 8 != 0); lengths shorter than the kernel, one span, a span and a bit.
@pytest.mark.parametrize("shape", [(2, 200, 1008), (2, 130, 1000), (3, 17, 1), (3, 17, 2), (3, 17, 3),
                                   (3, 17, 8), (3, 17, 9), (1, 64, 4096), (1, 64, 4095)])
@pytest.mark.parametrize("with_state", [True, False])
def test_conv_shapes(shape, with_state):
    c = make_conv_inputs(*shape, dtype="bf16", seed=31, with_state=with_state)
    announce(f"conv {shape} bf16 state={with_state}")
    run_conv(c)


@pytest.mark.parametrize("width", [1, 2, 3, 4])
@pytest.mark.parametrize("dtype,out", [("bf16", torch.float32), ("f32", torch.float32),
                                       ("f32", torch.bfloat16), ("bf16", torch.bfloat16)])
def test_conv_widths_and_dtypes(width, dtype, out):
    c = make_conv_inputs(2, 96, 520, width, dtype=dtype, seed=32, with_state=True)
    announce(f"conv width {width} {dtype} -> {out}")
    run_conv(c, out_dtype=out)


@pytest.mark.parametrize("apply_silu", [True, False])
def test_conv_no_bias_and_activation_switch(apply_silu):
    c = make_conv_inputs(2, 72, 264, dtype="bf16", seed=33, with_bias=False, with_state=True)
    announce(f"conv no bias, silu={apply_silu}")
    run_conv(c, apply_silu=apply_silu)


def test_conv_misaligned_rows_take_the_element_path():
    """A view starting one element into the buffer: rows no longer 16-byte aligned."""
    import paper_2401_13660_amd as mb
    c = make_conv_inputs(2, 40, 257, dtype="bf16", seed=34, with_state=True)
    announce("conv misaligned view")
    x_full = dev_tensor(c.x)
    buf = torch.empty(x_full.numel() + 8, dtype=x_full.dtype, device=x_full.device)
    xv = buf[1:1 + x_full.numel()].view(c.x.shape)        # one element past an aligned start
    xv.copy_(x_full)
    assert xv.data_ptr() % 16 != 0
    y, st = mb.conv1d(xv, dev_tensor(c.w), bias=dev_tensor(c.bias), state=dev_tensor(c.state),
                      return_state=True)
    torch.cuda.synchronize()
    y_ref, st_ref = oracle.default().conv1d(c.x, c.w, bias=c.bias, state=c.state, dtype=c.dtype)
    assert rel_err(y.float().cpu().numpy(), y_ref) <= TOL[torch.bfloat16]
    assert np.array_equal(st.cpu().numpy().astype(np.float64), st_ref)


def test_conv_seqlen_zero_passes_the_state_on():
    import paper_2401_13660_amd as mb
    c = make_conv_inputs(2, 24, 0, dtype="bf16", seed=35, with_state=True)
    announce("conv L = 0")
    x = torch.empty((2, 24, 0), dtype=torch.bfloat16, device="cuda:0")
    y, st = mb.conv1d(x, dev_tensor(c.w), bias=dev_tensor(c.bias), state=dev_tensor(c.state),
                      return_state=True)
    torch.cuda.synchronize()
    assert y.numel() == 0
    assert torch.equal(st.cpu(), torch.from_numpy(c.state))


def test_conv_split_and_steps_match_one_call():
    """Resume: [0, k) then [k, L) with the carried state, and L single-byte steps, give
    exactly the bits of one call."""
    import paper_2401_13660_amd as mb
    c = make_conv_inputs(3, 130, 200, dtype="bf16", seed=36, with_state=True)
    announce("conv split / steps")
    x, w, b, s0 = dev_tensor(c.x), dev_tensor(c.w), dev_tensor(c.bias), dev_tensor(c.state)
    y, st = mb.conv1d(x, w, bias=b, state=s0, return_state=True)
    for k in (1, 3, 8, 101, 199):
        y1, s1 = mb.conv1d(x[..., :k].contiguous(), w, bias=b, state=s0, return_state=True)
        y2, s2 = mb.conv1d(x[..., k:].contiguous(), w, bias=b, state=s1, return_state=True)
        assert torch.equal(torch.cat([y1, y2], dim=2), y), f"split at {k}"
        assert torch.equal(s2, st), f"state after split at {k}"
    state = s0.clone()
    for t in range(c.x.shape[2]):
        yt = mb.conv1d_step(state, x[..., t].contiguous(), w, bias=b)
        assert torch.equal(yt, y[..., t]), f"step {t}"
    assert torch.equal(state, st)


def test_conv_step_against_oracle():
    import paper_2401_13660_amd as mb
    c = make_conv_inputs(4, 300, 5, dtype="bf16", seed=37, with_state=True)
    announce("conv step vs oracle")
    state = dev_tensor(c.state).clone()
    ref_state = c.state.astype(np.float64)
    for t in range(c.x.shape[2]):
        yt = mb.conv1d_step(state, dev_tensor(np.ascontiguousarray(c.x[..., t])), dev_tensor(c.w),
                            bias=dev_tensor(c.bias), out_dtype=torch.float32)
        ry, ref_state = oracle.default().conv1d_step(np.ascontiguousarray(c.x[..., t]), c.w, ref_state,
                                                     bias=c.bias, dtype=c.dtype)
        torch.cuda.synchronize()
        assert rel_err(yt.cpu().numpy(), ry) <= TOL[torch.float32]
        assert np.array_equal(state.cpu().numpy().astype(np.float64), ref_state)


@pytest.mark.parametrize("name", ["mambabyte972m_L8192", "verify_b32_L16"])
def test_conv_full_size_sampled_rows(name):
    """The convolution in front of the 972M layer at full size (bf16 out, as it feeds
    x_proj and the scan) and of the verify chunk (with a carried state)."""
    c = conv_workload(name, seed=0)
    nb, dim, L = c.x.shape
    rows = np.sort(np.random.default_rng(38).choice(nb * dim, 64, replace=False))
    announce(f"conv full size {name} {(nb, dim, L)}")
    run_conv(c, out_dtype=torch.bfloat16, rows=rows)

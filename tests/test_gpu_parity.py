"""GPU parity of mb_scan_fwd / mb_scan_step against the fp64 oracle.

Tolerance (fp32 arithmetic, fp32 output): max relative error 2e-3 on y and
1e-4 on h_last under the metric of tests/parity.py.  A bf16 output adds one
bf16 rounding (2^-9 relative), so bf16-output cases allow 2e-3 + 2^-8.
"""
import numpy as np
import pytest
import torch

from gpu_util import announce, check_against_oracle, gpu_fwd, has_gpu, to_device
from parity import TOL_Y_BF16_OUT
from paper_2401_13660_amd.inputs import make_inputs, workload

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]



def run_case(inp, **kw):
    y, h = gpu_fwd(inp, **kw)
    return check_against_oracle(inp, y, h)


def test_tiny_config_full():
    inp = workload("tiny_f32")
    announce("tiny_f32 (1, 64, 256) fp32, full tensors")
    run_case(inp)


# Lengths that are multiples of 16 take the tiled kernel (1008 ends in a half
# chunk); other lengths take the row-per-thread kernel.  dim 200 leaves dead
# lanes in the last 8-channel group.
@pytest.mark.parametrize("L", [1008, 1000])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("gated,with_h0", [(True, True), (False, False), (True, False)])
def test_ragged_multi_tile(dtype, gated, with_h0, L):
    inp = make_inputs(2, 200, L, 16, dtype=dtype, seed=1, gated=gated, with_h0=with_h0)
    announce(f"ragged (2, 200, {L}) {dtype} gated={gated} h0={with_h0}")
    run_case(inp)


@pytest.mark.parametrize("L", [1, 2, 3, 16, 32, 48, 63, 64, 65, 80, 127, 511, 513, 4096, 4097, 4112])
def test_edge_lengths(L):
    inp = make_inputs(3, 130, L, 16, dtype="bf16", seed=2, with_h0=True)
    announce(f"edge length L={L} (3, 130) bf16")
    run_case(inp)


# L = 16: one half chunk per wave, the half-size-table instantiation (the
# verify shape), across input and output types, with and without the gate and
# softplus, and with dead lanes (dim 100).
@pytest.mark.parametrize("dtype,gated,softplus,out", [("f32", True, True, torch.float32),
                                                      ("bf16", False, True, torch.float32),
                                                      ("bf16", True, True, torch.bfloat16),
                                                      ("f32", False, False, torch.float32)])
def test_one_half_chunk(dtype, gated, softplus, out):
    inp = make_inputs(5, 100, 16, 16, dtype=dtype, seed=21, with_h0=True, gated=gated, with_bias=softplus)
    if not softplus:                                  # dlt = delta as given: keep it small and positive
        inp.delta = (np.abs(inp.delta) * np.float32(0.05)).astype(np.float32)
    announce(f"L=16 (5, 100) {dtype} gated={gated} softplus={softplus} out={out}")
    y, h = gpu_fwd(inp, out_dtype=out, delta_softplus=softplus)
    check_against_oracle(inp, y, h, tol_y=TOL_Y_BF16_OUT if out == torch.bfloat16 else 2e-3,
                         delta_softplus=softplus)


# The 16-byte kernel runs on a two-dimensional grid (channel groups x batch), whose
# second dimension holds at most 65535 batch elements; a larger batch takes the
# full-table kernel.  Both sides of that limit, on sampled rows.
@pytest.mark.parametrize("batch", [65535, 65536])
def test_one_half_chunk_at_the_grid_limit(batch):
    inp = make_inputs(batch, 8, 16, 16, dtype="bf16", seed=22, with_h0=True)
    announce(f"L=16 ({batch}, 8) bf16")
    y, h = gpu_fwd(inp)
    rows = np.unique(np.concatenate([np.arange(0, 64), np.arange(batch * 8 - 64, batch * 8),
                                     np.random.default_rng(5).integers(0, batch * 8, 128)]))
    check_against_oracle(inp, y, h, rows=rows)


def test_dskip_zero_isolates_ssm_term():
    inp = make_inputs(2, 192, 2048, 16, dtype="bf16", seed=3, with_D=False)
    announce("Dskip = 0 (2, 192, 2048)")
    run_case(inp)


def test_random_A():
    inp = make_inputs(2, 160, 1504, 16, dtype="bf16", seed=4, with_h0=True, A_kind="random")
    announce("random A (2, 160, 1504)")
    run_case(inp)


def test_extreme_delta():
    inp = make_inputs(1, 128, 704, 16, dtype="f32", seed=5, with_h0=True)
    rng = np.random.default_rng(55)
    inp.delta = (8.0 * rng.standard_normal(inp.delta.shape)).astype(np.float32)   # +-8 sigma
    announce("extreme delta_raw (1, 128, 704)")
    run_case(inp)


def test_large_h0():
    inp = make_inputs(2, 64, 304, 16, dtype="bf16", seed=6, with_h0=True)
    inp.h0 = (inp.h0 * 100.0).astype(np.float32)
    announce("h0 x 100 (2, 64, 304)")
    run_case(inp)


def test_no_softplus_no_bias():
    inp = make_inputs(1, 96, 400, 16, dtype="f32", seed=7, with_bias=False)
    inp.delta = np.abs(inp.delta).astype(np.float32) * np.float32(0.05)
    announce("delta_softplus=0 (1, 96, 400)")
    y, h = gpu_fwd(inp, delta_softplus=False)
    check_against_oracle(inp, y, h, delta_softplus=False)


@pytest.mark.parametrize("N", [1, 2, 4, 8])
def test_small_dstate(N):
    inp = make_inputs(2, 70, 333, N, dtype="bf16", seed=8, with_h0=True)
    announce(f"dstate={N} (2, 70, 333)")
    run_case(inp)


def test_bf16_output():
    inp = make_inputs(2, 128, 912, 16, dtype="bf16", seed=9)
    announce("bf16 output (2, 128, 912)")
    y, h = gpu_fwd(inp, out_dtype=torch.bfloat16)
    assert y.dtype == torch.bfloat16
    check_against_oracle(inp, y, h, tol_y=TOL_Y_BF16_OUT)


def test_seqlen_zero_returns_h0():
    inp = make_inputs(2, 32, 0, 16, dtype="bf16", seed=10, with_h0=True)
    announce("L=0")
    y, h = gpu_fwd(inp)
    assert y.numel() == 0
    assert np.array_equal(h.cpu().numpy(), inp.h0)
    y, h = gpu_fwd(inp, h0=None)
    assert np.all(h.cpu().numpy() == 0)


@pytest.mark.parametrize("L", [256, 257])
def test_h_last_may_alias_h0(L):
    import paper_2401_13660_amd as mb
    inp = make_inputs(2, 100, L, 16, dtype="bf16", seed=11, with_h0=True)
    announce(f"h_last is h0 (2, 100, {L})")
    t = to_device(inp)
    state = t["h0"].clone()
    y, h = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t["Dskip"], dt_bias=t["dt_bias"],
                       z=t["z"], h0=state, h_last=state)
    torch.cuda.synchronize()
    assert h.data_ptr() == state.data_ptr()
    check_against_oracle(inp, y, h)


# Shapes with few rows cut the sequence into time segments (a pre-pass of segment
# aggregates, then one wave per segment): (1, 64, 4096) takes 16 segments,
# (1, 61, 4112) 13 with dead lanes.  The waves of the last segment write h_last
# while waves of earlier segments of the same rows may not have started, so the
# scan must not read h0 itself there.  Each entry point that writes h_last is run
# with h_last on top of h0.
@pytest.mark.parametrize("shape", [(1, 64, 4096), (1, 61, 4112)])
@pytest.mark.parametrize("entry", ["fwd", "states", "ckpt"])
def test_h_last_may_alias_h0_segmented(shape, entry):
    import paper_2401_13660_amd as mb
    import oracle
    nb, dim, L = shape
    inp = make_inputs(nb, dim, L, 16, dtype="bf16", seed=21, with_h0=True)
    announce(f"h_last is h0, segmented {shape} via {entry}")
    t = to_device(inp)
    state = t["h0"].clone()
    kw = dict(D=t["Dskip"], dt_bias=t["dt_bias"], z=t["z"], h0=state, h_last=state)
    pos = np.array([[-1], [L // 3], [L - 1]], dtype=np.int32)
    if entry == "states":
        kw["positions"] = torch.from_numpy(pos).cuda()
    if entry == "ckpt":
        kw["return_ckpt"] = True
    res = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], **kw)
    torch.cuda.synchronize()
    y, h = res[0], res[1]
    assert h.data_ptr() == state.data_ptr()
    check_against_oracle(inp, y, h)
    if entry == "states":
        _, _, hp_ref = oracle.scan_inputs(inp, positions=pos)
        hp = res[2].cpu().numpy().astype(np.float64)
        from parity import rel_err
        assert rel_err(hp, hp_ref) <= 1e-4


# Shapes with at most one plain-kernel wave per SIMD and one time segment take the
# kernel that cuts every chunk into two time slices inside the wave; the
# checkpointing entry point always takes the plain kernel.  Both compute each
# state by the same operations in the same order, so y and h_last must be equal
# bit for bit (and both meet the oracle).
@pytest.mark.parametrize("shape,dtype,out_dtype,gated,with_h0,softplus", [
    ((4, 2048, 512), "bf16", torch.float32, True, False, True),       # 1024 plain waves
    ((3, 100, 320), "f32", torch.bfloat16, False, True, False),       # dead lanes, half chunk
    ((1, 8, 48), "bf16", torch.float32, True, True, True),            # one full and one half chunk
    ((2, 36, 32), "f32", torch.float32, True, True, True),            # a single full chunk
])
def test_time_split_kernel_equals_plain(shape, dtype, out_dtype, gated, with_h0, softplus):
    import paper_2401_13660_amd as mb
    nb, dim, L = shape
    inp = make_inputs(nb, dim, L, 16, dtype=dtype, seed=31, gated=gated, with_h0=with_h0,
                      with_bias=softplus)
    if not softplus:
        # used as given, Delta must stay positive (else abar > 1 and the state grows without bound)
        assert dtype == "f32"
        inp.delta = np.abs(inp.delta).astype(np.float32) * np.float32(0.05)
    announce(f"time-split vs plain kernel {shape} {dtype} out={out_dtype} gated={gated} h0={with_h0} "
             f"softplus={softplus}")
    t = to_device(inp)
    kw = dict(D=t["Dskip"], dt_bias=t.get("dt_bias"), z=t.get("z"), h0=t.get("h0"), delta_softplus=softplus,
              out_dtype=out_dtype)
    y1, h1 = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], return_last_state=True, **kw)
    y2, h2, _ = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], return_last_state=True,
                            return_ckpt=True, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2), "y differs between the time-split and the plain kernel"
    assert torch.equal(h1, h2), "h_last differs between the time-split and the plain kernel"
    tol = TOL_Y_BF16_OUT if out_dtype == torch.bfloat16 else 2e-3
    check_against_oracle(inp, y1, h1, tol_y=tol, delta_softplus=softplus)


def test_resume_split_on_gpu():
    """Scanning two halves with the carried state equals scanning the whole (Alg. 1 resume)."""
    import paper_2401_13660_amd as mb
    inp = make_inputs(2, 96, 1200, 16, dtype="bf16", seed=12, with_h0=True)
    announce("split resume (2, 96, 1200) at k=512")
    t = to_device(inp)
    k = 512
    common = dict(D=t["Dskip"], dt_bias=t["dt_bias"])
    sl = lambda x, a, b: x[..., a:b].contiguous()
    y1, h1 = mb.scan_fwd(sl(t["u"], 0, k), sl(t["delta"], 0, k), t["A"], sl(t["B"], 0, k), sl(t["C"], 0, k),
                         z=sl(t["z"], 0, k), h0=t["h0"], return_last_state=True, **common)
    y2, h2 = mb.scan_fwd(sl(t["u"], k, None), sl(t["delta"], k, None), t["A"], sl(t["B"], k, None),
                         sl(t["C"], k, None), z=sl(t["z"], k, None), h0=h1, return_last_state=True, **common)
    torch.cuda.synchronize()
    check_against_oracle(inp, torch.cat([y1, y2], dim=2), h2)


def test_deterministic():
    inp = make_inputs(2, 256, 3008, 16, dtype="bf16", seed=13, with_h0=True)
    announce("determinism (2, 256, 3008)")
    y1, h1 = gpu_fwd(inp)
    y2, h2 = gpu_fwd(inp)
    assert torch.equal(y1, y2) and torch.equal(h1, h2)


# (1, 5996, 1296): 750 eight-channel waves (4 dead lanes), 5 segments of 288 bytes
# (the last 144), and the pre-pass in one piece per segment (3,000 waves: 6 per
# SIMD either way); the other shapes take two pieces per segment.
@pytest.mark.parametrize("shape", [(1, 64, 4096), (1, 61, 4112), (2, 24, 8192), (1, 8, 640), (1, 5996, 1296)])
@pytest.mark.parametrize("gated", [True, False])
def test_time_segments(shape, gated):
    """Few (batch, channel) rows and a long sequence: the tiled path cuts time into
    segments, a pre-pass computes each segment's aggregate (in one or two pieces per
    segment) and the scan folds them."""
    nb, dim, L = shape
    inp = make_inputs(nb, dim, L, 16, dtype="bf16", seed=15, with_h0=True, gated=gated, A_kind="random")
    announce(f"time segments {shape} gated={gated}")
    run_case(inp)


def test_time_segments_f32_two_rounds():
    """fp32 inputs at the 1.6B layer's width, (1, 4608, 2048): 7 segments of 320 bytes
    (the last 128), the pre-pass in 2 pieces of 160 per segment.  Its 6,912 waves are
    more than the 5 per SIMD that fit with fp32 inputs (83 VGPRs), so it runs in two
    rounds."""
    inp = make_inputs(1, 4608, 2048, 16, dtype="f32", seed=17, with_h0=True, A_kind="random")
    announce("time segments fp32 (1, 4608, 2048), pre-pass in two rounds")
    run_case(inp)


def test_time_segments_deterministic():
    inp = make_inputs(1, 64, 4096, 16, dtype="bf16", seed=16, with_h0=True)
    announce("time segments determinism (1, 64, 4096)")
    y1, h1 = gpu_fwd(inp)
    y2, h2 = gpu_fwd(inp)
    assert torch.equal(y1, y2) and torch.equal(h1, h2)


# ---- step ------------------------------------------------------------------

def test_verify_config_fwd_and_step():
    """Speculative-verify shape: 16 steps from h0 == one forward scan over the 16 bytes."""
    import paper_2401_13660_amd as mb
    inp = workload("verify_b32_L16")
    announce("verify (32, 3584, 16) fwd vs 16 x step")
    y, h = gpu_fwd(inp)
    check_against_oracle(inp, y, h)
    t = to_device(inp)
    state = t["h0"].clone()
    ys = []
    for s in range(inp.seqlen):
        ys.append(mb.scan_step(state, t["u"][..., s].contiguous(), t["delta"][..., s].contiguous(), t["A"],
                               t["B"][..., s].contiguous(), t["C"][..., s].contiguous(), D=t["Dskip"],
                               dt_bias=t["dt_bias"], z_t=t["z"][..., s].contiguous()))
    torch.cuda.synchronize()
    ys = torch.stack(ys, dim=2)
    check_against_oracle(inp, ys, state)
    from parity import rel_err
    assert rel_err(ys.cpu().numpy(), y.cpu().numpy()) <= 1e-5
    assert rel_err(state.cpu().numpy(), h.cpu().numpy()) <= 1e-5


@pytest.mark.parametrize("N", [1, 4, 16])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_step_against_oracle(N, dtype):
    import oracle
    import paper_2401_13660_amd as mb
    from parity import rel_err
    inp = make_inputs(3, 77, 1, N, dtype=dtype, seed=14, with_h0=True)
    announce(f"step N={N} {dtype} (3, 77)")
    t = to_device(inp)
    state = t["h0"].clone()
    y = mb.scan_step(state, t["u"][..., 0].contiguous(), t["delta"][..., 0].contiguous(), t["A"],
                     t["B"][..., 0].contiguous(), t["C"][..., 0].contiguous(), D=t["Dskip"],
                     dt_bias=t["dt_bias"], z_t=t["z"][..., 0].contiguous())
    torch.cuda.synchronize()
    yr, hr = oracle.default().scan_step(inp.h0, inp.u[..., 0], inp.delta[..., 0], inp.A, inp.B[..., 0],
                                        inp.C[..., 0], z_t=inp.z[..., 0], Dskip=inp.Dskip,
                                        dt_bias=inp.dt_bias, dtype=inp.dtype)
    assert rel_err(y.cpu().numpy(), yr) <= 2e-3
    assert rel_err(state.cpu().numpy(), hr) <= 1e-4


@pytest.mark.parametrize("N", [1, 16])
@pytest.mark.parametrize("softplus", [True, False])
def test_step_without_optional_inputs(N, softplus):
    """A step with no gate, no skip term and no timestep bias: the kernel reads
    same-sized stand-ins for the absent inputs and must discard their values."""
    import oracle
    import paper_2401_13660_amd as mb
    from parity import rel_err
    inp = make_inputs(2, 45, 1, N, dtype="bf16", seed=15, with_h0=True)
    announce(f"step without z, Dskip, dt_bias: N={N} softplus={softplus}")
    t = to_device(inp)
    delta = t["delta"][..., 0].contiguous()
    if not softplus:                       # dlt = delta as given: keep it small and positive
        delta = (delta.float().abs() * 0.05).to(delta.dtype)
    state = t["h0"].clone()
    y = mb.scan_step(state, t["u"][..., 0].contiguous(), delta, t["A"], t["B"][..., 0].contiguous(),
                     t["C"][..., 0].contiguous(), delta_softplus=softplus)
    torch.cuda.synchronize()
    delta_bits = delta.cpu().view(torch.int16).numpy().view(np.uint16)      # the bf16 bits the GPU read
    yr, hr = oracle.default().scan_step(inp.h0, inp.u[..., 0], delta_bits, inp.A,
                                        inp.B[..., 0], inp.C[..., 0], delta_softplus=softplus, dtype=inp.dtype)
    assert rel_err(y.cpu().numpy(), yr) <= 2e-3
    assert rel_err(state.cpu().numpy(), hr) <= 1e-4

"""GPU parity of mb_scan_fwd_states: the state at requested positions.

Algorithm 1 (Appendix F) verifies drafted bytes with one parallel scan and then
continues from the state at the bifurcation position c.  The recorded states
are compared with the fp64 oracle's states at the same positions (tolerance
1e-4 under the metric of tests/parity.py, as for h_last); slots of invalid
positions must read NaN; y and h_last must be the same bits as a call without
positions; a state recorded at L - 1 must equal h_last bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, has_gpu, to_device
from parity import rel_err
from paper_2401_13660_amd.inputs import make_inputs, workload

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]

TOL_H = 1e-4


def position_table(L, nb, seed, extra_random=4):
    """(npos, nb) int32: chunk and segment edges, both ends, a repeat, invalid ones."""
    base = [-1, 0, 1, 15, 16, 31, 32, 33, L // 2, L - 17, L - 16, L - 2, L - 1, L - 1, L, -7]
    rng = np.random.default_rng(seed)
    cols = []
    for b in range(nb):
        col = [p if p in (-1, L, -7) else min(max(p + b, 0), L - 1) for p in base]
        col += list(rng.integers(0, L, extra_random))
        cols.append(col)
    return np.array(cols, dtype=np.int32).T.copy()


def run_states(inp, pos, **kw):
    import paper_2401_13660_amd as mb
    t = to_device(inp)
    pos_d = torch.from_numpy(pos).to("cuda:0")
    y, h_last, h_at = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t.get("Dskip"),
                                  dt_bias=t.get("dt_bias"), z=t.get("z"), h0=t.get("h0"),
                                  return_last_state=True, positions=pos_d, **kw)
    y0, h0_last = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t.get("Dskip"),
                              dt_bias=t.get("dt_bias"), z=t.get("z"), h0=t.get("h0"),
                              return_last_state=True, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y, y0), "recording positions changed y"
    assert torch.equal(h_last, h0_last), "recording positions changed h_last"
    return y, h_last, h_at


def check_states(inp, pos, h_at, h_last, rows=None):
    """Recorded states of (sampled) rows against the oracle's, position by position."""
    nb, dim, L = inp.u.shape
    npos = pos.shape[0]
    rows = np.arange(nb * dim) if rows is None else np.asarray(rows)
    _, _, h_ref = oracle.scan_inputs(inp, rows=rows, positions=pos)          # (npos, R, N)
    g32 = h_at.cpu().numpy().reshape(npos, nb * dim, -1)[:, rows]
    hl32 = h_last.cpu().numpy().reshape(nb * dim, -1)[rows]
    g = g32.astype(np.float64)
    bsel = rows // dim
    worst = 0.0
    for k in range(npos):
        for b in range(nb):
            m = bsel == b
            if not m.any():
                continue
            p = int(pos[k, b])
            if p < -1 or p >= L:
                assert np.all(np.isnan(g[k][m])), f"position {p}: slot not NaN"
                continue
            e = rel_err(g[k][m], h_ref[k][m])
            worst = max(worst, e)
            assert e <= TOL_H, f"state at position {p} (k {k}, b {b}): relative error {e:.3e}"
            if p == L - 1:
                assert np.array_equal(g32[k][m], hl32[m]), "state at L-1 differs from h_last"
    return worst


# (batch, dim, L): tiled with a half chunk and dead lanes; row-per-thread
# (L % 16 != 0); time-segmented shapes (few rows), where positions fall in
# later segments; a short verify-like length.
@pytest.mark.parametrize("shape", [(2, 200, 1008), (2, 130, 1000), (1, 64, 4096), (1, 8, 640),
                                   (3, 72, 4112), (4, 96, 16)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_states_at_positions(shape, dtype):
    nb, dim, L = shape
    inp = make_inputs(nb, dim, L, 16, dtype=dtype, seed=11, with_h0=True)
    pos = position_table(L, nb, seed=12)
    announce(f"states at {pos.shape[0]} positions, shape {shape} {dtype}")
    _, h_last, h_at = run_states(inp, pos)
    check_states(inp, pos, h_at, h_last)


@pytest.mark.parametrize("N", [4, 16])
def test_states_without_h0_and_small_dstate(N):
    inp = make_inputs(2, 40, 96, N, dtype="bf16", seed=13, with_h0=False)
    pos = position_table(96, 2, seed=14)
    announce(f"states, no h0, N={N}")
    _, h_last, h_at = run_states(inp, pos)
    check_states(inp, pos, h_at, h_last)


def test_states_seqlen_zero():
    inp = make_inputs(2, 24, 16, 16, dtype="bf16", seed=15, with_h0=True)
    import paper_2401_13660_amd as mb
    t = to_device(inp)
    pos = torch.tensor([[-1, 0], [3, -1]], dtype=torch.int32, device="cuda:0")
    announce("states with L = 0")
    e = lambda x: x[..., :0].contiguous()
    y, h_at = mb.scan_fwd(e(t["u"]), e(t["delta"]), t["A"], e(t["B"]), e(t["C"]), D=t["Dskip"],
                          dt_bias=t["dt_bias"], z=e(t["z"]), h0=t["h0"], positions=pos)
    torch.cuda.synchronize()
    assert y.numel() == 0
    h0 = t["h0"]
    assert torch.equal(h_at[0, 0], h0[0]) and torch.equal(h_at[1, 1], h0[1])
    assert torch.isnan(h_at[0, 1]).all() and torch.isnan(h_at[1, 0]).all()


def test_resume_from_recorded_state():
    """Verify-then-continue: the state at c, passed back as h0 for bytes c+1 .. L-1,
    reproduces the tail of the single scan (Section 3, resumable scan)."""
    import paper_2401_13660_amd as mb
    nb, dim, L, c = 2, 96, 2048, 1234
    inp = make_inputs(nb, dim, L, 16, dtype="bf16", seed=16, with_h0=True)
    t = to_device(inp)
    announce(f"resume from the state at c = {c}")
    pos = torch.full((1, nb), c, dtype=torch.int32, device="cuda:0")
    y, h_last, h_at = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t["Dskip"],
                                  dt_bias=t["dt_bias"], z=t["z"], h0=t["h0"], return_last_state=True,
                                  positions=pos)
    tail = lambda x: x[..., c + 1:].contiguous()
    y2, h2 = mb.scan_fwd(tail(t["u"]), tail(t["delta"]), t["A"], tail(t["B"]), tail(t["C"]),
                         D=t["Dskip"], dt_bias=t["dt_bias"], z=tail(t["z"]), h0=h_at[0].contiguous(),
                         return_last_state=True)
    torch.cuda.synchronize()
    ey = rel_err(y2.cpu().numpy().astype(np.float64), y[..., c + 1:].cpu().numpy().astype(np.float64))
    eh = rel_err(h2.cpu().numpy().astype(np.float64), h_last.cpu().numpy().astype(np.float64))
    assert ey <= 1e-5 and eh <= 1e-5, (ey, eh)


def test_states_verify_config_every_position():
    """The verify workload (batch 32, L 16, from a carried state): every position -1 .. 15."""
    inp = workload("verify_b32_L16", seed=0)
    nb, dim, L = inp.u.shape
    pos = np.repeat(np.arange(-1, L, dtype=np.int32)[:, None], nb, axis=1).copy()
    announce(f"verify config, {pos.shape[0]} positions x batch {nb}")
    _, h_last, h_at = run_states(inp, pos)
    check_states(inp, pos, h_at, h_last)


def test_states_972m_layer_sampled_rows():
    """The MambaByte-972M layer shape at full size, one bifurcation per batch element,
    checked on sampled rows."""
    inp = workload("mambabyte972m_L8192", seed=0)
    nb, dim, L = inp.u.shape
    pos = np.array([[5000 + 997 * b for b in range(nb)], [L - 1] * nb, [31 + b for b in range(nb)]],
                   dtype=np.int32)
    rng = np.random.default_rng(17)
    rows = np.sort(rng.choice(nb * dim, 48, replace=False))
    announce("972M layer (4, 3584, 8192), 3 positions per batch element, 48 sampled rows")
    _, h_last, h_at = run_states(inp, pos)
    check_states(inp, pos, h_at, h_last, rows=rows)

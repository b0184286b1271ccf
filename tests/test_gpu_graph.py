"""HIP-graph capture of the launch-bound paths: the 16 one-byte steps of a
verify chunk and the one-chunk verify scan.  Each replay (with eager work of
the program between replays) must give the bits of the eager calls, and the
16 captured steps must also agree with the oracle."""
import numpy as np
import pytest
import torch

from gpu_util import announce, check_against_oracle, has_gpu, to_device
from paper_2401_13660_amd.inputs import make_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_graph_of_sixteen_steps():
    import paper_2401_13660_amd as mb
    inp = make_inputs(6, 136, 16, 16, dtype="bf16", seed=81, with_h0=True)
    announce("HIP graph of 16 mb_scan_step calls (6, 136)")
    t = to_device(inp)
    cols = [{k: t[k][..., i].contiguous() for k in ("u", "delta", "B", "C", "z")} for i in range(16)]
    h = torch.empty_like(t["h0"])
    ys = [torch.empty((6, 136), dtype=torch.float32, device="cuda:0") for _ in range(16)]

    def steps():
        for i, c in enumerate(cols):
            mb.scan_step(h, c["u"], c["delta"], t["A"], c["B"], c["C"], D=t["Dskip"], dt_bias=t["dt_bias"],
                         z_t=c["z"], out=ys[i])

    h.copy_(t["h0"])
    steps()
    torch.cuda.synchronize()
    y_eager, h_eager = torch.stack(ys, dim=2).clone(), h.clone()
    check_against_oracle(inp, y_eager, h_eager)

    h.copy_(t["h0"])
    g = _capture(steps)
    for r in range(3):
        h.copy_(t["h0"])                              # eager work between replays
        for y in ys:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(torch.stack(ys, dim=2), y_eager), f"replay {r}: y differs from the eager steps"
        assert torch.equal(h, h_eager), f"replay {r}: h differs from the eager steps"


def test_graph_of_verify_scan():
    import paper_2401_13660_amd as mb
    inp = make_inputs(6, 136, 16, 16, dtype="bf16", seed=82, with_h0=True)
    announce("HIP graph of one mb_scan_fwd, L = 16 (6, 136)")
    t = to_device(inp)
    y = torch.empty(inp.u.shape, dtype=torch.float32, device="cuda:0")
    hl = torch.empty_like(t["h0"])

    def call():
        mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t["Dskip"], dt_bias=t["dt_bias"], z=t["z"],
                    h0=t["h0"], out=y, h_last=hl)

    call()
    torch.cuda.synchronize()
    y_eager, h_eager = y.clone(), hl.clone()
    g = _capture(call)
    for r in range(3):
        y.fill_(float("nan"))
        hl.zero_()
        call()                                        # an eager call between replays
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager) and torch.equal(hl, h_eager), f"replay {r} differs from the eager call"


def test_graph_of_segmented_scan():
    """Few rows and a long sequence: the captured call holds the stream-ordered
    allocation of the segment carry, the pre-pass, the scan and the free."""
    import paper_2401_13660_amd as mb
    inp = make_inputs(1, 64, 4096, 16, dtype="bf16", seed=83, with_h0=True)
    announce("HIP graph of one time-segmented mb_scan_fwd (1, 64, 4096)")
    t = to_device(inp)
    y = torch.empty(inp.u.shape, dtype=torch.float32, device="cuda:0")
    hl = torch.empty_like(t["h0"])

    def call():
        mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t["Dskip"], dt_bias=t["dt_bias"], z=t["z"],
                    h0=t["h0"], out=y, h_last=hl)

    call()
    torch.cuda.synchronize()
    y_eager, h_eager = y.clone(), hl.clone()
    check_against_oracle(inp, y_eager, h_eager)
    g = _capture(call)
    for r in range(3):
        y.fill_(float("nan"))
        hl.zero_()
        call()                                        # an eager call between replays
        y.fill_(float("nan"))
        hl.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager) and torch.equal(hl, h_eager), f"replay {r} differs from the eager call"


def test_graph_of_training_pair():
    """Forward with checkpoints, then the backward from them (its workspace is a
    stream-ordered allocation inside the captured region)."""
    import paper_2401_13660_amd as mb
    inp = make_inputs(2, 200, 1008, 16, dtype="bf16", seed=84, with_h0=True)
    announce("HIP graph of mb_scan_fwd_ckpt + mb_scan_bwd (2, 200, 1008)")
    t = to_device(inp)
    rng = np.random.default_rng(85)
    dy = torch.from_numpy(rng.standard_normal(inp.u.shape).astype(np.float32)).to("cuda:0")
    y = torch.empty(inp.u.shape, dtype=torch.float32, device="cuda:0")
    ck = torch.empty((inp.seqlen // 16, inp.batch, inp.dim, 16), dtype=torch.float32, device="cuda:0")
    kw = dict(D=t["Dskip"], dt_bias=t["dt_bias"], z=t["z"], h0=t["h0"])
    out = {}

    def pair():
        mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], out=y, ck=ck, **kw)
        out.update(mb.scan_bwd(t["u"], t["delta"], t["A"], t["B"], t["C"], dy, ck=ck, **kw))

    pair()
    torch.cuda.synchronize()
    ref = {k: (v.clone() if v is not None else None) for k, v in out.items()}
    y_ref = y.clone()
    g = _capture(pair)
    captured = dict(out)                              # the tensors the graph writes
    for r in range(3):
        pair()                                        # eager work between replays
        for v in captured.values():
            if v is not None:
                v.fill_(float("nan"))
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), f"replay {r}: y differs"
        for k, v in captured.items():
            if v is not None:
                assert torch.equal(v, ref[k]), f"replay {r}: {k} differs from the eager pair"

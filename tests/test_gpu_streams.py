"""Calls on two streams at once (default priority): each call works on the
stream it is given, with its own stream-ordered workspace, so concurrent
forward and backward calls give the bits of the same calls made one after the
other."""
import pytest
import torch

from gpu_util import announce, has_gpu, to_device
from paper_2401_13660_amd.inputs import make_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]


def test_two_streams_forward_and_backward():
    import paper_2401_13660_amd as mb
    cases = [make_inputs(2, 200, 1008, 16, dtype="bf16", seed=91 + i, with_h0=True) for i in range(2)]
    announce("forward and backward on two concurrent streams")
    ts = [to_device(c) for c in cases]
    dys = [torch.randn(c.u.shape, generator=torch.Generator().manual_seed(7 + i)).to("cuda:0")
           for i, c in enumerate(cases)]

    def run(t, dy):
        kw = dict(D=t["Dskip"], dt_bias=t["dt_bias"], z=t["z"], h0=t["h0"])
        y, hl = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], return_last_state=True, **kw)
        g = mb.scan_bwd(t["u"], t["delta"], t["A"], t["B"], t["C"], dy, **kw)
        return [y, hl] + [g[k] for k in sorted(g) if g[k] is not None]

    serial = [run(t, dy) for t, dy in zip(ts, dys)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    outs = []
    for s, t, dy in zip(streams, ts, dys):
        with torch.cuda.stream(s):
            outs.append(run(t, dy))
    torch.cuda.synchronize()
    for i in range(2):
        for a, b in zip(outs[i], serial[i]):
            assert torch.equal(a, b), f"case {i}: a concurrent result differs from the serial one"

"""GPU parity of mb_verify_rank (the top-beta check of drafted bytes) against the
oracle: ranks, accepted counts and last positions are integers, compared exactly,
with both sides reading the same logit bits."""
import numpy as np
import pytest
import torch

import oracle
from oracle import verify_rank as VR
from gpu_util import announce, dev_tensor, has_gpu
from parity import rel_err
from paper_2401_13660_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits, make_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not has_gpu(), reason="needs a GPU")]


def logits_case(B, n, V, seed, dtype="f32", scale=1.0):
    rng = np.random.default_rng(seed)
    lg = (rng.standard_normal((B, n, V)) * scale).astype(np.float32)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(lg).reshape(lg.shape)
        return bits, bf16_bits_to_f32(bits).reshape(lg.shape).astype(np.float64)
    return lg, lg.astype(np.float64)


def check(lg_dev_src, lg64, draft, beta):
    import paper_2401_13660_amd as mb
    acc, last, ranks = mb.verify_rank(dev_tensor(lg_dev_src), dev_tensor(draft), beta, return_ranks=True)
    torch.cuda.synchronize()
    r_ref = VR.ranks(lg64, draft)
    a_ref = VR.accepted(r_ref, beta)
    assert np.array_equal(ranks.cpu().numpy(), r_ref), "ranks differ"
    assert np.array_equal(acc.cpu().numpy(), a_ref), "accepted differ"
    assert np.array_equal(last.cpu().numpy(), a_ref - 1), "last positions differ"
    return a_ref


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("beta", [0, 1, 3, 256])
def test_rank_verify_shape(dtype, beta):
    """batch 32, 16 drafted bytes, 256-way byte logits; drafts biased towards good bytes
    so that accepted prefixes of every length occur."""
    B, n, V = 32, 16, 256
    lg, lg64 = logits_case(B, n, V, 41, dtype)
    rng = np.random.default_rng(42)
    order = np.argsort(-lg64, axis=2, kind="stable")
    pick = np.minimum(rng.geometric(0.5, (B, n)) - 1, V - 1)        # mostly top few
    draft = np.take_along_axis(order, pick[..., None], axis=2)[..., 0].astype(np.int32)
    announce(f"rank check ({B}, {n}, {V}) {dtype} beta={beta}")
    a = check(lg, lg64, draft, beta)
    if beta == 3:
        assert len(set(a.tolist())) > 3, "the case should exercise several prefix lengths"


def test_rank_edge_cases():
    B, n, V = 6, 9, 1000                      # vocab not a multiple of 64
    lg, lg64 = logits_case(B, n, V, 43)
    lg = np.round(lg * 2) / 2                 # ties
    lg64 = lg.astype(np.float64)
    draft = np.random.default_rng(44).integers(0, V, (B, n)).astype(np.int32)
    draft[0, 0] = -3                          # out of range: rejected at once
    draft[1, 4] = V
    lg[2, 1, draft[2, 1]] = np.nan            # NaN score: rejected
    lg64[2, 1, draft[2, 1]] = np.nan
    draft[3] = np.argmax(lg64[3], axis=1)     # all rank 1
    announce("rank edge cases")
    for beta in (1, 500, 1000):
        check(lg, lg64, draft, beta)


@pytest.mark.parametrize("n", [0, 1, 100])
def test_rank_draft_lengths(n):
    lg, lg64 = logits_case(5, n, 256, 45 + n)
    draft = np.random.default_rng(46).integers(0, 256, (5, n)).astype(np.int32)
    announce(f"rank n={n}")
    import paper_2401_13660_amd as mb
    if n == 0:
        acc, last = mb.verify_rank(torch.empty((5, 0, 256), device="cuda:0"),
                                   torch.empty((5, 0), dtype=torch.int32, device="cuda:0"), 3)
        torch.cuda.synchronize()
        assert acc.tolist() == [0] * 5 and last.tolist() == [-1] * 5
        return
    check(lg, lg64, draft, 200)


def test_verify_chain_rank_then_state():
    """Algorithm 1 on the device: scan the drafted chunk from the carried state, rank the
    drafts, and read the state at each row's last accepted byte, with no host round trip."""
    import paper_2401_13660_amd as mb
    inp = make_inputs(8, 256, 16, 16, dtype="bf16", seed=47, with_h0=True)
    t = {k: dev_tensor(v) for k, v in inp.arrays().items()}
    lg, lg64 = logits_case(8, 16, 256, 48)
    order = np.argsort(-lg64, axis=2, kind="stable")
    pick = np.minimum(np.random.default_rng(49).geometric(0.45, (8, 16)) - 1, 255)
    draft = np.take_along_axis(order, pick[..., None], axis=2)[..., 0].astype(np.int32)
    announce("verify chain: rank -> state at the bifurcation")
    acc, last = mb.verify_rank(dev_tensor(lg), dev_tensor(draft), 3)
    y, h_at = mb.scan_fwd(t["u"], t["delta"], t["A"], t["B"], t["C"], D=t["Dskip"], dt_bias=t["dt_bias"],
                          z=t["z"], h0=t["h0"], positions=last.view(1, -1))
    torch.cuda.synchronize()
    a_ref = VR.accepted(VR.ranks(lg64, draft), 3)
    pos = (a_ref - 1).reshape(1, -1)
    _, _, h_ref = oracle.scan_inputs(inp, positions=pos)
    assert np.array_equal(acc.cpu().numpy(), a_ref)
    assert rel_err(h_at.cpu().numpy(), h_ref) <= 1e-4

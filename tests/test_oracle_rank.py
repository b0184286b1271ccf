"""Pins of the top-beta rank oracle (oracle/verify_rank.py), on the CPU.

The rank is re-derived through sorting (a different route than counting), is
checked for invariance under monotone transforms of the logits (softmax,
temperature), and the accepted count is checked against the first-rejection
index of Algorithm 1's formula.  Planted mistakes must fail at least one pin.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import verify_rank as VR


def _case(seed, B=6, n=9, V=40, ties=True):
    rng = np.random.default_rng(seed)
    lg = rng.standard_normal((B, n, V))
    if ties:
        lg = np.round(lg * 2) / 2                    # many equal logits
    draft = rng.integers(0, V, (B, n))
    return lg, draft


def _rank_by_sorting(lg, draft):
    """1 + number of strictly larger candidates, read off the sorted logits."""
    B, n, V = lg.shape
    out = np.empty((B, n), dtype=np.int64)
    for b in range(B):
        for i in range(n):
            x = draft[b, i]
            if x < 0 or x >= V or np.isnan(lg[b, i, x]):
                out[b, i] = V + 1
                continue
            asc = np.sort(lg[b, i])
            # entries after the last one <= logit[x] are the strictly larger ones
            out[b, i] = 1 + (V - np.searchsorted(asc, lg[b, i, x], side="right"))
    return out


def pin_rank_sorting(ranks_fn, accepted_fn):
    for seed in range(4):
        lg, dr = _case(seed)
        assert np.array_equal(ranks_fn(lg, dr), _rank_by_sorting(lg, dr)), f"rank seed {seed}"


def pin_rank_monotone_invariance(ranks_fn, accepted_fn):
    lg, dr = _case(7)
    r = ranks_fn(lg, dr)
    p = np.exp(lg - lg.max(axis=2, keepdims=True))
    p /= p.sum(axis=2, keepdims=True)
    for t in (2.0 * lg + 3.0, p, lg / 0.7):
        assert np.array_equal(ranks_fn(t, dr), r), "rank changed under a monotone transform"


def pin_rank_top1_is_argmax(ranks_fn, accepted_fn):
    lg, _ = _case(8, ties=False)
    dr = np.argmax(lg, axis=2)
    assert np.all(ranks_fn(lg, dr) == 1), "the argmax byte must have rank 1"
    dr2 = np.argmin(lg, axis=2)
    assert np.all(ranks_fn(lg, dr2) == lg.shape[2]), "the argmin byte must have rank V"


def pin_rank_invalid(ranks_fn, accepted_fn):
    lg, dr = _case(9)
    V = lg.shape[2]
    dr = dr.copy()
    dr[0, 0], dr[1, 2] = -1, V
    lg = lg.copy()
    lg[2, 3, dr[2, 3]] = np.nan
    r = ranks_fn(lg, dr)
    assert r[0, 0] == V + 1 and r[1, 2] == V + 1 and r[2, 3] == V + 1, "invalid drafts must be rejected"


def pin_accepted_formula(ranks_fn, accepted_fn):
    """accepted = (first i, 1-based, with rank_i > beta) - 1, or n when none is rejected."""
    rng = np.random.default_rng(10)
    r = rng.integers(1, 8, (50, 7))
    for beta in (0, 1, 3, 7, 8):
        got = accepted_fn(r, beta)
        for b in range(r.shape[0]):
            bad = [i + 1 for i in range(r.shape[1]) if r[b, i] > beta]
            want = (bad[0] - 1) if bad else r.shape[1]
            assert got[b] == want, f"accepted beta {beta} row {b}: {got[b]} != {want}"


PINS = [pin_rank_sorting, pin_rank_monotone_invariance, pin_rank_top1_is_argmax, pin_rank_invalid,
        pin_accepted_formula]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_rank_pins(pin):
    pin(VR.ranks, VR.accepted)


# ---- planted mistakes ---------------------------------------------------------

def _ranks_ge(lg, dr):                      # ties counted against the draft
    lg = np.asarray(lg, np.float64)
    B, n, V = lg.shape
    out = np.empty((B, n), np.int64)
    for b in range(B):
        for i in range(n):
            x = dr[b, i]
            out[b, i] = V + 1 if (x < 0 or x >= V or np.isnan(lg[b, i, x])) else \
                np.count_nonzero(lg[b, i] >= lg[b, i, x])
    return out


def _ranks_zero_based(lg, dr):
    return VR.ranks(lg, dr) - 1


def _ranks_ascending(lg, dr):               # counts the smaller ones
    return VR.ranks(-np.asarray(lg, np.float64), dr)


def _ranks_nan_accepted(lg, dr):
    lg = np.nan_to_num(np.asarray(lg, np.float64), nan=np.inf)
    return VR.ranks(lg, dr)


def _accepted_any(rank, beta):              # counts all accepted, not the prefix
    return np.sum(np.asarray(rank) <= beta, axis=1)


def _accepted_first_reject(rank, beta):     # the printed formula, 1-based
    rank = np.asarray(rank)
    out = []
    for row in rank:
        bad = np.nonzero(row > beta)[0]
        out.append(bad[0] + 1 if bad.size else row.size)
    return np.array(out)


MUTANTS = [("ties_count_against", _ranks_ge, VR.accepted),
           ("zero_based", _ranks_zero_based, VR.accepted),
           ("ascending", _ranks_ascending, VR.accepted),
           ("nan_accepted", _ranks_nan_accepted, VR.accepted),
           ("accepted_not_prefix", VR.ranks, _accepted_any),
           ("accepted_first_reject_index", VR.ranks, _accepted_first_reject)]


@pytest.mark.parametrize("name,rf,af", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_rank_pins_catch_mutant(name, rf, af):
    failed = 0
    for pin in PINS:
        try:
            pin(rf, af)
        except AssertionError:
            failed += 1
    assert failed, f"no pin caught the planted mistake {name!r}"

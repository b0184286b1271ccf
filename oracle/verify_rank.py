"""The top-beta rank check of drafted bytes -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the product path never calls it.

Speculative decoding verifies each drafted byte against the byte-level model's
next-byte distribution p_i and accepts the draft up to the furthest position
whose bytes all lie among the model's top-beta candidates (Section 3,
"Speculative decoding through subword drafting"; Appendix F, Algorithm 1, with
beta = 3 in Table 6).  Written out plainly:

    rank_i   = 1 + #{y : logit_i[y] > logit_i[x_i]}       x_i = the drafted byte at i
               (a softmax, with or without temperature, is monotone, so logits rank
               exactly like probabilities; ties do not count against x_i)
    rank_i   = vocab + 1 when x_i is outside [0, vocab) or its logit is NaN
    accepted = the number of leading positions with rank_i <= beta   (0 .. n)

``accepted`` is the bifurcation position c of Algorithm 1's comment (drafted
bytes 1..c verified, byte c+1 not); its printed formula min{i | rank_i > beta}
is the first rejected index, i.e. c + 1 when some byte is rejected.
"""
from __future__ import annotations

import numpy as np


def ranks(logits, draft) -> np.ndarray:
    """logits: (B, n, V) floats; draft: (B, n) integers.  Returns (B, n) int64."""
    lg = np.asarray(logits, dtype=np.float64)
    dr = np.asarray(draft, dtype=np.int64)
    B, n, V = lg.shape
    out = np.empty((B, n), dtype=np.int64)
    for b in range(B):
        for i in range(n):
            x = dr[b, i]
            if x < 0 or x >= V or np.isnan(lg[b, i, x]):
                out[b, i] = V + 1
            else:
                out[b, i] = 1 + int(np.count_nonzero(lg[b, i] > lg[b, i, x]))
    return out


def accepted(rank, beta) -> np.ndarray:
    """(B, n) ranks -> (B,) count of leading positions with rank <= beta."""
    rank = np.asarray(rank)
    B, n = rank.shape
    out = np.zeros(B, dtype=np.int64)
    for b in range(B):
        a = 0
        while a < n and rank[b, a] <= beta:
            a += 1
        out[b] = a
    return out

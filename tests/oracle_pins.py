"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees.  None of them re-types the oracle's recurrence:
they use the continuous-time closed form on the grid t_k = sum Delta
(Section 2 after eq. (2)), the geometric series, special cases with textbook
answers (Appendix D, eq. (4); the Delta limits stated after it), the
associative tuple scan of Section 2 "Implementation", and structural
invariants (split/resume, state separability, linearity, step == forward).
``tests/test_oracle_mutants.py`` checks that these pins catch plausible bugs.
"""
from __future__ import annotations

import json
import os
import sys
from decimal import Decimal

import numpy as np
from scipy.special import expit

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bruteforce_tiny.json")


def _softplus_ref(v):
    # log(1 + e^v) as log(e^0 + e^v): a library routine, not the oracle's log1p form.
    return np.logaddexp(0.0, v)


def _relerr(g, r):
    g = np.asarray(g, np.float64).ravel()
    r = np.asarray(r, np.float64).ravel()
    den = np.abs(r) + np.sqrt(np.mean(r * r)) + 1e-300
    return float(np.max(np.abs(g - r) / den))


def _close(g, r, tol, what):
    e = _relerr(g, r)
    assert e <= tol, f"{what}: relative error {e:.3e} > {tol:.1e}"


def _rand_case(seed, nb=2, dim=3, L=40, N=4, *, gated=True, h0=True, D=True, bias=True):
    rng = np.random.default_rng(seed)
    c = dict(
        u=rng.standard_normal((nb, dim, L)),
        delta=rng.standard_normal((nb, dim, L)),
        A=-rng.uniform(0.1, 4.0, (dim, N)),
        B=rng.standard_normal((nb, N, L)),
        C=rng.standard_normal((nb, N, L)),
        z=rng.standard_normal((nb, dim, L)) if gated else None,
        Dskip=rng.uniform(0.5, 1.5, dim) if D else None,
        dt_bias=rng.uniform(-3.0, 0.5, dim) if bias else None,
        h0=0.5 * rng.standard_normal((nb, dim, N)) if h0 else None,
    )
    return c


def _run(orc, c, **kw):
    return orc.scan_fwd(c["u"], c["delta"], c["A"], c["B"], c["C"], z=c["z"], Dskip=c["Dskip"],
                        dt_bias=c["dt_bias"], h0=c["h0"], **kw)


def _brute(c, delta_softplus=True, all_states=False):
    """Time-grid closed form of every state (eq. (1) solved on t_k = sum Delta).
    With ``all_states`` also returns h_t for every t, shape (nb, dim, L, N)."""
    u, A, Bm, Cm = c["u"], c["A"], c["B"], c["C"]
    nb, dim, L = u.shape
    N = A.shape[1]
    y = np.zeros((nb, dim, L))
    h_last = np.zeros((nb, dim, N))
    h_all = np.zeros((nb, dim, L, N))
    for b in range(nb):
        for d in range(dim):
            v = c["delta"][b, d] + (0.0 if c["dt_bias"] is None else c["dt_bias"][d])
            dl = _softplus_ref(v) if delta_softplus else v
            S = np.cumsum(dl)                       # S_t = t-th grid point
            h0 = np.zeros(N) if c["h0"] is None else c["h0"][b, d]
            for t in range(L):
                w = np.exp(np.outer(A[d], S[t] - S[: t + 1]))          # (N, t+1) decay from s to t
                inp = dl[: t + 1] * Bm[b, :, : t + 1] * u[b, d, : t + 1]  # Euler B-bar x at each s
                h = np.exp(A[d] * S[t]) * h0 + (w * inp).sum(axis=1)
                h_all[b, d, t] = h
                yv = Cm[b, :, t] @ h + (0.0 if c["Dskip"] is None else c["Dskip"][d]) * u[b, d, t]
                if c["z"] is not None:
                    zz = c["z"][b, d, t]
                    yv = yv * zz * expit(zz)
                y[b, d, t] = yv
            h_last[b, d] = h if L > 0 else h0
    return (y, h_last, h_all) if all_states else (y, h_last)


# ---------------------------------------------------------------------------

def pin_golden_decimal(orc):
    """50-digit time-grid fixtures (tests/golden/bruteforce_tiny.json)."""
    with open(GOLDEN) as f:
        cases = json.load(f)
    for cs in cases:
        L, N = cs["L"], cs["N"]
        arr = lambda k, shape: np.array([float(v) for v in cs[k]]).reshape(shape)
        y, h = orc.scan_fwd(arr("u", (1, 1, L)), arr("delta", (1, 1, L)), arr("A", (1, N)),
                            arr("B", (1, N, L)), arr("C", (1, N, L)),
                            z=None if cs["z"] is None else arr("z", (1, 1, L)),
                            Dskip=np.array([float(cs["Dskip"])]),
                            dt_bias=np.array([float(cs["dt_bias"])]),
                            h0=None if cs["h0"] is None else arr("h0", (1, 1, N)),
                            delta_softplus=cs["delta_softplus"])
        ry = np.array([float(Decimal(v)) for v in cs["y"]])
        rh = np.array([float(Decimal(v)) for v in cs["h_last"]])
        _close(y.ravel(), ry, 1e-13, f"golden {cs['name']} y")
        _close(h.ravel(), rh, 1e-13, f"golden {cs['name']} h_last")


def pin_bruteforce(orc):
    """Oracle == time-grid materialisation on small random inputs (several batches)."""
    for seed, kw in ((1, {}), (2, dict(gated=False, h0=False)), (3, dict(D=False, bias=False))):
        c = _rand_case(seed, **kw)
        y, h = _run(orc, c)
        ry, rh = _brute(c)
        _close(y, ry, 1e-11, f"bruteforce y seed {seed}")
        _close(h, rh, 1e-11, f"bruteforce h_last seed {seed}")
    # softplus off: Delta = delta_raw + bias, used as given (kept positive here)
    c = _rand_case(4)
    rng = np.random.default_rng(40)
    c["delta"] = rng.uniform(0.01, 0.3, c["u"].shape)
    c["dt_bias"] = rng.uniform(0.0, 0.05, c["A"].shape[0])
    y, h = _run(orc, c, delta_softplus=False)
    ry, rh = _brute(c, delta_softplus=False)
    _close(y, ry, 1e-11, "bruteforce (no softplus) y")
    _close(h, rh, 1e-11, "bruteforce (no softplus) h_last")


def pin_geometric(orc):
    """Constant Delta, B, x, C: h_t = a^(t+1) h0 + b (1 - a^(t+1)) / (1 - a)."""
    L, N = 300, 5
    A = -np.array([[0.05, 0.3, 1.0, 2.5, 7.0]])
    v, bias, x, Bv, Cv, D = 0.4, -1.1, 0.7, np.array([0.9, -1.3, 0.25, 2.0, -0.6]), \
        np.array([1.5, 0.2, -0.8, 0.33, 1.1]), 0.6
    h0 = np.array([0.3, -0.2, 1.0, 0.0, -0.7])
    dlt = float(np.logaddexp(0.0, v + bias))
    a = np.exp(dlt * A[0])
    b = dlt * Bv * x
    t = np.arange(L)[:, None]
    h_ref = a ** (t + 1) * h0 + b * (1 - a ** (t + 1)) / (1 - a)        # (L, N)
    y_ref = h_ref @ Cv + D * x
    y, h = orc.scan_fwd(np.full((1, 1, L), x), np.full((1, 1, L), v), A,
                        np.repeat(Bv[None, :, None], L, axis=2), np.repeat(Cv[None, :, None], L, axis=2),
                        Dskip=np.array([D]), dt_bias=np.array([bias]), h0=h0[None, None])
    _close(y.ravel(), y_ref, 1e-12, "geometric y")
    _close(h.ravel(), h_ref[-1], 1e-12, "geometric h_last")


def pin_B_zero(orc):
    """B = 0: with h0 = 0 the output is D x silu(z); with h0 the state only decays."""
    c = _rand_case(5, h0=False)
    c["B"] = np.zeros_like(c["B"])
    y, h = _run(orc, c)
    ref = c["Dskip"][None, :, None] * c["u"] * c["z"] * expit(c["z"])
    _close(y, ref, 1e-15, "B=0 y")
    assert np.all(h == 0.0), "B=0, h0=0: state must stay exactly zero"
    c = _rand_case(6, gated=False)
    c["B"] = np.zeros_like(c["B"])
    y, h = _run(orc, c)
    dl = _softplus_ref(c["delta"] + c["dt_bias"][None, :, None])
    S = np.cumsum(dl, axis=2)                                             # (nb, dim, L)
    hs = np.exp(c["A"][None, :, :, None] * S[:, :, None, :]) * c["h0"][..., None]  # (nb,dim,N,L)
    ry = np.einsum("bnl,bdnl->bdl", c["C"], hs) + c["Dskip"][None, :, None] * c["u"]
    _close(y, ry, 1e-13, "B=0 decaying h0 y")
    _close(h, hs[..., -1], 1e-13, "B=0 decaying h0 h_last")


def pin_split(orc):
    """Resume: scan[0:L] == scan[0:k] followed by scan[k:L] started from its h_last."""
    c = _rand_case(7, L=50)
    y, h = _run(orc, c)
    for k in (0, 1, 17, 49, 50):
        c1 = dict(c, u=c["u"][..., :k], delta=c["delta"][..., :k], z=c["z"][..., :k],
                  B=c["B"][..., :k], C=c["C"][..., :k])
        y1, h1 = _run(orc, c1)
        c2 = dict(c, u=c["u"][..., k:], delta=c["delta"][..., k:], z=c["z"][..., k:],
                  B=c["B"][..., k:], C=c["C"][..., k:], h0=h1)
        y2, h2 = _run(orc, c2)
        _close(np.concatenate([y1, y2], axis=2), y, 1e-13, f"split at {k}: y")
        _close(h2, h, 1e-13, f"split at {k}: h_last")


def pin_eq4(orc):
    """Appendix D, eq. (4): A = -1, N = 1 gives Abar = 1/(1 + e^v) = sigmoid(-v) = 1 - sigmoid(v).

    Observed through the oracle with B = 0, C = 1, h0 = 1, D = 0, no gate, L = 1
    (then y = Abar), and over a sequence with B = 1 where the scan must equal
    the gated recurrence h[k] = (1 - sigmoid(v_k)) h[k-1] + softplus(v_k) x[k]
    (the simplified-Euler B-bar = Delta replaces the ZOH B-bar of eq. (4))."""
    v = np.linspace(-30.0, 30.0, 241)
    R = v.size
    bias = 0.3
    y, _ = orc.scan_rows(np.ones((R, 1)), (v - bias)[:, None], -np.ones((R, 1)),
                         np.zeros((1, 1, 1)), np.ones((1, 1, 1)), np.zeros(R, np.int64),
                         dt_bias=np.full(R, bias), h0=np.ones((R, 1)))
    _close(y[:, 0], expit(-v), 1e-14, "eq.(4) Abar = sigmoid(-v)")
    _close(y[:, 0], 1.0 - expit(v), 1e-9, "eq.(4) Abar = 1 - sigmoid(v)")
    rng = np.random.default_rng(8)
    L = 64
    vs = rng.uniform(-6, 6, L)
    xs = rng.standard_normal(L)
    y, h = orc.scan_fwd(xs[None, None], vs[None, None], -np.ones((1, 1)), np.ones((1, 1, L)),
                        np.ones((1, 1, L)), h0=np.full((1, 1, 1), 0.25))
    hh, ref = 0.25, []
    for k in range(L):
        hh = (1.0 - expit(vs[k])) * hh + _softplus_ref(vs[k]) * xs[k]
        ref.append(hh)
    _close(y.ravel(), ref, 1e-12, "eq.(4) gated recurrence")


def pin_tuple_scan(orc):
    """Section 2 "Implementation": a Hillis-Steele scan with e_j . e_k = (A_k A_j, A_k b_j + b_k)."""
    c = _rand_case(9, nb=1, dim=2, L=37, N=3, gated=False)
    y, h = _run(orc, c)
    nb, dim, L = c["u"].shape
    for d in range(dim):
        dl = _softplus_ref(c["delta"][0, d] + c["dt_bias"][d])
        a = np.exp(np.outer(dl, c["A"][d]))                               # (L, N)
        b = dl[:, None] * c["B"][0].T * c["u"][0, d][:, None]              # (L, N)
        # prepend the carried state as the element (1, h0)
        a = np.vstack([np.ones((1, a.shape[1])), a])
        b = np.vstack([c["h0"][0, d][None], b])
        off = 1
        while off < a.shape[0]:
            a_new, b_new = a.copy(), b.copy()
            a_new[off:] = a[off:] * a[:-off]
            b_new[off:] = a[off:] * b[:-off] + b[off:]
            a, b, off = a_new, b_new, off * 2
        hs = b[1:]                                                         # (L, N) states
        ry = (hs * c["C"][0].T).sum(axis=1) + c["Dskip"][d] * c["u"][0, d]
        _close(y[0, d], ry, 1e-12, "tuple scan y")
        _close(h[0, d], hs[-1], 1e-12, "tuple scan h_last")


def pin_separability(orc):
    """Only C couples the states: y(N states, D=0) = sum_n y(state n alone)."""
    c = _rand_case(10, gated=False, D=False)
    y, h = _run(orc, c)
    acc = np.zeros_like(y)
    for n in range(c["A"].shape[1]):
        cn = dict(c, A=c["A"][:, n:n + 1], B=c["B"][:, n:n + 1], C=c["C"][:, n:n + 1],
                  h0=c["h0"][..., n:n + 1])
        yn, hn = _run(orc, cn)
        acc += yn
        _close(hn[..., 0], h[..., n], 1e-14, f"separability h_last state {n}")
    _close(acc, y, 1e-12, "separability y")


def pin_linearity(orc):
    """With h0 = 0 and no gate, y is linear in x for a fixed Delta."""
    c1 = _rand_case(11, gated=False, h0=False)
    c2 = dict(c1, u=np.random.default_rng(12).standard_normal(c1["u"].shape))
    al, be = 0.75, -1.5
    c3 = dict(c1, u=al * c1["u"] + be * c2["u"])
    y1, h1 = _run(orc, c1)
    y2, h2 = _run(orc, c2)
    y3, h3 = _run(orc, c3)
    _close(y3, al * y1 + be * y2, 1e-12, "linearity y")
    _close(h3, al * h1 + be * h2, 1e-12, "linearity h_last")


def pin_step_equals_fwd(orc):
    """L recurrent steps (the generation mode of Section 2) == one forward scan."""
    c = _rand_case(13, L=20)
    y, h = _run(orc, c)
    hh = c["h0"]
    ys = []
    for t in range(c["u"].shape[2]):
        yt, hh = orc.scan_step(hh, c["u"][..., t], c["delta"][..., t], c["A"], c["B"][..., t],
                               c["C"][..., t], z_t=c["z"][..., t], Dskip=c["Dskip"],
                               dt_bias=c["dt_bias"])
        ys.append(yt)
    _close(np.stack(ys, axis=2), y, 1e-15, "step x L == fwd: y")
    _close(hh, h, 1e-15, "step x L == fwd: h")


def pin_limits(orc):
    """After eq. (4): Delta -> 0 keeps the state; Delta -> inf forgets it (h -> Delta B x under Euler)."""
    c = _rand_case(14, gated=False, bias=False, L=16)
    c["delta"] = np.full_like(c["u"], -45.0)                               # Delta ~ 3e-20
    y, h = _run(orc, c)
    _close(h, c["h0"], 1e-15, "Delta->0: h_last == h0")
    ry = np.einsum("bnl,bdn->bdl", c["C"], c["h0"]) + c["Dskip"][None, :, None] * c["u"]
    _close(y, ry, 1e-15, "Delta->0: y == C h0 + D x")
    c["delta"] = np.full_like(c["u"], 45.0)                                # Abar = exp(-45 |A|) ~ 0
    c["A"] = np.minimum(c["A"], -1.0)
    y, h = _run(orc, c)
    ref_h = 45.0 * c["B"][:, None, :, -1] * c["u"][..., -1:]               # (nb, dim, N)
    _close(h, ref_h, 1e-15, "Delta->inf: h == Delta B x")


def pin_softplus_extremes(orc):
    """softplus(v) over [-80, 80] observed as h after one step with A = 0, B = 1, x = 1."""
    v = np.concatenate([np.linspace(-80, 80, 321), [-740.0, 0.0, 1e-8, 700.0, 720.0]])
    R = v.size
    y, h = orc.scan_rows(np.ones((R, 1)), v[:, None], np.zeros((R, 1)), np.ones((1, 1, 1)),
                         np.zeros((1, 1, 1)), np.zeros(R, np.int64))
    ref = _softplus_ref(v)
    _close(h[:, 0], ref, 1e-15, "softplus")
    # softplus > 0 everywhere: also hold every value to a plain relative bound, so
    # that a form which underflows or overflows (log(1 + e^v)) cannot hide.
    rel = np.max(np.abs(h[:, 0] - ref) / ref)
    assert rel <= 1e-14, f"softplus elementwise relative error {rel:.3e}"


def pin_states_at_positions(orc):
    """Appendix F, Algorithm 1 restarts from h_c: the state recorded at position p is
    the time-grid closed form of h_p, p = -1 is the initial state, and a position
    outside [-1, L-1] reads NaN; recording changes neither y nor h_last."""
    for seed, kw in ((7, {}), (8, dict(h0=False, gated=False))):
        c = _rand_case(seed, nb=3, dim=2, L=24, N=3, **kw)
        L = c["u"].shape[2]
        pos = np.array([[-1, 5, L + 6],        # position k = 0 of batch elements 0, 1, 2
                        [0, 5, -2],            # k = 1 (a repeat, an invalid position)
                        [L - 1, 11, L - 1]])   # k = 2
        y, h, hp = _run(orc, c, positions=pos)
        y0, h0_ = _run(orc, c)
        assert np.array_equal(y, y0) and np.array_equal(h, h0_), "positions changed y or h_last"
        ry, rh, rall = _brute(c, all_states=True)
        init = np.zeros_like(rh) if c["h0"] is None else c["h0"]
        for k in range(pos.shape[0]):
            for b in range(pos.shape[1]):
                p = pos[k, b]
                if p == -1:
                    ref = init[b]
                elif 0 <= p < L:
                    ref = rall[b, :, p]
                else:
                    assert np.all(np.isnan(hp[k, b])), f"invalid position {p} not NaN"
                    continue
                _close(hp[k, b], ref, 1e-11, f"state at position {p} (seed {seed}, k {k}, b {b})")


def _module_of(orc):
    """The module that defines the oracle under test (a mutated copy in the mutant tests)."""
    return sys.modules[type(orc).__module__]


def pin_bf16_decode(orc):
    """BF16 mixed precision (Section 4): the oracle reads a bf16 activation as the exact
    value its bit pattern encodes.  All 65,536 patterns are decoded and compared with
    torch's own bfloat16 -> float conversion (an independent library routine) and with
    hand-worked values; then a scan and a step given bit patterns must equal the same
    scan and step given the decoded values as floats."""
    import torch
    m = _module_of(orc)
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):                # signalling-NaN patterns
        got = m.to_f64(bits, "bf16")
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan), "bf16 NaN patterns decoded wrongly"
    assert np.array_equal(got[~nan], ref[~nan]), "bf16 decode differs from torch's conversion"
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan])), "bf16 sign decoded wrongly"
    # sign | 8-bit exponent (bias 127) | 7-bit fraction
    hand = {0x3F80: 1.0, 0xBF80: -1.0, 0x4000: 2.0, 0xC0A0: -5.0, 0x3FC0: 1.5, 0x4049: 3.140625,
            0x3C00: 2.0 ** -7, 0x0080: 2.0 ** -126, 0x0001: 2.0 ** -133, 0x8000: -0.0,
            0x7F80: np.inf, 0xFF80: -np.inf, 0x7F7F: (2.0 - 2.0 ** -7) * 2.0 ** 127}
    for b, v in hand.items():
        g = m.to_f64(np.array([b], np.uint16), "bf16")[0]
        assert g == v and np.signbit(g) == np.signbit(v), f"bf16 {b:#06x} -> {g!r}, expected {v!r}"
    # the same decode inside the scan and the step
    c = _rand_case(31, nb=2, dim=3, L=24, N=4)
    keys = ("u", "delta", "z", "B", "C")
    bf = {k: torch.from_numpy(np.asarray(c[k], np.float32)).to(torch.bfloat16) for k in keys}
    as_bits = {k: v.view(torch.int16).numpy().view(np.uint16) for k, v in bf.items()}
    as_vals = {k: v.to(torch.float64).numpy() for k, v in bf.items()}
    common = dict(Dskip=c["Dskip"], dt_bias=c["dt_bias"], h0=c["h0"])
    y1, h1 = orc.scan_fwd(as_bits["u"], as_bits["delta"], c["A"], as_bits["B"], as_bits["C"],
                          z=as_bits["z"], dtype="bf16", **common)
    y2, h2 = orc.scan_fwd(as_vals["u"], as_vals["delta"], c["A"], as_vals["B"], as_vals["C"],
                          z=as_vals["z"], **common)
    assert np.array_equal(y1, y2) and np.array_equal(h1, h2), "bf16 scan differs from the decoded scan"
    t = 5
    s1 = orc.scan_step(c["h0"], as_bits["u"][..., t], as_bits["delta"][..., t], c["A"],
                       as_bits["B"][..., t], as_bits["C"][..., t], z_t=as_bits["z"][..., t],
                       Dskip=c["Dskip"], dt_bias=c["dt_bias"], dtype="bf16")
    s2 = orc.scan_step(c["h0"], as_vals["u"][..., t], as_vals["delta"][..., t], c["A"],
                       as_vals["B"][..., t], as_vals["C"][..., t], z_t=as_vals["z"][..., t],
                       Dskip=c["Dskip"], dt_bias=c["dt_bias"])
    assert np.array_equal(s1[0], s2[0]) and np.array_equal(s1[1], s2[1]), "bf16 step differs"


def pin_rows_selection(orc):
    """``rows=`` (how the full-size workloads are sampled) returns exactly the flat rows
    b * dim + d it names, in the order given: unsorted rows spread over three batch
    elements equal the time-grid closed form of those (b, d), and so do their states
    at requested positions."""
    c = _rand_case(33, nb=3, dim=5, L=20, N=3)
    nb, dim, L = c["u"].shape
    rows = np.array([14, 0, 7, 5, 9, 3, 12, 13])
    pos = np.array([[4, -1, L - 1], [L - 1, 7, 0]])       # (npos, batch)
    y, h, hp = _run(orc, c, rows=rows, positions=pos)
    ry, rh, rall = _brute(c, all_states=True)
    _close(y, ry.reshape(nb * dim, L)[rows], 1e-11, "rows= y")
    _close(h, rh.reshape(nb * dim, -1)[rows], 1e-11, "rows= h_last")
    assert hp.shape == (pos.shape[0], rows.size, c["A"].shape[1])
    for i, r in enumerate(rows):
        b, d = divmod(int(r), dim)
        for k in range(pos.shape[0]):
            p = pos[k, b]
            ref = c["h0"][b, d] if p == -1 else rall[b, d, p]
            _close(hp[k, i], ref, 1e-11, f"rows= state at position {p} of row {r}")


# ---- the backward of the scan: reverse-mode gradients against central finite
#      differences of the (pinned) forward -----------------------------------

_GRAD_OF = dict(u="du", delta="ddelta", z="dz", A="dA", B="dB", C="dC", Dskip="dD", dt_bias="dbias",
                h0="dh0")


def _bwd_loss(orc, c, dy, dhl, delta_softplus):
    y, h = _run(orc, c, delta_softplus=delta_softplus)
    return float(np.sum(dy * y) + (0.0 if dhl is None else np.sum(dhl * h)))


def _bwd_grads(orc, c, dy, dhl, delta_softplus):
    return orc.scan_bwd(c["u"], c["delta"], c["A"], c["B"], c["C"], dy, z=c["z"], Dskip=c["Dskip"],
                        dt_bias=c["dt_bias"], h0=c["h0"], dh_last=dhl, delta_softplus=delta_softplus)


def pin_bwd_finite_differences(orc):
    """Every gradient agrees with a central difference of the forward oracle's loss
    sum(dy y) + sum(dh_last h_last) at sampled elements."""
    cases = ((51, {}, True, True), (52, dict(gated=False, h0=False), True, False),
             (53, dict(D=False, bias=False), False, True))
    for seed, kw, sp, with_dhl in cases:
        c = _rand_case(seed, nb=2, dim=3, L=11, N=4, **kw)
        if not sp:                               # keep Delta positive without softplus
            c["delta"] = np.abs(c["delta"]) * 0.2 + 0.01
        rng = np.random.default_rng(seed + 100)
        dy = rng.standard_normal(c["u"].shape)
        dhl = rng.standard_normal((2, 3, 4)) if with_dhl else None
        g = _bwd_grads(orc, c, dy, dhl, sp)
        for name, gname in _GRAD_OF.items():
            if c[name] is None:
                continue
            x = c[name]
            for _ in range(4):
                idx = tuple(int(rng.integers(0, n)) for n in x.shape)
                eps = 1e-6 * max(1.0, abs(x[idx]))
                old = x[idx]
                x[idx] = old + eps
                lp = _bwd_loss(orc, c, dy, dhl, sp)
                x[idx] = old - eps
                lm = _bwd_loss(orc, c, dy, dhl, sp)
                x[idx] = old
                fd = (lp - lm) / (2 * eps)
                an = g[gname][idx]
                assert abs(fd - an) <= 1e-6 * (abs(fd) + 1.0), \
                    f"{gname}{idx} seed {seed}: analytic {an:.9g} vs finite difference {fd:.9g}"


def pin_bwd_geometric(orc):
    """Constant dlt, B, C, x, no gate, h0 = 0, dy = 1: every gradient in closed form.

    With a = e^(dlt A) and b = dlt B x the forward is the geometric series
    h_t = b (1 - a^(t+1)) / (1 - a), and the gradient of the loss with respect to
    h_t is lambda_t = C (1 - a^(L-t)) / (1 - a) (each later output sees h_t
    decayed by a per step).  The derivatives of eq. (2) with the Euler input term
    then read off as sums of products of these closed forms."""
    L, d, x, Ds = 20, 0.3, 0.7, 0.9
    A = np.array([-1.0, -0.5])
    Bn, Cn = np.array([0.5, -1.2]), np.array([1.3, 0.4])
    a, b = np.exp(d * A), d * Bn * x
    t = np.arange(L)[:, None]
    h = b * (1 - a ** (t + 1)) / (1 - a)                    # (L, N): h_t
    h_prev = b * (1 - a ** t) / (1 - a)                     # h_{t-1}, zero at t = 0
    lam = Cn * (1 - a ** (L - t)) / (1 - a)                 # (L, N): lambda_t
    want = dict(
        du=Ds + d * (lam * Bn).sum(axis=1),
        ddelta=(lam * (A * a * h_prev + x * Bn)).sum(axis=1),
        dA=(d * lam * a * h_prev).sum(axis=0),
        dB=(lam * d * x).T, dC=h.T, dD=np.array([L * x]), dh0=a * lam[0])
    g = orc.scan_bwd(np.full((1, 1, L), x), np.full((1, 1, L), d), A[None, :],
                     np.repeat(Bn[None, :, None], L, axis=2), np.repeat(Cn[None, :, None], L, axis=2),
                     np.ones((1, 1, L)), Dskip=np.array([Ds]), h0=np.zeros((1, 1, 2)), delta_softplus=False)
    for k, w in want.items():
        _close(np.asarray(g[k]).ravel(), np.asarray(w).ravel(), 1e-12, f"bwd geometric {k}")


def pin_bwd_linearity(orc):
    """Gradients are linear in the incoming (dy, dh_last)."""
    c = _rand_case(54, nb=2, dim=2, L=9, N=3)
    rng = np.random.default_rng(55)
    d1, d2 = rng.standard_normal(c["u"].shape), rng.standard_normal(c["u"].shape)
    h1, h2 = rng.standard_normal((2, 2, 3)), rng.standard_normal((2, 2, 3))
    g1 = _bwd_grads(orc, c, d1, h1, True)
    g2 = _bwd_grads(orc, c, d2, h2, True)
    g12 = _bwd_grads(orc, c, 2.0 * d1 - d2, 2.0 * h1 - h2, True)
    for k, v in g12.items():
        if v is not None:
            _close(v, 2.0 * g1[k] - g2[k], 1e-12, f"bwd linearity {k}")


# ---- the causal depthwise convolution upstream of the scan (Table 8, "Pre-SSM
#      1D convolution"; Fig. 5, right: Swish after the convolution) -----------

def _conv_case(seed, nb=2, dim=3, L=21, K=4, state=True, bias=True):
    rng = np.random.default_rng(seed)
    return dict(x=rng.standard_normal((nb, dim, L)), w=rng.standard_normal((dim, K)),
                bias=rng.standard_normal(dim) if bias else None,
                state=rng.standard_normal((nb, dim, K - 1)) if state else None)


def _conv_library(c, apply_silu):
    """The same convolution through numpy's 1D convolution over the carried history."""
    x, w = c["x"], c["w"]
    nb, dim, L = x.shape
    K = w.shape[1]
    hist = np.zeros((nb, dim, K - 1)) if c["state"] is None else c["state"]
    xx = np.concatenate([hist, x], axis=2)
    y = np.zeros_like(x)
    for b in range(nb):
        for d in range(dim):
            # np.convolve flips its second argument: taps reversed give sum_i w[i] xx[t + i]
            y[b, d] = np.convolve(xx[b, d], w[d][::-1], mode="valid")
            if c["bias"] is not None:
                y[b, d] += c["bias"][d]
    if apply_silu:
        y = y * expit(y)
    return y, xx[..., xx.shape[2] - (K - 1):]


def pin_conv_library(orc):
    """Oracle convolution == numpy.convolve over [state, x], Swish by scipy's expit."""
    for seed, kw in ((21, {}), (22, dict(state=False, bias=False)), (23, dict(K=2)), (24, dict(K=1)),
                     (25, dict(L=2)), (26, dict(L=1, K=4))):
        c = _conv_case(seed, **kw)
        for act in (True, False):
            y, st = orc.conv1d(c["x"], c["w"], bias=c["bias"], state=c["state"], apply_silu=act)
            ry, rst = _conv_library(c, act)
            _close(y, ry, 1e-13, f"conv seed {seed} silu={act}")
            assert np.array_equal(st, rst), f"conv state seed {seed}: not the last K-1 inputs"


def pin_conv_impulse(orc):
    """A one-hot tap is a pure delay: tap K-1 gives y = x, tap 0 gives y[t] = x[t-(K-1)]."""
    c = _conv_case(27, L=9)
    K = c["w"].shape[1]
    xx = np.concatenate([c["state"], c["x"]], axis=2)
    for tap, ref in ((K - 1, c["x"]), (0, xx[..., : c["x"].shape[2]])):
        w = np.zeros_like(c["w"])
        w[:, tap] = 1.0
        y, _ = orc.conv1d(c["x"], w, state=c["state"], apply_silu=False)
        assert np.array_equal(y, ref), f"one-hot tap {tap} is not a delay of {K - 1 - tap}"


def pin_conv_split_and_step(orc):
    """Resume: conv over [0, L) == conv over [0, k) then [k, L) from its state; and L
    single steps == one call."""
    c = _conv_case(28, L=17)
    y, st = orc.conv1d(c["x"], c["w"], bias=c["bias"], state=c["state"])
    for k in (1, 2, 3, 8, 16):
        y1, s1 = orc.conv1d(c["x"][..., :k], c["w"], bias=c["bias"], state=c["state"])
        y2, s2 = orc.conv1d(c["x"][..., k:], c["w"], bias=c["bias"], state=s1)
        assert np.array_equal(np.concatenate([y1, y2], axis=2), y), f"conv split at {k}"
        assert np.array_equal(s2, st), f"conv state after split at {k}"
    state = c["state"].copy()
    for t in range(c["x"].shape[2]):
        yt, state = orc.conv1d_step(c["x"][..., t], c["w"], state, bias=c["bias"])
        assert np.array_equal(yt, y[..., t]), f"conv step {t}"
    assert np.array_equal(state, st), "conv state after steps"


ALL_PINS = [
    pin_golden_decimal, pin_bruteforce, pin_geometric, pin_B_zero, pin_split, pin_eq4,
    pin_tuple_scan, pin_separability, pin_linearity, pin_step_equals_fwd, pin_limits,
    pin_softplus_extremes, pin_states_at_positions, pin_bf16_decode, pin_rows_selection,
    pin_conv_library, pin_conv_impulse, pin_conv_split_and_step,
    pin_bwd_finite_differences, pin_bwd_geometric, pin_bwd_linearity,
]

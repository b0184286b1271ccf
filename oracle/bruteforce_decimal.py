"""High-precision brute-force materialisation of the scan -- TEST INFRASTRUCTURE ONLY.

An independent second formulation used to write the small golden fixtures
under ``tests/golden/``.  It does not run the recurrence step by step: it
places the inputs on the continuous time grid t_k = sum_{j<=k} Delta[j]
(Section 2, after eq. (2)) and writes every state as the closed-form response
of the diagonal system dh/dt = A h + B x (eq. (1)) under zero-order hold on A
and simplified-Euler on B (Appendix D):

    h_t[n] = exp(A_n (S_t - S_-1)) h0[n]
             + sum_{s <= t} exp(A_n (S_t - S_s)) Delta_s B_s[n] x_s,
    S_t    = sum_{r <= t} Delta_r,
    y_t    = sum_n C_t[n] h_t[n] + D x_t, then times z_t sigmoid(z_t) (Table 8).

All arithmetic uses Python's ``decimal`` module at 50 significant digits, so
its rounding error is far below any fp64 comparison.
"""
from __future__ import annotations

from decimal import Decimal, getcontext

getcontext().prec = 50


def _softplus(v: Decimal) -> Decimal:
    return (Decimal(1) + v.exp()).ln()


def _sigmoid(z: Decimal) -> Decimal:
    return Decimal(1) / (Decimal(1) + (-z).exp())


def scan_row(u, delta_raw, A, B, C, *, dt_bias=0.0, Dskip=0.0, z=None, h0=None,
             delta_softplus=True):
    """One row.  u, delta_raw, z: length-L sequences; A, h0: length N;
    B, C: N sequences of length L.  Floats are converted exactly to Decimal.
    Returns (y as list of Decimal, h_last as list of Decimal)."""
    L, N = len(u), len(A)
    D = lambda v: Decimal(float(v))  # exact: every float is a dyadic rational
    x = [D(v) for v in u]
    dlt = []
    for v in delta_raw:
        w = D(v) + D(dt_bias)
        dlt.append(_softplus(w) if delta_softplus else w)
    S = []
    acc = Decimal(0)
    for d in dlt:
        acc += d
        S.append(acc)
    An = [D(a) for a in A]
    h0n = [D(v) for v in h0] if h0 is not None else [Decimal(0)] * N
    y, h = [], None
    for t in range(L):
        h = []
        for n in range(N):
            v = (An[n] * S[t]).exp() * h0n[n]
            for s in range(t + 1):
                v += (An[n] * (S[t] - S[s])).exp() * dlt[s] * D(B[n][s]) * x[s]
            h.append(v)
        yv = sum(D(C[n][t]) * h[n] for n in range(N)) + D(Dskip) * x[t]
        if z is not None:
            zt = D(z[t])
            yv = yv * zt * _sigmoid(zt)
        y.append(yv)
    return y, (h if h is not None else list(h0n))

"""Writes the golden fixtures in this folder.  Calls only ``oracle/``.

Each fixture is a tiny scan whose inputs are fp32 values (stored exactly as
decimal strings) and whose expected outputs come from the 50-digit brute-force
materialisation in ``oracle/bruteforce_decimal.py`` (the time-grid form of the
selective SSM, MambaByte Section 2 eq. (1)-(2) and Appendix D), not from the
step-by-step recurrence that the C oracle runs.

    python tests/golden/make_golden.py
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle.bruteforce_decimal import scan_row  # noqa: E402


def f32list(a):
    return [repr(float(v)) for v in np.asarray(a, dtype=np.float32).ravel()]


def make_case(name, seed, L, N, *, gated, with_h0, delta_softplus, with_bias, with_D):
    rng = np.random.default_rng(seed)
    u = rng.standard_normal(L).astype(np.float32)
    if delta_softplus:
        delta = rng.standard_normal(L).astype(np.float32)
    else:
        delta = rng.uniform(0.01, 0.5, L).astype(np.float32)
    A = (-rng.uniform(0.2, 3.0, N)).astype(np.float32)
    B = rng.standard_normal((N, L)).astype(np.float32)
    C = rng.standard_normal((N, L)).astype(np.float32)
    z = rng.standard_normal(L).astype(np.float32) if gated else None
    h0 = (0.5 * rng.standard_normal(N)).astype(np.float32) if with_h0 else None
    dt_bias = np.float32(-1.25) if with_bias else np.float32(0.0)
    Dskip = np.float32(0.875) if with_D else np.float32(0.0)
    y, h = scan_row(u, delta, A, B, C, dt_bias=dt_bias, Dskip=Dskip, z=z, h0=h0,
                    delta_softplus=delta_softplus)
    return {
        "name": name,
        "source": "oracle/bruteforce_decimal.py (time-grid closed form, 50 digits)",
        "L": L, "N": N, "delta_softplus": delta_softplus,
        "u": f32list(u), "delta": f32list(delta), "A": f32list(A),
        "B": f32list(B), "C": f32list(C),
        "z": None if z is None else f32list(z),
        "h0": None if h0 is None else f32list(h0),
        "dt_bias": repr(float(dt_bias)), "Dskip": repr(float(Dskip)),
        "y": [str(v) for v in y], "h_last": [str(v) for v in h],
    }


def main():
    cases = [
        make_case("gated_h0_softplus", 11, 12, 3, gated=True, with_h0=True,
                  delta_softplus=True, with_bias=True, with_D=True),
        make_case("plain_no_softplus", 12, 10, 2, gated=False, with_h0=False,
                  delta_softplus=False, with_bias=False, with_D=False),
        make_case("skip_and_gate_no_h0", 13, 9, 4, gated=True, with_h0=False,
                  delta_softplus=True, with_bias=True, with_D=True),
    ]
    out = os.path.join(HERE, "bruteforce_tiny.json")
    with open(out, "w") as f:
        json.dump(cases, f, indent=1)
        f.write("\n")
    print("wrote", out)


if __name__ == "__main__":
    main()

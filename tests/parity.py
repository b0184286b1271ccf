"""Error metrics shared by the oracle pins and the GPU parity tests."""
from __future__ import annotations

import numpy as np

# Parity bar for the HIP path against the fp64 oracle (fp32 arithmetic):
# max relative error 2e-3 on y and 1e-4 on h_last, with the relative error of
# element i measured against |r_i| + rms(r) so that zero crossings of the
# reference do not turn rounding noise into an unbounded ratio.
TOL_Y = 2e-3
TOL_H = 1e-4
# y rounded to bf16 on output: the bar plus one bf16 rounding (2^-8 relative)
TOL_Y_BF16_OUT = TOL_Y + 2.0 ** -8


def rel_err(got, ref) -> float:
    """max_i |g_i - r_i| / (|r_i| + rms(r)); 0 for empty arrays."""
    g = np.asarray(got, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    if g.shape != r.shape:
        raise ValueError(f"shape mismatch {g.shape} vs {r.shape}")
    if r.size == 0:
        return 0.0
    if not np.all(np.isfinite(g)):
        return float("inf")
    rms = float(np.sqrt(np.mean(r * r)))
    den = np.abs(r) + rms
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(g - r) / den))


def max_abs(got, ref) -> float:
    g = np.asarray(got, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    return float(np.max(np.abs(g - r))) if r.size else 0.0

"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check that
at least one pin fails for each: the pins are strong enough to trust the oracle.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

import oracle
import oracle_pins as P

SRC = os.path.join(os.path.dirname(oracle.__file__), "mbscan_oracle.c")

# (name, exact text in the oracle, replacement)
MUTANTS = [
    ("drop_skip", "acc + (Dskip ? Dskip[r] * x : 0.0)", "acc"),
    ("skip_uses_delta", "Dskip[r] * x", "Dskip[r] * dlt"),
    ("exp_sign", "exp(dlt * A[r * N + n])", "exp(-dlt * A[r * N + n])"),
    ("exp_without_delta", "exp(dlt * A[r * N + n])", "exp(A[r * N + n])"),
    ("B_index_prev_t", "Bm[(b * N + n) * L + t]", "Bm[(b * N + n) * L + (t > 0 ? t - 1 : 0)]"),
    ("B_transposed", "Bm[(b * N + n) * L + t]", "Bm[(b * L + t) * N + n]"),
    ("C_transposed", "Cm[(b * N + n) * L + t]", "Cm[(b * L + t) * N + n]"),
    ("B_C_swapped", "const double bbar_x = (dlt * Bm[", "const double bbar_x = (dlt * Cm["),
    ("y_before_update", "h[n] = abar * h[n] + bbar_x;\n            acc += Cm[(b * N + n) * L + t] * h[n];",
     "acc += Cm[(b * N + n) * L + t] * h[n];\n            h[n] = abar * h[n] + bbar_x;"),
    ("zoh_B", "const double bbar_x = (dlt * Bm[(b * N + n) * L + t]) * x;",
     "const double bbar_x = ((abar - 1.0) / A[r * N + n] * Bm[(b * N + n) * L + t]) * x;"),
    ("euler_missing_x", "(dlt * Bm[(b * N + n) * L + t]) * x;", "(dlt * Bm[(b * N + n) * L + t]);"),
    ("euler_missing_delta", "(dlt * Bm[(b * N + n) * L + t]) * x;", "(Bm[(b * N + n) * L + t]) * x;"),
    ("no_bias", "delta[r * L + t] + (dt_bias ? dt_bias[r] : 0.0)", "delta[r * L + t]"),
    ("bias_sign", "delta[r * L + t] + (dt_bias ? dt_bias[r] : 0.0)", "delta[r * L + t] - (dt_bias ? dt_bias[r] : 0.0)"),
    ("softplus_sign", "log1p(exp(-fabs(v)))", "log1p(exp(fabs(v)))"),
    ("softplus_no_max", "fmax(v, 0.0) + log1p", "log1p"),
    ("softplus_naive_log", "fmax(v, 0.0) + log1p(exp(-fabs(v)))", "log(1.0 + exp(v))"),
    ("no_gate", "z ? yv * silu(z[r * L + t]) : yv", "yv"),
    ("gate_sigmoid_only", "return z / (1.0 + exp(-z));", "return 1.0 / (1.0 + exp(-z));"),
    ("gate_wrong_sign", "return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));"),
    ("h0_ignored", "h[n] = h0 ? h0[r * N + n] : 0.0;", "h[n] = 0.0;"),
    ("h0_wrong_row", "h[n] = h0 ? h0[r * N + n] : 0.0;", "h[n] = h0 ? h0[n] : 0.0;"),
    ("batch_ignored", "const int64_t b = bidx[r];", "const int64_t b = 0;"),
    ("A_shared_row0", "exp(dlt * A[r * N + n])", "exp(dlt * A[n])"),
    ("state_reset_each_step", "double acc = 0.0;", "double acc = 0.0; if (t > 0) for (int64_t m = 0; m < N; ++m) h[m] *= 0.5;"),
    ("h_last_stale", "h_last[r * N + n] = h[n];", "h_last[r * N + n] = h0 ? h0[r * N + n] : 0.0;"),
    ("delta_from_prev_t", "double v = delta[r * L + t]", "double v = delta[r * L + (t > 0 ? t - 1 : 0)]"),
    ("C_state_shift", "acc += Cm[(b * N + n) * L + t] * h[n];", "acc += Cm[(b * N + (n + 1) % N) * L + t] * h[n];"),
    ("position_off_by_one", "record_states(t, L, N, h, row_pos, P, row_out);",
     "record_states(t + 1, L, N, h, row_pos, P, row_out);"),
    ("position_initial_dropped", "record_states(-1, L, N, h, row_pos, P, row_out);", ""),
    ("position_invalid_zero", "out[k * N + n] = NAN;", "out[k * N + n] = 0.0;"),
    ("conv_bias_dropped", "double pre = bias ? bias[r] : 0.0;", "double pre = 0.0;"),
    ("conv_taps_reversed", "pre += w[r * K + i] * xv;", "pre += w[r * K + (K - 1 - i)] * xv;"),
    ("conv_state_ignored", "xv = state_in ? state_in[r * H + (H + src)] : 0.0;", "xv = 0.0;"),
    ("conv_state_reversed", "xv = state_in ? state_in[r * H + (H + src)] : 0.0;",
     "xv = state_in ? state_in[r * H + (-1 - src)] : 0.0;"),
    ("conv_state_out_shifted", "state_out[r * H + j] = src >= 0 ? x[r * L + src]",
     "state_out[r * H + j] = src >= 0 ? x[r * L + (src > 0 ? src - 1 : 0)]"),
    ("conv_no_silu", "y[r * L + t] = apply_silu ? silu(pre) : pre;", "y[r * L + t] = pre;"),
    ("conv_silu_always", "y[r * L + t] = apply_silu ? silu(pre) : pre;", "y[r * L + t] = silu(pre);"),
    ("bwd_carry_without_abar", "lam_next[n] = lam * ab;", "lam_next[n] = lam;"),
    ("bwd_dC_uses_previous_state", "dC[(b * N + n) * L + t] += ds * hcur;", "dC[(b * N + n) * L + t] += ds * hprev;"),
    ("bwd_dB_missing_x", "dB[(b * N + n) * L + t] += lam * dl[t] * x;", "dB[(b * N + n) * L + t] += lam * dl[t];"),
    ("bwd_ddelta_missing_Bx", "ddl += lam * (A[r * N + n] * ab * hprev + Bv * x);",
     "ddl += lam * (A[r * N + n] * ab * hprev);"),
    ("bwd_dA_uses_current_state", "dA[r * N + n] += lam * dl[t] * ab * hprev;",
     "dA[r * N + n] += lam * dl[t] * ab * hcur;"),
    ("bwd_dz_sigmoid_only", "sg * (1.0 + zz * (1.0 - sg))", "sg"),
    ("bwd_dh_last_ignored", "lam_next[n] = dh_last ? dh_last[r * N + n] : 0.0;", "lam_next[n] = 0.0;"),
    ("bwd_softplus_grad_dropped", "ddl * sigmoid(v)", "ddl"),
    ("bwd_ds_without_gate", "const double ds = dy[r * L + t] * g;", "const double ds = dy[r * L + t];"),
    ("bwd_du_without_skip", "double dut = ds * (Dskip ? Dskip[r] : 0.0);", "double dut = 0.0;"),
    ("last_state_dropped_from_y", "for (int64_t n = 0; n < N; ++n) {\n            const double abar",
     "for (int64_t n = 0; n < N; ++n) {\n            if (n == N - 1 && N > 1) continue;\n            const double abar"),
]


# Mistakes in the Python side of the oracle (oracle/__init__.py): the bf16 decode
# every bf16 input goes through, and the row selection that samples the full-size
# workloads.  Several leave the whole-tensor path unchanged, so only the pins of
# those two helpers can catch them.
PY_SRC = os.path.join(os.path.dirname(oracle.__file__), "__init__.py")
PY_MUTANTS = [
    ("bf16_shift_15", "astype(np.uint32) << 16", "astype(np.uint32) << 15"),
    ("bf16_not_shifted", "astype(np.uint32) << 16", "astype(np.uint32)"),
    ("bf16_value_cast", "bits.view(np.float32)", "bits.astype(np.float32)"),
    ("bf16_sign_dropped", "np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << 16",
     "(np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) & 0x7FFF) << 16"),
    ("bf16_rounded_to_f32_then_bf16", "return bits.view(np.float32).astype(np.float64)",
     "return (bits & 0xFFFE0000).view(np.float32).astype(np.float64)"),
    ("rows_batch_mod", "bidx = flat // dim", "bidx = flat % nb"),
    ("rows_sorted", "reshape(nb * dim, -1)[flat]", "reshape(nb * dim, -1)[np.sort(flat)]"),
    ("rows_h0_prefix", "reshape(nb * dim, N)[flat]", "reshape(nb * dim, N)[:len(flat)]"),
    ("rows_A_by_position", "Af = to_f64(A)[didx]", "Af = to_f64(A)[np.arange(len(flat)) % A.shape[0]]"),
    ("rows_skip_by_position", "to_f64(Dskip)[didx]", "to_f64(Dskip)[np.arange(len(flat)) % dim]"),
    ("rows_positions_first_batch", "row_pos = np.ascontiguousarray(pos[:, bidx].T)",
     "row_pos = np.ascontiguousarray(pos[:, np.sort(bidx)].T)"),
]


def _run_pins(lib_path, module=oracle):
    orc = module.Oracle(lib_path)
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(orc)
        except AssertionError as e:
            failed.append(f"{pin.__name__}: {e}")
        except (ValueError, FloatingPointError, OverflowError, IndexError, TypeError) as e:
            failed.append(f"{pin.__name__}: raised {type(e).__name__}")
    return failed


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation target for {name} not found: the oracle changed"
    mutated = src.replace(old, new, 1)
    path = tmp_path / f"mut_{name}.c"
    path.write_text(mutated)
    lib = str(tmp_path / f"libmut_{name}.so")
    oracle.build(src=str(path), out=lib)
    failed = _run_pins(lib)
    assert failed, f"no pin caught the planted mistake {name!r}"


@pytest.mark.parametrize("name,old,new", PY_MUTANTS, ids=[m[0] for m in PY_MUTANTS])
def test_pins_catch_python_mutant(tmp_path, name, old, new):
    import importlib.util
    import sys
    src = open(PY_SRC).read()
    assert src.count(old) >= 1, f"mutation target for {name} not found: the oracle changed"
    path = tmp_path / f"oracle_mut_{name}.py"
    path.write_text(src.replace(old, new, 1))
    modname = f"oracle_mut_{name}"
    spec = importlib.util.spec_from_file_location(modname, path)
    mod = importlib.util.module_from_spec(spec)
    sys.modules[modname] = mod
    try:
        spec.loader.exec_module(mod)
        failed = _run_pins(oracle.LIB_PATH, mod)
    finally:
        del sys.modules[modname]
    assert failed, f"no pin caught the planted mistake {name!r}"


def test_unmutated_python_oracle_passes(tmp_path):
    """The mechanism above, with no mutation, leaves every pin green."""
    import importlib.util
    import sys
    path = tmp_path / "oracle_copy.py"
    path.write_text(open(PY_SRC).read())
    spec = importlib.util.spec_from_file_location("oracle_copy", path)
    mod = importlib.util.module_from_spec(spec)
    sys.modules["oracle_copy"] = mod
    try:
        spec.loader.exec_module(mod)
        assert _run_pins(oracle.LIB_PATH, mod) == []
    finally:
        del sys.modules["oracle_copy"]

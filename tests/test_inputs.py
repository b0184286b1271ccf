"""The seeded input generator: determinism, layout, rounding and distributions."""
import numpy as np

from paper_2401_13660_amd.inputs import (WORKLOADS, bf16_bits_to_f32, f32_to_bf16_bits,
                                         make_inputs)


def test_deterministic_and_independent_streams():
    a = make_inputs(2, 8, 33, 16, seed=3)
    b = make_inputs(2, 8, 33, 16, seed=3, gated=False)
    assert a.digest()["u"] == b.digest()["u"]            # z not drawn: u unchanged
    assert np.array_equal(a.B, b.B)
    c = make_inputs(2, 8, 33, 16, seed=4)
    assert not np.array_equal(a.u, c.u)


def test_layouts_and_dtypes():
    w = make_inputs(3, 5, 7, 16, dtype="bf16", with_h0=True)
    assert w.u.shape == (3, 5, 7) and w.u.dtype == np.uint16
    assert w.B.shape == (3, 16, 7) and w.C.shape == (3, 16, 7)
    assert w.A.shape == (5, 16) and w.A.dtype == np.float32
    assert w.h0.shape == (3, 5, 16) and w.h0.dtype == np.float32
    assert np.array_equal(w.A[0], -np.arange(1, 17, dtype=np.float32))
    f = make_inputs(1, 4, 9, 16, dtype="f32")
    assert f.u.dtype == np.float32


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-9, -(1 + 2**-8), 0.0], np.float32)
    got = bf16_bits_to_f32(f32_to_bf16_bits(x))
    assert np.array_equal(got, np.array([1.0, 1.0, 1 + 2**-6, 1.0, -1.0, 0.0], np.float32))


def test_distributions():
    w = make_inputs(1, 512, 512, 16, dtype="f32", seed=0)
    assert abs(w.u.mean()) < 0.02 and abs(w.u.std() - 1) < 0.02
    dt = np.log1p(np.exp(w.dt_bias.astype(np.float64)))     # softplus(dt_bias) = dt
    assert dt.min() >= 1e-3 - 1e-7 and dt.max() <= 0.1 + 1e-7
    assert w.Dskip.min() >= 0.5 and w.Dskip.max() <= 1.5
    r = make_inputs(1, 64, 4, 16, A_kind="random")
    assert np.all(r.A < 0) and len(np.unique(r.A)) > 500


def test_named_workloads():
    assert WORKLOADS["mambabyte972m_L8192"]["dim"] == 3584
    assert WORKLOADS["mambabyte1p6b_L65536"]["seqlen"] == 65536

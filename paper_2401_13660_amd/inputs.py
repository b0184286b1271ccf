"""Seeded synthetic inputs for the selective scan.

This module only draws random numbers and lays them out; it holds none of the
scan's arithmetic.  Both the HIP path (through the tests and the benchmark) and
the fp64 oracle receive the exact same bits from it.

Recipe (the layer shapes of MambaByte's Table 9 at the 8,192-byte training
context of Section 4; the paper trains on PG19 and other corpora, which these
tensors stand in for -- the scan's cost does not depend on the data):

* u, z, Delta_raw ~ N(0, 1), shape (batch, dim, seqlen), time contiguous;
* B, C ~ N(0, 1), shape (batch, dstate, seqlen), time contiguous (shared by all
  channels of a batch element, Section 2 after eq. (3));
* A[d, n] = -(n + 1) for every channel (S4D-real initialisation,
  A = -exp(log(1..N))), or, with ``A_kind="random"``, an unstructured negative
  matrix A = -exp(N(0, 1)) so that no test can lean on the integer pattern;
* dt_bias = log(expm1(dt)) with dt ~ U[1e-3, 0.1] (the inverse of softplus, so
  that softplus(dt_bias) = dt), Dskip ~ U[0.5, 1.5], h0 ~ N(0, 0.1^2);
* activations (u, Delta_raw, z, B, C) are bf16 (round-to-nearest-even from the
  fp32 draw) for ``dtype="bf16"``, fp32 for ``dtype="f32"``; A, Dskip, dt_bias
  and h0 are always fp32.

Every tensor draws from its own child stream of ``SeedSequence(seed)`` (in the
order u, Delta_raw, z, B, C, dt, Dskip, h0, A), in fixed chunks, so a tensor's
values do not depend on which other tensors are requested.

The causal convolution upstream of the scan (``make_conv_inputs``) gets its own
streams: x ~ N(0, 1) (bf16 or fp32, shape (batch, dim, seqlen)); taps and bias
~ U[-1/sqrt(k), 1/sqrt(k)] (the default initialisation of a depthwise Conv1d
with fan-in k; k = 4 as in Table 9); a carried state of k - 1 earlier inputs,
drawn like x (bf16-exact values) and held as fp32.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

_CHUNK = 1 << 24

# Stream indices of the child generators; fixed forever so that seeds are stable.
_STREAMS = ("u", "delta", "z", "B", "C", "dt", "Dskip", "h0", "A",
            "conv_x", "conv_w", "conv_bias", "conv_state")


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    rounded = (bits + 0x7FFF + ((bits >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def _rng(seed: int, name: str) -> np.random.Generator:
    child = np.random.SeedSequence(seed).spawn(len(_STREAMS))[_STREAMS.index(name)]
    return np.random.Generator(np.random.PCG64(child))


def _normal_f32(rng: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        out[s:e] = rng.standard_normal(e - s, dtype=np.float32)
    if scale != 1.0:
        out *= np.float32(scale)
    return out.reshape(shape)


def _activation(rng, shape, dtype: str) -> np.ndarray:
    x = _normal_f32(rng, shape)
    if dtype == "bf16":
        return f32_to_bf16_bits(x).reshape(shape)
    return x


@dataclass
class ScanInputs:
    """One seeded workload.  bf16 tensors are uint16 bit patterns."""

    batch: int
    dim: int
    seqlen: int
    dstate: int
    dtype: str                      # "bf16" or "f32" for u, delta, z, B, C
    u: np.ndarray
    delta: np.ndarray
    A: np.ndarray
    B: np.ndarray
    C: np.ndarray
    Dskip: np.ndarray | None
    dt_bias: np.ndarray | None
    z: np.ndarray | None
    h0: np.ndarray | None
    meta: dict = field(default_factory=dict)

    def arrays(self) -> dict:
        names = ("u", "delta", "A", "B", "C", "Dskip", "dt_bias", "z", "h0")
        return {k: getattr(self, k) for k in names if getattr(self, k) is not None}

    def digest(self) -> dict:
        """SHA-256 of every tensor's bytes (documents exactly what was run)."""
        return {k: hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest()[:16]
                for k, v in self.arrays().items()}


def make_inputs(batch: int, dim: int, seqlen: int, dstate: int = 16, *,
                dtype: str = "bf16", seed: int = 0, gated: bool = True,
                with_h0: bool = False, with_D: bool = True, with_bias: bool = True,
                A_kind: str = "s4d") -> ScanInputs:
    """Draw one workload following the recipe in the module docstring."""
    if dtype not in ("bf16", "f32"):
        raise ValueError(f"dtype must be 'bf16' or 'f32', got {dtype!r}")
    if min(batch, dim, dstate) < 1 or seqlen < 0:
        raise ValueError("batch, dim, dstate must be >= 1 and seqlen >= 0")
    act = (batch, dim, seqlen)
    u = _activation(_rng(seed, "u"), act, dtype)
    delta = _activation(_rng(seed, "delta"), act, dtype)
    z = _activation(_rng(seed, "z"), act, dtype) if gated else None
    Bm = _activation(_rng(seed, "B"), (batch, dstate, seqlen), dtype)
    Cm = _activation(_rng(seed, "C"), (batch, dstate, seqlen), dtype)
    dt = _rng(seed, "dt").uniform(1e-3, 0.1, size=dim)
    dt_bias = np.log(np.expm1(dt)).astype(np.float32) if with_bias else None
    Dskip = _rng(seed, "Dskip").uniform(0.5, 1.5, size=dim).astype(np.float32) if with_D else None
    h0 = _normal_f32(_rng(seed, "h0"), (batch, dim, dstate), scale=0.1) if with_h0 else None
    if A_kind == "s4d":
        A = np.broadcast_to(-np.arange(1, dstate + 1, dtype=np.float32), (dim, dstate)).copy()
    elif A_kind == "random":
        A = (-np.exp(_rng(seed, "A").standard_normal((dim, dstate)))).astype(np.float32)
    else:
        raise ValueError(f"unknown A_kind {A_kind!r}")
    return ScanInputs(batch, dim, seqlen, dstate, dtype, u, delta, A, Bm, Cm,
                      Dskip, dt_bias, z, h0,
                      meta=dict(seed=seed, gated=gated, with_h0=with_h0, A_kind=A_kind))


# The workloads, by name.  Shapes: MambaByte Table 9 with expansion e = 2
# (dim = e * d), n_state = 16, the 8,192-byte training context (Section 4),
# 8x that context for length extrapolation (Fig. 3), and a speculative-verify
# chunk of 16 drafted bytes (three subwords per draft at about four bytes per
# subword, Table 6 and Table 10) over a batch of 32 prompts.
WORKLOADS = {
    "tiny_f32": dict(batch=1, dim=64, seqlen=256, dstate=16, dtype="f32"),
    "mambabyte353m_L8192": dict(batch=4, dim=2048, seqlen=8192, dstate=16, dtype="bf16"),
    "mambabyte972m_L8192": dict(batch=4, dim=3584, seqlen=8192, dstate=16, dtype="bf16"),
    "mambabyte1p6b_L65536": dict(batch=1, dim=4608, seqlen=65536, dstate=16, dtype="bf16"),
    "verify_b32_L16": dict(batch=32, dim=3584, seqlen=16, dstate=16, dtype="bf16", with_h0=True),
}


def workload(name: str, seed: int = 0, **overrides) -> ScanInputs:
    cfg = dict(WORKLOADS[name])
    cfg.update(overrides)
    return make_inputs(**cfg, seed=seed)


@dataclass
class ConvInputs:
    """One seeded convolution workload.  bf16 tensors are uint16 bit patterns."""

    batch: int
    dim: int
    seqlen: int
    width: int
    dtype: str                      # "bf16" or "f32" for x
    x: np.ndarray
    w: np.ndarray
    bias: np.ndarray | None
    state: np.ndarray | None
    meta: dict = field(default_factory=dict)

    def arrays(self) -> dict:
        names = ("x", "w", "bias", "state")
        return {k: getattr(self, k) for k in names if getattr(self, k) is not None}


def make_conv_inputs(batch: int, dim: int, seqlen: int, width: int = 4, *, dtype: str = "bf16",
                     seed: int = 0, with_bias: bool = True, with_state: bool = False) -> ConvInputs:
    """Draw one convolution workload following the recipe in the module docstring."""
    if dtype not in ("bf16", "f32"):
        raise ValueError(f"dtype must be 'bf16' or 'f32', got {dtype!r}")
    if min(batch, dim, width) < 1 or seqlen < 0:
        raise ValueError("batch, dim, width must be >= 1 and seqlen >= 0")
    x = _activation(_rng(seed, "conv_x"), (batch, dim, seqlen), dtype)
    bound = 1.0 / np.sqrt(width)
    w = _rng(seed, "conv_w").uniform(-bound, bound, size=(dim, width)).astype(np.float32)
    bias = _rng(seed, "conv_bias").uniform(-bound, bound, size=dim).astype(np.float32) if with_bias else None
    state = None
    if with_state:
        st = _normal_f32(_rng(seed, "conv_state"), (batch, dim, width - 1))
        state = bf16_bits_to_f32(f32_to_bf16_bits(st)).reshape(st.shape) if dtype == "bf16" else st
    return ConvInputs(batch, dim, seqlen, width, dtype, x, w, bias, state,
                      meta=dict(seed=seed, with_state=with_state))


def conv_workload(name: str, seed: int = 0, width: int = 4, **overrides) -> ConvInputs:
    """The convolution in front of the scan of a named workload (same batch, dim, L, dtype)."""
    cfg = dict(WORKLOADS[name])
    conv = dict(batch=cfg["batch"], dim=cfg["dim"], seqlen=cfg["seqlen"], dtype=cfg["dtype"],
                with_state=bool(cfg.get("with_h0", False)))
    conv.update(overrides)
    return make_conv_inputs(**conv, width=width, seed=seed)

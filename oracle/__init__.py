"""The fp64 CPU oracle of the selective scan -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never calls it, and it never calls the product path.

The arithmetic lives in ``mbscan_oracle.c`` (plain C, IEEE double, built by
gcc without fast-math).  This wrapper only decodes the input formats (bf16 bit
patterns and fp32 widen exactly to fp64), arranges rows and hands pointers to
the C code.  See the C file for what is computed and which passage of the paper
each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mbscan_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.POINTER(ctypes.c_int64)


def build(src: str = _SRC, out: str = LIB_PATH, extra_flags=()) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           *extra_flags, "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def to_f64(x, dtype: str | None = None) -> np.ndarray:
    """Exact widening to fp64.  ``dtype="bf16"`` means x holds bf16 bit patterns."""
    x = np.asarray(x)
    if dtype == "bf16" or x.dtype == np.uint16:
        bits = np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_D)


class Oracle:
    """ctypes handle on a built oracle library (the default one, or a test build)."""

    def __init__(self, lib_path: str = LIB_PATH):
        if not os.path.exists(lib_path):
            build(out=lib_path)
        self.lib = ctypes.CDLL(lib_path)
        self.lib.mbo_scan_rows.restype = ctypes.c_int
        self.lib.mbo_scan_rows.argtypes = [
            ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
            _D, _D, _D, _D, _D, _D, _D, _I64, ctypes.c_int64, _D, _D, _D, _D]
        self.lib.mbo_scan_rows_states.restype = ctypes.c_int
        self.lib.mbo_scan_rows_states.argtypes = [
            ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
            _D, _D, _D, _D, _D, _D, _D, _I64, ctypes.c_int64, _D, _D, _D, _D,
            _I64, ctypes.c_int64, _D]
        self.lib.mbo_scan_bwd_rows.restype = ctypes.c_int
        self.lib.mbo_scan_bwd_rows.argtypes = [
            ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
            _D, _D, _D, _D, _D, _D, _D, _I64, ctypes.c_int64, _D, _D, _D, _D,
            _D, _D, _D, _D, _D, _D, _D, _D, _D]
        self.lib.mbo_conv1d_rows.restype = ctypes.c_int
        self.lib.mbo_conv1d_rows.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                             _D, _D, _D, _D, _D, _D]
        self.lib.mbo_conv1d_step.restype = ctypes.c_int
        self.lib.mbo_conv1d_step.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                             _D, _D, _D, _D, _D]
        self.lib.mbo_max_threads.restype = ctypes.c_int
        self.lib.mbo_set_threads.restype = None
        self.lib.mbo_set_threads.argtypes = [ctypes.c_int]
        self.lib.mbo_scan_step.restype = ctypes.c_int
        self.lib.mbo_scan_step.argtypes = [
            ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
            _D, _D, _D, _D, _D, _D, _I64, ctypes.c_int64, _D, _D, _D, _D]

    def max_threads(self) -> int:
        return int(self.lib.mbo_max_threads())

    def set_threads(self, n: int) -> None:
        """Threads of later calls (for timing the oracle on fewer cores)."""
        self.lib.mbo_set_threads(int(n))

    # -- rows ---------------------------------------------------------------
    def scan_rows(self, u, delta, A, Bm, Cm, bidx, *, z=None, Dskip=None, dt_bias=None,
                  h0=None, delta_softplus=True, want_h_last=True, positions=None):
        """Scan R independent rows.

        u, delta, z: (R, L); A, h0: (R, N); Dskip, dt_bias: (R,);
        Bm, Cm: (nbatch, N, L); bidx: (R,) batch index of each row.
        All float arguments must already be fp64.  Returns (y (R, L), h_last (R, N) or None),
        and with ``positions`` (R, P) integers also h_pos (R, P, N): the state after
        each requested timestep (-1: the initial state; outside [-1, L-1]: NaN).
        """
        u = np.ascontiguousarray(u, dtype=np.float64)
        R, L = u.shape
        Bm = np.ascontiguousarray(Bm, dtype=np.float64)
        nb, N, Lb = Bm.shape
        if Lb != L:
            raise ValueError("B/C length does not match u")
        args = dict(delta=delta, z=z, A=A, Dskip=Dskip, dt_bias=dt_bias, h0=h0, Cm=Cm)
        a = {k: (None if v is None else np.ascontiguousarray(v, dtype=np.float64))
             for k, v in args.items()}
        bidx = np.ascontiguousarray(bidx, dtype=np.int64)
        y = np.empty((R, L), dtype=np.float64)
        h_last = np.empty((R, N), dtype=np.float64) if want_h_last else None
        if positions is None:
            rc = self.lib.mbo_scan_rows(R, L, N, int(bool(delta_softplus)),
                                        _ptr(u), _ptr(a["delta"]), _ptr(a["z"]), _ptr(a["A"]),
                                        _ptr(a["Dskip"]), _ptr(a["dt_bias"]), _ptr(a["h0"]),
                                        bidx.ctypes.data_as(_I64), nb, _ptr(Bm), _ptr(a["Cm"]),
                                        _ptr(y), _ptr(h_last))
            if rc != 0:
                raise ValueError(f"oracle rejected the arguments (status {rc})")
            return y, h_last
        pos = np.ascontiguousarray(positions, dtype=np.int64).reshape(R, -1)
        P = pos.shape[1]
        h_pos = np.empty((R, P, N), dtype=np.float64)
        rc = self.lib.mbo_scan_rows_states(R, L, N, int(bool(delta_softplus)),
                                           _ptr(u), _ptr(a["delta"]), _ptr(a["z"]), _ptr(a["A"]),
                                           _ptr(a["Dskip"]), _ptr(a["dt_bias"]), _ptr(a["h0"]),
                                           bidx.ctypes.data_as(_I64), nb, _ptr(Bm), _ptr(a["Cm"]),
                                           _ptr(y), _ptr(h_last), pos.ctypes.data_as(_I64), P,
                                           _ptr(h_pos))
        if rc != 0:
            raise ValueError(f"oracle rejected the arguments (status {rc})")
        return y, h_last, h_pos

    # -- whole tensors --------------------------------------------------------
    def scan_fwd(self, u, delta, A, Bm, Cm, *, z=None, Dskip=None, dt_bias=None, h0=None,
                 delta_softplus=True, dtype: str | None = None, rows=None, positions=None):
        """Scan (batch, dim, L) tensors; ``rows`` optionally picks flat (b*dim + d) rows.

        Activations may be bf16 bit patterns (``dtype="bf16"``) or floats.
        Returns y of shape (batch, dim, L) -- or (len(rows), L) -- and h_last
        of shape (batch, dim, N) -- or (len(rows), N) -- in fp64.  With
        ``positions`` of shape (npos, batch) (position k of batch element b) it
        also returns the states there, (npos, batch, dim, N) -- or (npos, len(rows), N).
        """
        u = np.asarray(u)
        nb, dim, L = u.shape
        N = np.asarray(A).shape[1]
        flat = np.arange(nb * dim) if rows is None else np.asarray(rows, dtype=np.int64)
        bidx = flat // dim
        didx = flat % dim

        def act(x):
            return None if x is None else to_f64(np.asarray(x).reshape(nb * dim, -1)[flat], dtype)

        Af = to_f64(A)[didx]
        row_pos = None
        if positions is not None:
            pos = np.asarray(positions, dtype=np.int64).reshape(-1, nb)
            row_pos = np.ascontiguousarray(pos[:, bidx].T)                 # (rows, npos)
        out = self.scan_rows(
            act(u), act(delta), Af, to_f64(Bm, dtype), to_f64(Cm, dtype), bidx,
            z=act(z),
            Dskip=None if Dskip is None else to_f64(Dskip)[didx],
            dt_bias=None if dt_bias is None else to_f64(dt_bias)[didx],
            h0=None if h0 is None else to_f64(h0).reshape(nb * dim, N)[flat],
            delta_softplus=delta_softplus, positions=row_pos)
        y, h_last = out[0], out[1]
        if rows is None:
            y, h_last = y.reshape(nb, dim, L), h_last.reshape(nb, dim, N)
        if positions is None:
            return y, h_last
        h_pos = np.moveaxis(out[2], 1, 0)                                  # (npos, rows, N)
        if rows is None:
            h_pos = h_pos.reshape(-1, nb, dim, N)
        return y, h_last, h_pos

    def scan_step(self, h, u_t, delta_t, A, B_t, C_t, *, z_t=None, Dskip=None, dt_bias=None,
                  delta_softplus=True, dtype: str | None = None):
        """One step for (batch, dim) inputs; returns (y_t (batch, dim), new h (batch, dim, N))."""
        h_new = np.array(to_f64(h), dtype=np.float64, copy=True)
        nb, dim, N = h_new.shape
        R = nb * dim
        bidx = np.repeat(np.arange(nb, dtype=np.int64), dim)
        didx = np.tile(np.arange(dim), nb)

        def flat(x):
            return None if x is None else to_f64(x, dtype).reshape(R)

        y = np.empty(R, dtype=np.float64)
        Af = np.ascontiguousarray(to_f64(A)[didx])
        Ds = None if Dskip is None else np.ascontiguousarray(to_f64(Dskip)[didx])
        db = None if dt_bias is None else np.ascontiguousarray(to_f64(dt_bias)[didx])
        hv = h_new.reshape(R, N)
        ut, dtt, zt = flat(u_t), flat(delta_t), flat(z_t)
        Bt = np.ascontiguousarray(to_f64(B_t, dtype).reshape(nb, N))
        Ct = np.ascontiguousarray(to_f64(C_t, dtype).reshape(nb, N))
        rc = self.lib.mbo_scan_step(R, N, int(bool(delta_softplus)), _ptr(ut), _ptr(dtt), _ptr(zt),
                                    _ptr(Af), _ptr(Ds), _ptr(db), bidx.ctypes.data_as(_I64), nb,
                                    _ptr(Bt), _ptr(Ct), _ptr(hv), _ptr(y))
        if rc != 0:
            raise ValueError(f"oracle rejected the arguments (status {rc})")
        return y.reshape(nb, dim), h_new


    # -- the backward of the scan -------------------------------------------------
    def scan_bwd(self, u, delta, A, Bm, Cm, dy, *, z=None, Dskip=None, dt_bias=None, h0=None,
                 dh_last=None, delta_softplus=True, dtype: str | None = None):
        """Gradients of sum(dy * y) + sum(dh_last * h_last) for (batch, dim, L) inputs.

        Activations may be bf16 bit patterns (``dtype="bf16"``); dy is decoded by its own
        type (uint16 arrays are bf16 bit patterns).  Returns a dict of fp64
        arrays: du, ddelta, dz (batch, dim, L); dA (dim, N); dB, dC (batch, N, L);
        dD, dbias (dim,); dh0 (batch, dim, N).  Absent inputs get no gradient (None).
        """
        u = np.asarray(u)
        nb, dim, L = u.shape
        N = np.asarray(A).shape[1]
        R = nb * dim
        bidx = np.repeat(np.arange(nb, dtype=np.int64), dim)
        didx = np.tile(np.arange(dim), nb)

        def act(x):
            return None if x is None else np.ascontiguousarray(to_f64(x, dtype).reshape(R, L))

        def flat(x, width):
            return None if x is None else np.ascontiguousarray(to_f64(x).reshape(R, width))

        Af = np.ascontiguousarray(to_f64(A)[didx])
        Ds = None if Dskip is None else np.ascontiguousarray(to_f64(Dskip)[didx])
        db = None if dt_bias is None else np.ascontiguousarray(to_f64(dt_bias)[didx])
        Bf = np.ascontiguousarray(to_f64(Bm, dtype))
        Cf = np.ascontiguousarray(to_f64(Cm, dtype))
        zf = act(z)
        out = {k: np.empty((R, L)) for k in ("du", "ddelta")}
        out["dz"] = np.empty((R, L)) if z is not None else None
        dA = np.empty((R, N))
        dD = np.empty(R)
        dbias = np.empty(R)
        dh0 = np.empty((R, N))
        dB = np.empty((nb, N, L))
        dC = np.empty((nb, N, L))
        rc = self.lib.mbo_scan_bwd_rows(
            R, L, N, int(bool(delta_softplus)), _ptr(act(u)), _ptr(act(delta)), _ptr(zf), _ptr(Af),
            _ptr(Ds), _ptr(db), _ptr(flat(h0, N)), bidx.ctypes.data_as(_I64), nb, _ptr(Bf), _ptr(Cf),
            _ptr(np.ascontiguousarray(to_f64(dy).reshape(R, L))), _ptr(flat(dh_last, N)), _ptr(out["du"]), _ptr(out["ddelta"]), _ptr(out["dz"]),
            _ptr(dA), _ptr(dD), _ptr(dbias), _ptr(dh0), _ptr(dB), _ptr(dC))
        if rc != 0:
            raise ValueError(f"oracle rejected the arguments (status {rc})")
        g = {k: (None if v is None else v.reshape(nb, dim, L)) for k, v in out.items()}
        g["dA"] = dA.reshape(nb, dim, N).sum(axis=0)
        g["dD"] = dD.reshape(nb, dim).sum(axis=0) if Dskip is not None else None
        g["dbias"] = dbias.reshape(nb, dim).sum(axis=0) if dt_bias is not None else None
        g["dh0"] = dh0.reshape(nb, dim, N)
        g["dB"], g["dC"] = dB, dC
        return g

    # -- the causal depthwise convolution ---------------------------------------
    def conv1d(self, x, w, *, bias=None, state=None, apply_silu=True, dtype: str | None = None):
        """Causal depthwise convolution of (batch, dim, L) inputs with taps w (dim, K).

        ``state`` (batch, dim, K-1) holds the K-1 inputs before x, oldest first (zeros
        when absent).  Returns y (batch, dim, L) and the new state (batch, dim, K-1),
        both fp64.  ``dtype="bf16"`` means x holds bf16 bit patterns.
        """
        x = np.asarray(x)
        nb, dim, L = x.shape
        w64 = to_f64(w)
        K = w64.shape[1]
        R = nb * dim
        xf = np.ascontiguousarray(to_f64(x, dtype).reshape(R, L))
        wf = np.ascontiguousarray(np.tile(w64, (nb, 1)))
        bf = None if bias is None else np.ascontiguousarray(np.tile(to_f64(bias), nb))
        sf = None if state is None else np.ascontiguousarray(to_f64(state).reshape(R, K - 1))
        y = np.empty((R, L), dtype=np.float64)
        st = np.empty((R, max(K - 1, 0)), dtype=np.float64)
        rc = self.lib.mbo_conv1d_rows(R, L, K, int(bool(apply_silu)), _ptr(xf), _ptr(wf), _ptr(bf),
                                      _ptr(sf), _ptr(y), _ptr(st) if K > 1 else None)
        if rc != 0:
            raise ValueError(f"oracle rejected the arguments (status {rc})")
        return y.reshape(nb, dim, L), st.reshape(nb, dim, K - 1)

    def conv1d_step(self, x_t, w, state, *, bias=None, apply_silu=True, dtype: str | None = None):
        """One step for (batch, dim) inputs; returns (y_t (batch, dim), new state (batch, dim, K-1))."""
        x_t = np.asarray(x_t)
        nb, dim = x_t.shape
        w64 = to_f64(w)
        K = w64.shape[1]
        R = nb * dim
        xf = np.ascontiguousarray(to_f64(x_t, dtype).reshape(R))
        wf = np.ascontiguousarray(np.tile(w64, (nb, 1)))
        bf = None if bias is None else np.ascontiguousarray(np.tile(to_f64(bias), nb))
        st = np.array(to_f64(state), dtype=np.float64, copy=True).reshape(R, K - 1)
        y = np.empty(R, dtype=np.float64)
        rc = self.lib.mbo_conv1d_step(R, K, int(bool(apply_silu)), _ptr(xf), _ptr(wf), _ptr(bf),
                                      _ptr(st) if K > 1 else None, _ptr(y))
        if rc != 0:
            raise ValueError(f"oracle rejected the arguments (status {rc})")
        return y.reshape(nb, dim), st.reshape(nb, dim, K - 1)


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def scan_inputs(inp, rows=None, delta_softplus=True, positions=None):
    """Run the oracle on a ``ScanInputs`` workload (any object with the same fields)."""
    return default().scan_fwd(inp.u, inp.delta, inp.A, inp.B, inp.C, z=inp.z, Dskip=inp.Dskip,
                              dt_bias=inp.dt_bias, h0=inp.h0, delta_softplus=delta_softplus,
                              dtype=inp.dtype, rows=rows, positions=positions)

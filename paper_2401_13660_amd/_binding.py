"""Python binding of libmbscan.so: argument marshalling only.

Every step of the scan runs in the HIP kernels behind the C ABI declared in
``include/mbscan.h``; this module checks torch tensors, allocates outputs with
torch (device memory and streams are all PyTorch is used for) and passes raw
device pointers plus the current HIP stream.  There is no fallback: without the
built library every call raises ``MBScanError``.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmbscan.so")

MB_F32, MB_BF16 = 0, 1
_STATUS_OK = 0


class MBScanError(RuntimeError):
    pass


class ScanDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("dim", ctypes.c_int64), ("seqlen", ctypes.c_int64),
                ("dstate", ctypes.c_int64), ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("delta_softplus", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class ConvDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("dim", ctypes.c_int64), ("seqlen", ctypes.c_int64),
                ("width", ctypes.c_int32), ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("apply_silu", ctypes.c_int32), ("reserved", ctypes.c_int32), ("reserved2", ctypes.c_int32)]


_lib = None
_VP = ctypes.c_void_p


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load (once) and return the HIP library; raise loudly if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise MBScanError(f"{path} is not built; run `python -m paper_2401_13660_amd.build` "
                          "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(path)
    lib.mb_scan_fwd.restype = ctypes.c_int
    lib.mb_scan_fwd.argtypes = [ctypes.POINTER(ScanDesc)] + [_VP] * 12
    lib.mb_scan_fwd_noalloc.restype = ctypes.c_int
    lib.mb_scan_fwd_noalloc.argtypes = [ctypes.POINTER(ScanDesc)] + [_VP] * 12
    lib.mb_scan_fwd_states.restype = ctypes.c_int
    lib.mb_scan_fwd_states.argtypes = [ctypes.POINTER(ScanDesc)] + [_VP] * 11 + [_VP, ctypes.c_int64, _VP, _VP]
    lib.mb_scan_step.restype = ctypes.c_int
    lib.mb_scan_step.argtypes = [ctypes.c_int64] * 3 + [ctypes.c_int32] * 3 + [_VP] * 11
    lib.mb_conv1d_fwd.restype = ctypes.c_int
    lib.mb_conv1d_fwd.argtypes = [ctypes.POINTER(ConvDesc)] + [_VP] * 7
    lib.mb_conv1d_step.restype = ctypes.c_int
    lib.mb_conv1d_step.argtypes = [ctypes.c_int64] * 2 + [ctypes.c_int32] * 4 + [_VP] * 6
    lib.mb_scan_bwd.restype = ctypes.c_int
    lib.mb_scan_bwd.argtypes = [ctypes.POINTER(ScanDesc)] + [_VP] * 22
    lib.mb_scan_fwd_ckpt.restype = ctypes.c_int
    lib.mb_scan_fwd_ckpt.argtypes = [ctypes.POINTER(ScanDesc)] + [_VP] * 13
    lib.mb_verify_rank.restype = ctypes.c_int
    lib.mb_verify_rank.argtypes = [ctypes.c_int64] * 3 + [ctypes.c_int32] * 2 + [_VP] * 6
    lib.mb_status_string.restype = ctypes.c_char_p
    lib.mb_status_string.argtypes = [ctypes.c_int]
    lib.mb_abi_version.restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status: int, what: str):
    if status != _STATUS_OK:
        msg = load_library().mb_status_string(status).decode()
        raise MBScanError(f"{what} failed with status {status}: {msg}")


def _dt(t: torch.dtype) -> int:
    if t == torch.float32:
        return MB_F32
    if t == torch.bfloat16:
        return MB_BF16
    raise MBScanError(f"unsupported element type {t}; use float32 or bfloat16")


def _ptr(t):
    return None if t is None else t.data_ptr()


# Per-call host work bounds a decode step called from Python (the kernel of a
# one-byte step takes a few microseconds), so the stream and device lookups use
# torch's raw accessors where it has them, and a well-formed argument passes its
# checks in one expression.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(dev):
    """The raw HIP stream torch currently uses on device ``dev``."""
    if _raw_stream is not None and dev.index is not None:
        return _raw_stream(dev.index)
    return torch.cuda.current_stream(dev).cuda_stream


def _on_device(dev):
    """A context making ``dev`` current for the call; nothing if it already is."""
    cur = _cur_device() if _cur_device is not None else torch.cuda.current_device()
    return contextlib.nullcontext() if dev.index == cur else torch.cuda.device(dev)


def _need(t, name, shape, dtype=None, device=None):
    if (isinstance(t, torch.Tensor) and t.is_cuda and t.shape == shape and (dtype is None or t.dtype == dtype)
            and (device is None or t.device == device) and t.is_contiguous()):
        return
    if not isinstance(t, torch.Tensor):
        raise MBScanError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise MBScanError(f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise MBScanError(f"{name} is on {t.device}, expected {device}")
    if tuple(t.shape) != tuple(shape):
        raise MBScanError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise MBScanError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise MBScanError(f"{name} must be contiguous")


def scan_fwd(u, delta, A, B, C, D=None, dt_bias=None, z=None, h0=None, *, delta_softplus=True,
             out_dtype=torch.float32, return_last_state=False, out=None, h_last=None,
             positions=None, h_at=None, return_ckpt=False, ck=None):
    """Selective scan over (batch, dim, L) inputs; returns y or (y, h_last).

    u, delta, z: (batch, dim, L); B, C: (batch, N, L), all of one dtype (fp32 or bf16);
    A: (dim, N) fp32; D, dt_bias: (dim,) fp32; h0: (batch, dim, N) fp32.

    ``positions``: int32 (npos, batch) on the GPU; position k of batch element b is a
    timestep in [0, L) or -1 (the initial state).  The states there are returned as a
    last extra element ``h_at`` of shape (npos, batch, dim, N) (NaN for a position
    outside [-1, L-1]); ``h_at[k]`` can be passed back as ``h0`` to resume.

    ``return_ckpt`` (or a given ``ck``): also store the backward's checkpoints, the
    state before every 16th timestep, as a last extra element of shape
    (L // 16, batch, dim, N) (mb_scan_fwd_ckpt; not combined with positions).
    """
    lib = load_library()
    if not isinstance(u, torch.Tensor) or u.dim() != 3:
        raise MBScanError("u must be a (batch, dim, L) tensor")
    nb, dim, L = u.shape
    if not isinstance(A, torch.Tensor) or A.dim() != 2:
        raise MBScanError("A must be a (dim, N) tensor")
    N = A.shape[1]
    dev, act = u.device, u.dtype
    _need(u, "u", (nb, dim, L), act, dev)
    _need(delta, "delta", (nb, dim, L), act, dev)
    _need(A, "A", (dim, N), torch.float32, dev)
    _need(B, "B", (nb, N, L), act, dev)
    _need(C, "C", (nb, N, L), act, dev)
    if z is not None:
        _need(z, "z", (nb, dim, L), act, dev)
    if D is not None:
        _need(D, "D", (dim,), torch.float32, dev)
    if dt_bias is not None:
        _need(dt_bias, "dt_bias", (dim,), torch.float32, dev)
    if h0 is not None:
        _need(h0, "h0", (nb, dim, N), torch.float32, dev)
    if out is None:
        out = torch.empty((nb, dim, L), dtype=out_dtype, device=dev)
    else:
        _need(out, "out", (nb, dim, L), None, dev)
    if return_last_state and h_last is None:
        h_last = torch.empty((nb, dim, N), dtype=torch.float32, device=dev)
    elif h_last is not None:
        _need(h_last, "h_last", (nb, dim, N), torch.float32, dev)
    npos = 0
    if positions is not None:
        if not isinstance(positions, torch.Tensor) or positions.dim() != 2:
            raise MBScanError("positions must be an int32 (npos, batch) tensor")
        npos = positions.shape[0]
        _need(positions, "positions", (npos, nb), torch.int32, dev)
        if h_at is None:
            h_at = torch.empty((npos, nb, dim, N), dtype=torch.float32, device=dev)
        else:
            _need(h_at, "h_at", (npos, nb, dim, N), torch.float32, dev)
    elif h_at is not None:
        raise MBScanError("h_at given without positions")
    want_ck = return_ckpt or ck is not None
    if want_ck:
        if positions is not None:
            raise MBScanError("checkpoints and positions are not recorded by the same call")
        if ck is None:
            ck = torch.empty((L // 16, nb, dim, N), dtype=torch.float32, device=dev)
        else:
            _need(ck, "ck", (L // 16, nb, dim, N), torch.float32, dev)
    desc = ScanDesc(nb, dim, L, N, _dt(act), _dt(out.dtype), 1 if delta_softplus else 0, 0)
    stream = _stream(dev)
    with _on_device(dev):
        if want_ck:
            st = lib.mb_scan_fwd_ckpt(ctypes.byref(desc), _ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C),
                                      _ptr(D), _ptr(dt_bias), _ptr(z), _ptr(h0), _ptr(out), _ptr(h_last),
                                      _ptr(ck), stream)
        elif positions is None:
            st = lib.mb_scan_fwd(ctypes.byref(desc), _ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C),
                                 _ptr(D), _ptr(dt_bias), _ptr(z), _ptr(h0), _ptr(out), _ptr(h_last),
                                 stream)
        else:
            st = lib.mb_scan_fwd_states(ctypes.byref(desc), _ptr(u), _ptr(delta), _ptr(A), _ptr(B),
                                        _ptr(C), _ptr(D), _ptr(dt_bias), _ptr(z), _ptr(h0), _ptr(out),
                                        _ptr(h_last), _ptr(positions), npos, _ptr(h_at), stream)
    _check(st, "mb_scan_fwd_ckpt" if want_ck else "mb_scan_fwd" if positions is None else "mb_scan_fwd_states")
    res = (out,)
    if return_last_state or h_last is not None:
        res += (h_last,)
    if positions is not None:
        res += (h_at,)
    if want_ck:
        res += (ck,)
    return res[0] if len(res) == 1 else res


def scan_fwd_noalloc(u, delta, A, B, C, D=None, dt_bias=None, z=None, h0=None, *, out, h_last=None,
                     delta_softplus=True):
    """scan_fwd through mb_scan_fwd_noalloc: nothing is allocated, so the output y
    (``out``) and, if wanted, ``h_last`` are given by the caller (h_last may be h0).
    Returns y or (y, h_last)."""
    lib = load_library()
    if not isinstance(u, torch.Tensor) or u.dim() != 3 or not isinstance(A, torch.Tensor) or A.dim() != 2:
        raise MBScanError("u must be a (batch, dim, L) tensor and A a (dim, N) tensor")
    nb, dim, L = u.shape
    N = A.shape[1]
    dev, act = u.device, u.dtype
    for t, name, shape, dt in ((u, "u", (nb, dim, L), act), (delta, "delta", (nb, dim, L), act),
                               (A, "A", (dim, N), torch.float32), (B, "B", (nb, N, L), act),
                               (C, "C", (nb, N, L), act)):
        _need(t, name, shape, dt, dev)
    for t, name, shape, dt in ((z, "z", (nb, dim, L), act), (D, "D", (dim,), torch.float32),
                               (dt_bias, "dt_bias", (dim,), torch.float32),
                               (h0, "h0", (nb, dim, N), torch.float32),
                               (h_last, "h_last", (nb, dim, N), torch.float32)):
        if t is not None:
            _need(t, name, shape, dt, dev)
    if not isinstance(out, torch.Tensor) or out.dtype not in (torch.float32, torch.bfloat16):
        raise MBScanError("out must be a float32 or bfloat16 tensor")
    _need(out, "out", (nb, dim, L), out.dtype, dev)
    desc = ScanDesc(nb, dim, L, N, _dt(act), _dt(out.dtype), 1 if delta_softplus else 0, 0)
    with _on_device(dev):
        st = lib.mb_scan_fwd_noalloc(ctypes.byref(desc), _ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C),
                                     _ptr(D), _ptr(dt_bias), _ptr(z), _ptr(h0), _ptr(out), _ptr(h_last),
                                     _stream(dev))
    _check(st, "mb_scan_fwd_noalloc")
    return out if h_last is None else (out, h_last)


def scan_step(h, u_t, delta_t, A, B_t, C_t, D=None, dt_bias=None, z_t=None, *, delta_softplus=True,
              out_dtype=torch.float32, out=None):
    """One recurrent step; h (batch, dim, N) fp32 is updated in place.  Returns y_t (batch, dim)."""
    lib = load_library()
    if not isinstance(h, torch.Tensor) or h.dim() != 3:
        raise MBScanError("h must be a (batch, dim, N) tensor")
    nb, dim, N = h.shape
    dev, act = h.device, u_t.dtype
    _need(h, "h", (nb, dim, N), torch.float32, dev)
    _need(u_t, "u_t", (nb, dim), act, dev)
    _need(delta_t, "delta_t", (nb, dim), act, dev)
    _need(A, "A", (dim, N), torch.float32, dev)
    _need(B_t, "B_t", (nb, N), act, dev)
    _need(C_t, "C_t", (nb, N), act, dev)
    if z_t is not None:
        _need(z_t, "z_t", (nb, dim), act, dev)
    if D is not None:
        _need(D, "D", (dim,), torch.float32, dev)
    if dt_bias is not None:
        _need(dt_bias, "dt_bias", (dim,), torch.float32, dev)
    if out is None:
        out = torch.empty((nb, dim), dtype=out_dtype, device=dev)
    else:
        _need(out, "out", (nb, dim), None, dev)
    stream = _stream(dev)
    with _on_device(dev):
        st = lib.mb_scan_step(nb, dim, N, _dt(act), _dt(out.dtype), 1 if delta_softplus else 0,
                              _ptr(u_t), _ptr(delta_t), _ptr(A), _ptr(B_t), _ptr(C_t), _ptr(D),
                              _ptr(dt_bias), _ptr(z_t), _ptr(h), _ptr(out), stream)
    _check(st, "mb_scan_step")
    return out


def conv1d(x, w, bias=None, state=None, *, apply_silu=True, out_dtype=None, return_state=False,
           out=None, state_out=None):
    """Causal depthwise convolution (+ Swish) of x (batch, dim, L) with taps w (dim, k).

    bias: (dim,) fp32; state: (batch, dim, k-1) fp32, the k-1 inputs before x (zeros when
    None).  Returns y, or (y, state_out) where state_out holds the last k-1 inputs.
    """
    lib = load_library()
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise MBScanError("x must be a (batch, dim, L) tensor")
    nb, dim, L = x.shape
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise MBScanError("w must be a (dim, k) tensor")
    K = w.shape[1]
    dev = x.device
    _need(x, "x", (nb, dim, L), None, dev)
    _need(w, "w", (dim, K), torch.float32, dev)
    if bias is not None:
        _need(bias, "bias", (dim,), torch.float32, dev)
    if state is not None:
        _need(state, "state", (nb, dim, K - 1), torch.float32, dev)
    if out is None:
        out = torch.empty((nb, dim, L), dtype=out_dtype or x.dtype, device=dev)
    else:
        _need(out, "out", (nb, dim, L), None, dev)
    if return_state and state_out is None:
        state_out = torch.empty((nb, dim, max(K - 1, 0)), dtype=torch.float32, device=dev)
    elif state_out is not None:
        _need(state_out, "state_out", (nb, dim, K - 1), torch.float32, dev)
    desc = ConvDesc(nb, dim, L, K, _dt(x.dtype), _dt(out.dtype), 1 if apply_silu else 0, 0, 0)
    stream = _stream(dev)
    with _on_device(dev):
        st = lib.mb_conv1d_fwd(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias), _ptr(state), _ptr(out),
                               _ptr(state_out) if K > 1 else None, stream)
    _check(st, "mb_conv1d_fwd")
    return (out, state_out) if (return_state or state_out is not None) else out


def conv1d_step(state, x_t, w, bias=None, *, apply_silu=True, out_dtype=None, out=None):
    """One byte of the convolution; state (batch, dim, k-1) fp32 is updated in place.
    Returns y_t (batch, dim)."""
    lib = load_library()
    if not isinstance(x_t, torch.Tensor) or x_t.dim() != 2:
        raise MBScanError("x_t must be a (batch, dim) tensor")
    nb, dim = x_t.shape
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise MBScanError("w must be a (dim, k) tensor")
    K = w.shape[1]
    dev = x_t.device
    _need(x_t, "x_t", (nb, dim), None, dev)
    _need(w, "w", (dim, K), torch.float32, dev)
    if bias is not None:
        _need(bias, "bias", (dim,), torch.float32, dev)
    if K > 1:
        _need(state, "state", (nb, dim, K - 1), torch.float32, dev)
    if out is None:
        out = torch.empty((nb, dim), dtype=out_dtype or x_t.dtype, device=dev)
    else:
        _need(out, "out", (nb, dim), None, dev)
    stream = _stream(dev)
    with _on_device(dev):
        st = lib.mb_conv1d_step(nb, dim, K, _dt(x_t.dtype), _dt(out.dtype), 1 if apply_silu else 0,
                                _ptr(x_t), _ptr(w), _ptr(bias), _ptr(state) if K > 1 else None,
                                _ptr(out), stream)
    _check(st, "mb_conv1d_step")
    return out


def verify_rank(logits, draft, beta, *, return_ranks=False):
    """Top-beta check of drafted bytes.  logits: (batch, ndraft, vocab) fp32 or bf16;
    draft: int32 (batch, ndraft).  Returns (accepted, last_pos), each int32 (batch,),
    and the int32 (batch, ndraft) ranks when ``return_ranks``."""
    lib = load_library()
    if not isinstance(logits, torch.Tensor) or logits.dim() != 3:
        raise MBScanError("logits must be a (batch, ndraft, vocab) tensor")
    nb, n, V = logits.shape
    dev = logits.device
    _need(logits, "logits", (nb, n, V), None, dev)
    _need(draft, "draft", (nb, n), torch.int32, dev)
    accepted = torch.empty(nb, dtype=torch.int32, device=dev)
    last_pos = torch.empty(nb, dtype=torch.int32, device=dev)
    ranks = torch.empty((nb, n), dtype=torch.int32, device=dev) if return_ranks else None
    stream = _stream(dev)
    with _on_device(dev):
        st = lib.mb_verify_rank(nb, n, V, _dt(logits.dtype), int(beta), _ptr(logits), _ptr(draft),
                                _ptr(ranks), _ptr(accepted), _ptr(last_pos), stream)
    _check(st, "mb_verify_rank")
    return (accepted, last_pos, ranks) if return_ranks else (accepted, last_pos)


def scan_bwd(u, delta, A, B, C, dy, D=None, dt_bias=None, z=None, h0=None, dh_last=None, *,
             delta_softplus=True, ck=None):
    """Gradients of sum(dy * y) + sum(dh_last * h_last) for the scan of scan_fwd.

    ``ck``: the checkpoints of ``scan_fwd(..., return_ckpt=True)`` on the same inputs;
    without them the call recomputes them with one more forward pass.

    dy has y's dtype (fp32 or bf16), shape (batch, dim, L).  Returns a dict: du, ddelta,
    dz (dy's dtype, (batch, dim, L); dz None without a gate), dA (dim, N), dB, dC
    (batch, N, L), dD and dt_bias gradients ``dD``, ``ddt_bias`` (dim,) or None, and
    dh0 (batch, dim, N), all fp32 but the first three.
    """
    lib = load_library()
    if not isinstance(u, torch.Tensor) or u.dim() != 3:
        raise MBScanError("u must be a (batch, dim, L) tensor")
    nb, dim, L = u.shape
    if not isinstance(A, torch.Tensor) or A.dim() != 2:
        raise MBScanError("A must be a (dim, N) tensor")
    N = A.shape[1]
    dev, act = u.device, u.dtype
    for t, name, shape, dt in ((u, "u", (nb, dim, L), act), (delta, "delta", (nb, dim, L), act),
                               (A, "A", (dim, N), torch.float32), (B, "B", (nb, N, L), act),
                               (C, "C", (nb, N, L), act), (dy, "dy", (nb, dim, L), None)):
        _need(t, name, shape, dt, dev)
    for t, name, shape, dt in ((z, "z", (nb, dim, L), act), (D, "D", (dim,), torch.float32),
                               (dt_bias, "dt_bias", (dim,), torch.float32),
                               (h0, "h0", (nb, dim, N), torch.float32),
                               (dh_last, "dh_last", (nb, dim, N), torch.float32),
                               (ck, "ck", (L // 16, nb, dim, N), torch.float32)):
        if t is not None:
            _need(t, name, shape, dt, dev)
    f32 = dict(dtype=torch.float32, device=dev)
    g = {"du": torch.empty((nb, dim, L), dtype=dy.dtype, device=dev),
         "ddelta": torch.empty((nb, dim, L), dtype=dy.dtype, device=dev),
         "dz": torch.empty((nb, dim, L), dtype=dy.dtype, device=dev) if z is not None else None,
         "dA": torch.empty((dim, N), **f32), "dB": torch.empty((nb, N, L), **f32),
         "dC": torch.empty((nb, N, L), **f32),
         "dD": torch.empty(dim, **f32) if D is not None else None,
         "ddt_bias": torch.empty(dim, **f32) if dt_bias is not None else None,
         "dh0": torch.empty((nb, dim, N), **f32)}
    desc = ScanDesc(nb, dim, L, N, _dt(act), _dt(dy.dtype), 1 if delta_softplus else 0, 0)
    stream = _stream(dev)
    with _on_device(dev):
        st = lib.mb_scan_bwd(ctypes.byref(desc), _ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C), _ptr(D),
                             _ptr(dt_bias), _ptr(z), _ptr(h0), _ptr(dy), _ptr(dh_last), _ptr(ck),
                             _ptr(g["du"]),
                             _ptr(g["ddelta"]), _ptr(g["dz"]), _ptr(g["dA"]), _ptr(g["dB"]), _ptr(g["dC"]),
                             _ptr(g["dD"]), _ptr(g["ddt_bias"]), _ptr(g["dh0"]), stream)
    _check(st, "mb_scan_bwd")
    return g

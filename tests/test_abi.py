"""The C ABI on the CPU: the library loads, exports what the header declares,
and rejects bad arguments before touching the GPU (no compute call is made)."""
import ctypes
import os
import re

import pytest

import paper_2401_13660_amd as mb
from paper_2401_13660_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mbscan.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="libmbscan.so not built")

# The argument-error cases hand the library fake device addresses.  Each case
# is invalid, so validation rejects it before any launch; as a second guard
# they only run where no GPU driver is present (the CPU suite), never on a GPU.
no_gpu_only = pytest.mark.skipif(os.path.exists("/dev/kfd"),
                                 reason="fake-pointer error paths run only on a machine without a GPU")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mb_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = mb.load_library()
    names = declared_functions()
    assert {"mb_scan_fwd", "mb_scan_fwd_states", "mb_scan_step", "mb_conv1d_fwd", "mb_conv1d_step",
            "mb_verify_rank", "mb_scan_bwd", "mb_scan_fwd_ckpt", "mb_status_string",
            "mb_abi_version"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in mbscan.h but not exported"


def test_version_and_status_strings():
    lib = mb.load_library()
    assert lib.mb_abi_version() == 6
    for code in range(-7, 1):
        assert lib.mb_status_string(code)
    assert lib.mb_status_string(-99) == b"unknown status"


def _desc(**kw):
    d = dict(batch=2, dim=8, seqlen=16, dstate=16, in_dtype=1, out_dtype=0, delta_softplus=1, reserved=0)
    d.update(kw)
    return B.ScanDesc(**d)


# Fake, distinct, well-aligned "device" addresses: every call below must fail
# validation, so none of them is ever dereferenced.
P = {k: 0x10000000 * (i + 1) for i, k in enumerate(
    ["u", "delta", "A", "B", "C", "D", "bias", "z", "h0", "y", "hl"])}


def _fwd(desc, **over):
    a = dict(P)
    a.update(over)
    lib = mb.load_library()
    return lib.mb_scan_fwd(ctypes.byref(desc) if desc is not None else None, a["u"], a["delta"], a["A"],
                           a["B"], a["C"], a["D"], a["bias"], a["z"], a["h0"], a["y"], a["hl"], None)


@no_gpu_only
@pytest.mark.parametrize("desc,over,code", [
    (None, {}, -1),
    (_desc(batch=-1), {}, -2),
    (_desc(seqlen=-5), {}, -2),
    (_desc(batch=1 << 40, dim=1 << 20, seqlen=1 << 10), {}, -2),
    (_desc(batch=1 << 61, dim=1, seqlen=16), {}, -2),   # batch x dstate alone past the bound
    (_desc(in_dtype=7), {}, -3),
    (_desc(out_dtype=-1), {}, -3),
    (_desc(dstate=3), {}, -5),
    (_desc(dstate=32), {}, -5),
    (_desc(reserved=1), {}, -5),
    (_desc(), dict(u=None), -1),
    (_desc(), dict(A=None), -1),
    (_desc(), dict(y=None), -1),
    (_desc(), dict(B=None), -1),
    (_desc(), dict(u=P["u"] + 1), -4),                  # bf16 needs 2-byte alignment
    (_desc(in_dtype=0), dict(delta=P["delta"] + 2), -4),  # fp32 needs 4-byte alignment
    (_desc(), dict(hl=P["hl"] + 2), -4),
    (_desc(), dict(y=P["u"] + 64), -7),                  # y inside u
    (_desc(), dict(hl=P["z"]), -7),                      # h_last on top of z
    (_desc(), dict(hl=P["h0"] + 64), -7),                # h_last partially over h0
])
def test_fwd_rejects(desc, over, code):
    assert _fwd(desc, **over) == code


def _fwd_states(desc, npos, **over):
    a = dict(P, pos=0x0c000000, hpos=0x0e000000)
    a.update(over)
    lib = mb.load_library()
    return lib.mb_scan_fwd_states(ctypes.byref(desc), a["u"], a["delta"], a["A"], a["B"], a["C"], a["D"],
                                  a["bias"], a["z"], a["h0"], a["y"], a["hl"], a["pos"], npos, a["hpos"],
                                  None)


@no_gpu_only
@pytest.mark.parametrize("npos,over,code", [
    (-1, {}, -2),
    (1 << 62, {}, -2),
    (2, dict(pos=None), -1),
    (2, dict(hpos=None), -1),
    (2, dict(pos=0x0c000002), -4),                      # int32 positions need 4-byte alignment
    (2, dict(hpos=0x0e000002), -4),
    (2, dict(hpos=P["u"] + 256), -7),                   # h_pos inside u
    (2, dict(hpos=P["h0"]), -7),                        # h_pos on top of h0
    (2, dict(hpos=P["hl"]), -7),                        # h_pos on top of h_last
    (2, dict(pos=P["y"]), -7),                          # positions inside the output
    (2, dict(hpos=0x0c000000 - 64), -7),                # h_pos running into the positions
    (1, dict(u=None), -1),                              # the mb_scan_fwd checks still apply
])
def test_fwd_states_rejects(npos, over, code):
    assert _fwd_states(_desc(), npos, **over) == code


CK = 0x0a000000


def _fwd_ckpt(desc, **over):
    a = dict(P, ck=CK)
    a.update(over)
    lib = mb.load_library()
    return lib.mb_scan_fwd_ckpt(ctypes.byref(desc), a["u"], a["delta"], a["A"], a["B"], a["C"], a["D"],
                                a["bias"], a["z"], a["h0"], a["y"], a["hl"], a["ck"], None)


@no_gpu_only
@pytest.mark.parametrize("desc,over,code", [
    (_desc(), dict(ck=None), -1),
    (_desc(dstate=8), {}, -5),                          # checkpoints exist for dstate 16 only
    (_desc(seqlen=24), {}, -5),                         # and L a multiple of 16
    (_desc(), dict(u=P["u"] + 2), -4),                  # activations 16-byte aligned
    (_desc(), dict(y=P["y"] + 8), -4),
    (_desc(), dict(ck=CK + 4), -4),
    (_desc(), dict(ck=P["u"] + 16), -7),                # checkpoints inside u
    (_desc(), dict(ck=P["y"]), -7),                     # on top of y
    (_desc(), dict(ck=P["hl"] - 64), -7),               # running into h_last
    (_desc(), dict(A=None), -1),                        # the mb_scan_fwd checks still apply
])
def test_fwd_ckpt_rejects(desc, over, code):
    assert _fwd_ckpt(desc, **over) == code


BP = {k: 0x30000000 + 0x01000000 * i for i, k in enumerate(
    ["u", "delta", "A", "B", "C", "D", "bias", "z", "h0", "dy", "dhl", "ck", "du", "ddelta", "dz", "dA", "dB",
     "dC", "dD", "dbias", "dh0"])}


def _bwd(desc, **over):
    a = dict(BP)
    a.update(over)
    lib = mb.load_library()
    order = ["u", "delta", "A", "B", "C", "D", "bias", "z", "h0", "dy", "dhl", "ck", "du", "ddelta", "dz", "dA",
             "dB", "dC", "dD", "dbias", "dh0"]
    return lib.mb_scan_bwd(ctypes.byref(desc) if desc is not None else None, *[a[k] for k in order], None)


@no_gpu_only
@pytest.mark.parametrize("desc,over,code", [
    (None, {}, -1),
    (_desc(batch=-1), {}, -2),
    (_desc(batch=1 << 61, dim=1, seqlen=16), {}, -2),
    (_desc(in_dtype=9), {}, -3),
    (_desc(dstate=8), {}, -5),
    (_desc(seqlen=24), {}, -5),
    (_desc(seqlen=1 << 25), {}, -5),                    # lane offsets are 32-bit
    (_desc(reserved=1), {}, -5),
    (_desc(), dict(dy=None), -1),
    (_desc(), dict(dA=None), -1),
    (_desc(), dict(dz=None), -1),                       # z given, dz missing
    (_desc(), dict(dD=None), -1),                       # Dskip given, its gradient missing
    (_desc(), dict(du=BP["du"] + 4), -4),               # activations and gradients 16-byte aligned
    (_desc(), dict(ck=BP["ck"] + 4), -4),
    (_desc(), dict(du=BP["u"] + 32), -7),               # an output inside an input
    (_desc(), dict(dB=BP["ck"]), -7),                   # an output on the checkpoints
    (_desc(), dict(dC=BP["dB"] + 64), -7),              # two outputs overlapping
])
def test_bwd_rejects(desc, over, code):
    assert _bwd(desc, **over) == code


def _cdesc(**kw):
    d = dict(batch=2, dim=8, seqlen=16, width=4, in_dtype=1, out_dtype=1, apply_silu=1, reserved=0,
             reserved2=0)
    d.update(kw)
    return B.ConvDesc(**d)


CP = {k: 0x20000000 * (i + 1) for i, k in enumerate(["x", "w", "bias", "sin", "y", "sout"])}


def _conv(desc, **over):
    a = dict(CP)
    a.update(over)
    lib = mb.load_library()
    return lib.mb_conv1d_fwd(ctypes.byref(desc) if desc is not None else None, a["x"], a["w"], a["bias"],
                             a["sin"], a["y"], a["sout"], None)


@no_gpu_only
@pytest.mark.parametrize("desc,over,code", [
    (None, {}, -1),
    (_cdesc(seqlen=-1), {}, -2),
    (_cdesc(batch=1 << 40, dim=1 << 20, seqlen=1 << 10), {}, -2),
    (_cdesc(in_dtype=5), {}, -3),
    (_cdesc(width=0), {}, -5),
    (_cdesc(width=5), {}, -5),
    (_cdesc(reserved=1), {}, -5),
    (_cdesc(reserved2=3), {}, -5),
    (_cdesc(), dict(x=None), -1),
    (_cdesc(), dict(w=None), -1),
    (_cdesc(), dict(y=None), -1),
    (_cdesc(), dict(x=CP["x"] + 1), -4),
    (_cdesc(), dict(sout=CP["sout"] + 2), -4),
    (_cdesc(), dict(y=CP["x"] + 32), -7),                # y inside x
    (_cdesc(), dict(sout=CP["sin"]), -7),                # state_out on top of state_in
    (_cdesc(), dict(sout=CP["y"] + 16), -7),             # state_out inside y
])
def test_conv_rejects(desc, over, code):
    assert _conv(desc, **over) == code


@no_gpu_only
def test_conv_step_rejects():
    lib = mb.load_library()
    f = lib.mb_conv1d_step
    ok = [CP["x"], CP["w"], CP["bias"], CP["sin"], CP["y"], None]
    assert f(-1, 8, 4, 1, 1, 1, *ok) == -2
    assert f(2, 8, 9, 1, 1, 1, *ok) == -5
    assert f(2, 8, 4, 2, 1, 1, *ok) == -3
    bad = list(ok); bad[3] = None                       # the state is required for k > 1
    assert f(2, 8, 4, 1, 1, 1, *bad) == -1
    bad = list(ok); bad[4] = CP["x"]                    # y_t on top of x_t
    assert f(2, 8, 4, 1, 1, 1, *bad) == -7
    bad = list(ok); bad[3] = CP["w"]                    # state on top of w
    assert f(2, 8, 4, 1, 1, 1, *bad) == -7
    assert f(0, 8, 4, 1, 1, 1, *ok) == 0


RP = {k: 0x30000000 * (i + 1) for i, k in enumerate(["logits", "draft", "ranks", "acc", "last"])}


@no_gpu_only
@pytest.mark.parametrize("args,over,code", [
    ((-1, 16, 256), {}, -2),
    ((4, -1, 256), {}, -2),
    ((4, 16, 0), {}, -2),
    ((4, 1 << 31, 256), {}, -2),
    ((4, 16, 256, 7), {}, -3),
    ((4, 16, 256), dict(acc=None), -1),
    ((4, 16, 256), dict(logits=None), -1),
    ((4, 16, 256), dict(draft=RP["draft"] + 2), -4),
    ((4, 16, 256), dict(acc=RP["logits"] + 64), -7),     # output inside the logits
    ((4, 16, 256), dict(last=RP["acc"]), -7),            # two outputs on top of each other
    ((4, 16, 256), dict(ranks=RP["draft"]), -7),
])
def test_verify_rank_rejects(args, over, code):
    a = dict(RP)
    a.update(over)
    batch, n, V = args[:3]
    dt = args[3] if len(args) > 3 else 0
    lib = mb.load_library()
    assert lib.mb_verify_rank(batch, n, V, dt, 3, a["logits"], a["draft"], a["ranks"], a["acc"], a["last"],
                              None) == code


@no_gpu_only
def test_fwd_empty_problem_is_ok_and_launches_nothing():
    assert _fwd(_desc(batch=0)) == 0
    assert _fwd(_desc(dim=0), u=None, delta=None, A=None) == 0


@no_gpu_only
def test_step_rejects():
    lib = mb.load_library()
    f = lib.mb_scan_step
    ok = [P["u"], P["delta"], P["A"], P["B"], P["C"], P["D"], P["bias"], P["z"], P["h0"], P["y"], None]
    assert f(-1, 8, 16, 1, 0, 1, *ok) == -2
    assert f(1, 1 << 36, 16, 1, 0, 1, *ok) == -2         # dim at the launch bound (2^36)
    assert f(2, 8, 12, 1, 0, 1, *ok) == -5
    assert f(2, 8, 16, 4, 0, 1, *ok) == -3
    bad = list(ok); bad[8] = None                       # h is required
    assert f(2, 8, 16, 1, 0, 1, *bad) == -1
    bad = list(ok); bad[9] = P["u"]                     # y_t on top of u_t
    assert f(2, 8, 16, 1, 0, 1, *bad) == -7
    bad = list(ok); bad[8] = P["A"]                     # h on top of A
    assert f(2, 8, 16, 1, 0, 1, *bad) == -7
    assert f(0, 8, 16, 1, 0, 1, *ok) == 0


def test_binding_fails_loudly_without_library(tmp_path):
    saved = B._lib
    try:
        B._lib = None
        with pytest.raises(B.MBScanError):
            B.load_library(str(tmp_path / "missing.so"))
    finally:
        B._lib = saved


def test_header_is_c_and_matches_the_binding(tmp_path):
    """include/mbscan.h compiles as C99 (-pedantic), and its structs have the
    layout the ctypes binding declares."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = tmp_path / "layout.c"
    src.write_text(
        '#include "mbscan.h"\n#include <stddef.h>\n#include <stdio.h>\n'
        "int main(void) {\n"
        '  printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(mb_scan_desc), offsetof(mb_scan_desc, in_dtype),\n'
        "         offsetof(mb_scan_desc, reserved), sizeof(mb_conv_desc), offsetof(mb_conv_desc, width),\n"
        "         offsetof(mb_conv_desc, reserved2));\n"
        "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-pedantic", "-I", os.path.dirname(HEADER), str(src),
                    "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()]
    want = [ctypes.sizeof(B.ScanDesc), B.ScanDesc.in_dtype.offset, B.ScanDesc.reserved.offset,
            ctypes.sizeof(B.ConvDesc), B.ConvDesc.width.offset, B.ConvDesc.reserved2.offset]
    assert got == want, f"C layout {got} != ctypes layout {want}"

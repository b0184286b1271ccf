#!/usr/bin/env python3
"""Benchmark of the selective scan on one MI355X.

One step = one mb_scan_fwd over the MambaByte-972M layer shape (batch 4,
L = 8,192 bytes, dim 3,584, N = 16; bf16 activations, fp32 output and state,
z-gated) with inputs already resident in HBM.  Prints one JSON line with the
whole-job throughput (algorithmic GB/s), B*L*D elements/s, the HBM roofline of
the scan kernel and the fp64 CPU oracle timed on this host's cores over the
same workload (which doubles as the parity gate).

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s

# Issue model of the scan, reported beside the HBM roofline (which is the
# roofline of record).  Rates measured on MI355X by paper_2401_13660_amd/issue_rates
# (csrc/issue_rates.hip; register-only instruction streams, kernel time from events
# over a grid with W waves on every SIMD, shader clock read in the kernel):
#  - a transcendental (v_exp_f32) holds its SIMD for 8.0-9.2 cycles at any
#    occupancy (8.6 with 2 waves per SIMD) and no other VALU instruction issues
#    meanwhile, not even from another wave;
#  - other fp32 VALU instructions reach 2.3-2.5 cycles with two or more waves per
#    SIMD only in streams without transcendentals (two waves issue in the same
#    cycle; one wave alone issues one about every 7 cycles), and only when no
#    operand is an SGPR and the two multiplicand VGPRs of a multiply-add differ in
#    parity (index mod 2);
#  - with one transcendental per four other instructions, as in the scan, and 2
#    waves per SIMD (the scan's occupancy), the mix averages 5.0 cycles per
#    instruction: 8.6 for the exponential and 4.1 for each of the others.
# Per element the forward needs at least 76 VALU and 20 transcendental
# lane-operations: per state dlt * A, its exponential, dlt * u * B, the state FMA
# and the C FMA (64 + 16), and per element softplus (exp, log), silu (exp, rcp) and
# about 12 VALU operations.  At those rates and 2.4 GHz that is 7.6 SIMD-cycles per
# element.
VALU_CYCLES, TRANS_CYCLES = 4.1, 8.6
ALU_SIMD_CYCLES_PER_ELEMENT = (76 * VALU_CYCLES + 20 * TRANS_CYCLES) / 64.0
ALU_PEAK_GELEMS = 1024 * 2.4e9 / ALU_SIMD_CYCLES_PER_ELEMENT / 1e9
# The same model for the backward (the gradients of eq. (2) by reverse-mode
# differentiation), per element.  Per state: the forward recomputed (dlt * A, the
# exponential, dlt * u * B, the state FMA), lambda and its carry (2), dB and dC
# (a product and a sum over channels each: 4), sum_n lambda B (1), the decay term
# lambda abar h_{t-1} with its A-weighted sum and the dA sum (3) and C . h for dz
# (1): 14 VALU + 1 transcendental.  Per element at least 5 transcendentals
# (softplus: exp, log, its derivative: rcp; silu: exp, rcp) and 16 VALU
# operations (ds, dz, du, ddelta, the dDskip and dbias sums, dlt * u).
BWD_SIMD_CYCLES_PER_ELEMENT = ((16 + 5) * TRANS_CYCLES + (16 * 14 + 16) * VALU_CYCLES) / 64.0
BWD_ALU_PEAK_GELEMS = 1024 * 2.4e9 / BWD_SIMD_CYCLES_PER_ELEMENT / 1e9
TRAIN_ALU_PEAK_GELEMS = 1024 * 2.4e9 / (ALU_SIMD_CYCLES_PER_ELEMENT + BWD_SIMD_CYCLES_PER_ELEMENT) / 1e9
METRIC = "selective-scan GB/s & %HBM peak (972M layer, L=8192); B·L·D elems/s"
DEFAULT_WORKLOAD = "mambabyte972m_L8192"
from paper_2401_13660_amd.profile_summary import (  # noqa: E402
    CONV_KERNEL_SOURCES, KERNEL_SOURCES, TRAFFIC_FILE, kernel_sources_digest)


def algorithmic_bytes(inp, out_bytes=4, want_h_last=False) -> int:
    """Each input read once and each output written once (the roofline's bytes)."""
    act = 2 if inp.dtype == "bf16" else 4
    E = inp.batch * inp.dim * inp.seqlen
    n_act = 2 + (1 if inp.z is not None else 0)                  # u, delta (, z)
    b = E * (n_act * act + out_bytes)
    b += 2 * inp.batch * inp.dstate * inp.seqlen * act            # B, C
    b += inp.dim * inp.dstate * 4                                 # A
    b += inp.dim * 4 * ((inp.Dskip is not None) + (inp.dt_bias is not None))
    state = inp.batch * inp.dim * inp.dstate * 4
    b += state * ((inp.h0 is not None) + bool(want_h_last))
    return int(b)


def step_bytes(inp) -> int:
    """Algorithmic bytes of seqlen successive one-byte steps: each step reads its
    activations, B_t, C_t and the parameters, reads and writes the whole state,
    and writes y_t."""
    act = 2 if inp.dtype == "bf16" else 4
    rows = inp.batch * inp.dim
    per = rows * ((2 + (inp.z is not None)) * act + 4)
    per += 2 * inp.batch * inp.dstate * act
    per += inp.dim * inp.dstate * 4 + inp.dim * 4 * ((inp.Dskip is not None) + (inp.dt_bias is not None))
    per += 2 * rows * inp.dstate * 4
    return int(per * inp.seqlen)


def measured_traffic(workload: str, sources=KERNEL_SOURCES):
    """HBM bytes per step from the committed rocprofv3 PMC summary (the scan
    kernel, plus the segment pre-pass where the workload has one), if it was
    taken on the current kernel sources (else None)."""
    try:
        with open(TRAFFIC_FILE) as f:
            recs = json.load(f)
    except (OSError, ValueError):
        return None
    digest = kernel_sources_digest(sources)
    total = 0
    for key in (workload, "prepass:" + workload):
        rec = recs.get(key)
        if rec is None and key != workload:
            continue
        if not rec or rec.get("kernel_sources") != digest:
            return None
        total += rec.get("hbm_bytes_per_launch", 0)
    return total


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# An idle GPU's clocks settle over the first tens of milliseconds of sustained
# work: back to back, the 972M-layer scan goes from about 760 to 545 us per
# launch over its first 35 ms.  The warm-up therefore runs its W steps and then
# keeps stepping until WARMUP_MIN_S seconds have passed.
WARMUP_MIN_S = 0.2


def warm_up(step, n: int) -> int:
    """n untimed steps, then more until WARMUP_MIN_S has passed; returns the extra steps."""
    import torch

    t0 = time.perf_counter()
    for _ in range(n):
        step()
    torch.cuda.synchronize()
    extra = 0
    while time.perf_counter() - t0 < WARMUP_MIN_S:
        for _ in range(8):
            step()
        extra += 8
        torch.cuda.synchronize()
    return extra


def per_launch_ms(run, n, flush=None):
    """Device time of each of n back-to-back launches, from events recorded between
    consecutive launches on the launch stream (no synchronisation inside the loop,
    so the host stays ahead and no idle time falls between the events).  With
    ``flush``, that callable is enqueued before every launch, outside its events.
    Returns the sorted times."""
    import torch
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    for i in range(n):
        if flush is not None:
            flush()
        starts[i].record()
        run()
        ends[i].record()
    torch.cuda.synchronize()
    return sorted(a.elapsed_time(b) for a, b in zip(starts, ends))


def copy_bandwidth_gbs(dev, mib=1024, reps=5) -> float:
    """Bandwidth of a plain device copy (mib MiB read + mib MiB written): the
    practical ceiling that a streaming kernel is also compared with."""
    import torch
    src = torch.ones((mib << 20) // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    secs = a.elapsed_time(b) / reps * 1e-3
    del src, dst
    return 2 * (mib << 20) / secs / 1e9


CPU_REPEATS = 3                 # the oracle's time is the best of this many runs


def cpu_baseline(inp, y_gpu, h_gpu=None):
    """fp64 oracle on this host's cores over the whole workload, batch by batch, best
    of CPU_REPEATS runs; the first run is also the parity gate for the GPU output of
    the same inputs.  A workload of at most 2^20 elements is also timed on one core."""
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import TOL_H, TOL_Y, TOL_Y_BF16_OUT, rel_err

    orc = oracle.default()
    threads = orc.max_threads()

    def whole(check):
        elapsed, worst_y, worst_h = 0.0, 0.0, 0.0
        for b in range(inp.batch):
            rows = np.arange(b * inp.dim, (b + 1) * inp.dim)
            t0 = time.perf_counter()
            y_ref, h_ref = oracle.scan_inputs(inp, rows=rows)
            elapsed += time.perf_counter() - t0
            if check:
                yg = y_gpu[b].float().cpu().numpy().astype(np.float64)
                worst_y = max(worst_y, rel_err(yg, y_ref))
                if h_gpu is not None:
                    worst_h = max(worst_h, rel_err(h_gpu[b].cpu().numpy().astype(np.float64), h_ref))
        return elapsed, worst_y, worst_h

    runs = []
    worst_y = worst_h = 0.0
    for i in range(CPU_REPEATS):
        el, wy, wh = whole(i == 0)
        runs.append(el)
        if i == 0:
            worst_y, worst_h = wy, wh
    E = inp.batch * inp.dim * inp.seqlen
    tol = TOL_Y_BF16_OUT if y_gpu.element_size() == 2 else TOL_Y
    res = dict(elapsed=min(runs), runs=runs, elems_per_s=E / min(runs), threads=threads, y_err=worst_y,
               h_err=worst_h if h_gpu is not None else None, parity_ok=worst_y <= tol and worst_h <= TOL_H)
    if E <= (1 << 20):
        orc.set_threads(1)
        try:
            one = [whole(False)[0] for _ in range(CPU_REPEATS)]
        finally:
            orc.set_threads(threads)
        res["single_thread"] = dict(elapsed=min(one), elems_per_s=E / min(one))
    return res


def cpu_baseline_steps(inp, ycols, state_gpu):
    """The oracle's one-byte step, applied seqlen times over the batch (best of
    CPU_REPEATS); the first pass checks every step's y and the final state."""
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import TOL_H, TOL_Y, rel_err

    orc = oracle.default()
    runs, worst_y, worst_h = [], 0.0, 0.0
    for i in range(CPU_REPEATS):
        h = inp.h0 if inp.h0 is not None else np.zeros((inp.batch, inp.dim, inp.dstate))
        el = 0.0
        for t in range(inp.seqlen):
            col = lambda a: None if a is None else np.ascontiguousarray(a[..., t])
            t0 = time.perf_counter()
            y_ref, h = orc.scan_step(h, col(inp.u), col(inp.delta), inp.A, col(inp.B), col(inp.C),
                                     z_t=col(inp.z), Dskip=inp.Dskip, dt_bias=inp.dt_bias, dtype=inp.dtype)
            el += time.perf_counter() - t0
            if i == 0:
                worst_y = max(worst_y, rel_err(ycols[t].cpu().numpy().astype(np.float64), y_ref))
        if i == 0:
            worst_h = rel_err(state_gpu.cpu().numpy().astype(np.float64), h)
        runs.append(el)
    E = inp.batch * inp.dim * inp.seqlen
    return dict(elapsed=min(runs), runs=runs, elems_per_s=E / min(runs), threads=orc.max_threads(),
                y_err=worst_y, h_err=worst_h, parity_ok=worst_y <= TOL_Y and worst_h <= TOL_H)


def conv_bytes(c, out_bytes=2) -> int:
    """Each input read once and each output written once (the roofline's bytes)."""
    act = 2 if c.dtype == "bf16" else 4
    E = c.batch * c.dim * c.seqlen
    b = E * (act + out_bytes) + c.dim * c.width * 4 + (c.dim * 4 if c.bias is not None else 0)
    st = c.batch * c.dim * (c.width - 1) * 4
    return int(b + st * (1 + (c.state is not None)))


def bench_conv(args):
    """One mb_conv1d_fwd per step over the named workload's (batch, dim, L): the
    convolution + Swish whose bf16 output is the scan's u (and x_proj's input)."""
    import torch

    import paper_2401_13660_amd as mb
    from paper_2401_13660_amd.inputs import WORKLOADS, conv_workload

    c = conv_workload(args.workload, seed=0)
    dev = torch.device("cuda:0")

    def t(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    x, w, bias, state = t(c.x), t(c.w), t(c.bias), t(c.state)
    y = torch.empty_like(x, dtype=torch.bfloat16)
    state_out = torch.empty((c.batch, c.dim, c.width - 1), dtype=torch.float32, device=dev)

    def step():
        mb.conv1d(x, w, bias=bias, state=state, out=y, state_out=state_out)

    extra_warmup = warm_up(step, args.warmup)
    if args.graph:
        # one step captured once (warm-up on a side stream first), then replayed:
        # the per-call host work of the binding leaves the timed region
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run = graph.replay
    else:
        run = step
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    E = c.batch * c.dim * c.seqlen
    nbytes = conv_bytes(c)
    gbs = nbytes / (ms * 1e-3) / 1e9
    line = {
        "metric": "causal-conv1d GB/s & %HBM peak (in front of the scan); B·L·D elems/s",
        "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "warmup_extra_steps": extra_warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "mode": "conv", "width": c.width,
                   **{k: v for k, v in WORKLOADS[args.workload].items() if k != "dstate"},
                   "state": c.state is not None, "out_dtype": "bf16", "parallelism": "single GPU"},
        "elems_per_s": round(E / (ms * 1e-3), 1),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("conv:" + args.workload, CONV_KERNEL_SOURCES),
                     "algorithmic_bytes": nbytes},
    }
    if not args.no_cpu_baseline:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from parity import rel_err

        orc = oracle.default()
        t0 = time.perf_counter()
        y_ref, st_ref = orc.conv1d(c.x, c.w, bias=c.bias, state=c.state, dtype=c.dtype)
        elapsed = time.perf_counter() - t0
        err = rel_err(y.float().cpu().numpy(), y_ref)
        ok = err <= 1e-5 + 2.0 ** -8 and np.array_equal(state_out.cpu().numpy().astype(np.float64), st_ref)
        line["cpu_baseline"] = {
            "value": round(nbytes / elapsed / 1e9, 3), "unit": "GB/s", "elems_per_s": round(E / elapsed, 1),
            "cores": orc.max_threads(), "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"whole workload: {c.batch} x {c.dim} rows of L={c.seqlen}, fp64, {elapsed:.1f} s"}
        line["parity"] = {"y_rel_err_vs_oracle": err, "ok": bool(ok)}
        if not ok:
            print(json.dumps(line))
            print("parity gate failed: GPU output disagrees with the oracle", file=sys.stderr)
            sys.exit(1)
    print(json.dumps(line))


def bwd_bytes(inp) -> int:
    """Each input read once and each output written once: u, delta, z, dy in and du,
    ddelta, dz out (bf16), B and C in (bf16), dB and dC out (fp32), the parameters."""
    E = inp.batch * inp.dim * inp.seqlen
    bnl = inp.batch * inp.dstate * inp.seqlen
    b = E * 2 * (4 + 3) + bnl * (2 * 2 + 2 * 4)
    b += inp.dim * inp.dstate * 4 * 2 + inp.dim * 4 * 2 * 2
    b += inp.batch * inp.dim * inp.dstate * 4 * (1 + (inp.h0 is not None))
    return int(b)


def bench_bwd(args, train=False):
    """One mb_scan_bwd per step over the workload: the backward of the scan in the
    training setting (bf16 activations and incoming gradient, bf16 activation
    gradients, fp32 parameter gradients).  ``train``: a step is the training pair,
    the forward that stores the checkpoints (bf16 y) and the backward that reads
    them."""
    import torch

    import paper_2401_13660_amd as mb
    from paper_2401_13660_amd.inputs import WORKLOADS, workload

    inp = workload(args.workload, seed=0)
    dev = torch.device("cuda:0")

    def t(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    g = {k: t(v) for k, v in inp.arrays().items()}
    dy = torch.randn(inp.u.shape, generator=torch.Generator().manual_seed(1)).to(dev).to(torch.bfloat16)

    kw = dict(D=g.get("Dskip"), dt_bias=g.get("dt_bias"), z=g.get("z"), h0=g.get("h0"))
    y_buf = torch.empty(inp.u.shape, dtype=torch.bfloat16, device=dev)
    ck_buf = torch.empty((inp.seqlen // 16, inp.batch, inp.dim, inp.dstate), dtype=torch.float32, device=dev)

    def step():
        if not train:
            return mb.scan_bwd(g["u"], g["delta"], g["A"], g["B"], g["C"], dy, **kw)
        mb.scan_fwd(g["u"], g["delta"], g["A"], g["B"], g["C"], out=y_buf, ck=ck_buf, **kw)
        return mb.scan_bwd(g["u"], g["delta"], g["A"], g["B"], g["C"], dy, ck=ck_buf, **kw)

    extra_warmup = warm_up(step, args.warmup)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        grads = step()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    E = inp.batch * inp.dim * inp.seqlen
    nbytes = bwd_bytes(inp)
    gbs = nbytes / (ms * 1e-3) / 1e9
    gel = E / (ms * 1e-3) / 1e9
    peak = TRAIN_ALU_PEAK_GELEMS if train else BWD_ALU_PEAK_GELEMS
    what = "forward + backward (training pair)" if train else "backward"
    line = {
        "metric": f"selective-scan {what}: B·L·D elems/s ({args.workload})",
        "value": round(E / (ms * 1e-3), 1), "unit": "elems/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "warmup_extra_steps": extra_warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "mode": "train" if train else "bwd",
                   **{k: v for k, v in WORKLOADS[args.workload].items()},
                   "dy_dtype": "bf16", "grad_dtype": "bf16 (activations), f32 (parameters, dB, dC)",
                   "parallelism": "single GPU"},
        # the whole call (checkpoint pass, backward, two reductions) against the
        # backward's ALU minimum; its HBM side for comparison
        "roofline": {"bound": "alu", "achieved": round(gel, 2), "peak": round(peak, 1),
                     "unit": "Gelem/s", "frac": round(gel / peak, 4), "traffic": None,
                     "scope": "whole step: every kernel of the call(s)", "hbm_gbs": round(gbs, 1),
                     "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": nbytes},
    }
    if not args.no_cpu_baseline:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from parity import rel_err

        orc = oracle.default()
        import dataclasses
        nb = 1                                      # a bounded sample: the first batch element
        cut = lambda a: None if a is None else np.ascontiguousarray(a[:nb])
        sub = dataclasses.replace(inp, batch=nb, u=cut(inp.u), delta=cut(inp.delta), z=cut(inp.z), B=cut(inp.B),
                                  C=cut(inp.C), h0=cut(inp.h0))
        dy_bits = dy[:nb].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        t0 = time.perf_counter()
        if train:                                   # the oracle's forward is part of the pair
            orc.scan_fwd(sub.u, sub.delta, sub.A, sub.B, sub.C, z=sub.z, Dskip=sub.Dskip, dt_bias=sub.dt_bias,
                         h0=sub.h0, dtype=sub.dtype)
        ref = orc.scan_bwd(sub.u, sub.delta, sub.A, sub.B, sub.C, dy_bits, z=sub.z, Dskip=sub.Dskip,
                           dt_bias=sub.dt_bias, h0=sub.h0, dtype=sub.dtype)
        elapsed = time.perf_counter() - t0
        Es = sub.batch * sub.dim * sub.seqlen
        err = max(rel_err(grads["du"][:nb].float().cpu().numpy(), ref["du"]),
                  rel_err(grads["dB"][:nb].cpu().numpy(), ref["dB"]))
        ok = err <= 1e-4 + 2.0 ** -8
        line["cpu_baseline"] = {"value": round(Es / elapsed, 1), "unit": "elems/s", "cores": orc.max_threads(),
                                "kind": "oracle", "cpu_model": cpu_model(),
                                "sample": f"batch element 0: {sub.dim} rows of L={sub.seqlen}, fp64, {elapsed:.1f} s"}
        line["parity"] = {"du_dB_rel_err_vs_oracle": err, "ok": bool(ok)}
        if not ok:
            print(json.dumps(line))
            print("parity gate failed: GPU output disagrees with the oracle", file=sys.stderr)
            sys.exit(1)
    print(json.dumps(line))


def bench_rank(args):
    """One mb_verify_rank per step: the top-3 check (Table 6) of 16 drafted bytes per
    prompt over fp32 256-way byte logits, batch 32 (the verify workload)."""
    import torch

    import paper_2401_13660_amd as mb

    B, n, V, beta = 32, 16, 256, 3
    rng = np.random.default_rng(0)
    lg = rng.standard_normal((B, n, V)).astype(np.float32)
    order = np.argsort(-lg.astype(np.float64), axis=2, kind="stable")
    pick = np.minimum(rng.geometric(0.5, (B, n)) - 1, V - 1)
    draft = np.take_along_axis(order, pick[..., None], axis=2)[..., 0].astype(np.int32)
    dev = torch.device("cuda:0")
    lg_d, dr_d = torch.from_numpy(lg).to(dev), torch.from_numpy(draft).to(dev)

    def step():
        return mb.verify_rank(lg_d, dr_d, beta, return_ranks=True)

    extra_warmup = warm_up(step, args.warmup)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        acc, last, ranks = step()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    nbytes = lg.nbytes + draft.nbytes + draft.nbytes + 2 * B * 4
    gbs = nbytes / (ms * 1e-3) / 1e9
    line = {
        "metric": "top-beta verify check: drafted bytes checked per second (batch 32, 16 bytes, 256-way)",
        "value": round(B * n / (ms * 1e-3), 1), "unit": "bytes/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "warmup_extra_steps": extra_warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "verify_rank_b32_n16_v256", "mode": "rank", "batch": B, "ndraft": n,
                   "vocab": V, "beta": beta, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "algorithmic_bytes": nbytes,
                     "note": "0.5 MB per call: launch- and latency-bound, not bandwidth-bound"},
    }
    if not args.no_cpu_baseline:
        from oracle import verify_rank as VR
        t0 = time.perf_counter()
        r_ref = VR.ranks(lg, draft)
        a_ref = VR.accepted(r_ref, beta)
        elapsed = time.perf_counter() - t0
        ok = np.array_equal(ranks.cpu().numpy(), r_ref) and np.array_equal(acc.cpu().numpy(), a_ref)
        line["cpu_baseline"] = {"value": round(B * n / elapsed, 1), "unit": "bytes/s", "cores": 1,
                                "kind": "oracle", "cpu_model": cpu_model(),
                                "sample": f"the whole check, numpy, {elapsed * 1e3:.1f} ms"}
        line["parity"] = {"ranks_and_accepted_equal": bool(ok), "ok": bool(ok)}
        if not ok:
            print(json.dumps(line))
            print("parity gate failed: GPU output disagrees with the oracle", file=sys.stderr)
            sys.exit(1)
    print(json.dumps(line))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=["fwd", "step", "conv", "rank", "bwd", "train"], default="fwd",
                    help="fwd: one mb_scan_fwd per step; step: seqlen successive mb_scan_step calls per step "
                         "(the recurrent-generation form of the same workload); conv: one mb_conv1d_fwd "
                         "(the causal convolution + Swish in front of the scan, k = 4, bf16 out); rank: one "
                         "mb_verify_rank (top-3 check of 16 drafted bytes over 256-way logits, batch 32); "
                         "bwd: one mb_scan_bwd (bf16 dy and activation gradients, fp32 parameter gradients); "
                         "train: one mb_scan_fwd_ckpt (bf16 y) and one mb_scan_bwd from its checkpoints")
    ap.add_argument("--out-dtype", choices=["f32", "bf16"], default="f32",
                    help="fwd: y in fp32 (the headline) or rounded to bf16 (8 instead of 10 bytes per element)")
    ap.add_argument("--graph", action="store_true",
                    help="fwd / step modes: capture one step in a HIP graph and time its replays")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the scan, run a plain device copy of MIB MiB (reference for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: there is no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n,
                          "launches": args.warmup + args.steps}))
        return

    import paper_2401_13660_amd as mb
    from paper_2401_13660_amd.inputs import WORKLOADS, workload

    if args.mode == "conv":
        return bench_conv(args)
    if args.mode == "rank":
        return bench_rank(args)
    if args.mode in ("bwd", "train"):
        return bench_bwd(args, train=args.mode == "train")

    inp = workload(args.workload, seed=0)
    dev = torch.device("cuda:0")

    def t(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    want_h_last = inp.h0 is not None or args.workload == "mambabyte1p6b_L65536"
    g = {k: t(v) for k, v in inp.arrays().items()}
    out_bf16 = args.mode == "fwd" and args.out_dtype == "bf16"
    y = torch.empty((inp.batch, inp.dim, inp.seqlen), dtype=torch.bfloat16 if out_bf16 else torch.float32,
                    device=dev)
    h_last = torch.empty((inp.batch, inp.dim, inp.dstate), dtype=torch.float32, device=dev) if want_h_last else None

    if args.mode == "fwd":
        def step():
            mb.scan_fwd(g["u"], g["delta"], g["A"], g["B"], g["C"], D=g.get("Dskip"), dt_bias=g.get("dt_bias"),
                        z=g.get("z"), h0=g.get("h0"), out=y, h_last=h_last)
    else:
        # per-byte slices made once, outside the timed region
        cols = [{k: (v[..., i].contiguous() if k in ("u", "delta", "z", "B", "C") else None)
                 for k, v in g.items()} for i in range(inp.seqlen)]
        state = g["h0"].clone() if g.get("h0") is not None else torch.zeros(
            (inp.batch, inp.dim, inp.dstate), dtype=torch.float32, device=dev)
        ycols = [torch.empty((inp.batch, inp.dim), dtype=torch.float32, device=dev) for _ in range(inp.seqlen)]

        def step():
            for i, c in enumerate(cols):
                mb.scan_step(state, c["u"], c["delta"], g["A"], c["B"], c["C"], D=g.get("Dskip"),
                             dt_bias=g.get("dt_bias"), z_t=c.get("z"), out=ycols[i])

    extra_warmup = warm_up(step, args.warmup)
    if args.graph:
        # one step captured once (warm-up on a side stream first), then replayed:
        # the per-call host work of the binding leaves the timed region
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run = graph.replay
    else:
        run = step
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    # per-launch device times (median, min), and for a cache-resident workload the
    # same after a 512 MB scrub write before every launch (inputs no longer in the
    # 256 MB Infinity Cache)
    pl = per_launch_ms(run, args.steps)
    per_launch = {"median": round(pl[len(pl) // 2], 5), "min": round(pl[0], 5)}
    if inp.batch * inp.dim * inp.seqlen * 10 < (256 << 20):
        scrub = torch.empty(512 << 18, dtype=torch.float32, device=dev)
        pf = per_launch_ms(run, args.steps, flush=lambda: scrub.fill_(1.0))
        per_launch["flushed_median"] = round(pf[len(pf) // 2], 5)
        per_launch["flushed_min"] = round(pf[0], 5)
        del scrub

    copy_gbs = copy_bandwidth_gbs(dev)
    E = inp.batch * inp.dim * inp.seqlen
    nbytes = algorithmic_bytes(inp, 2 if out_bf16 else 4, want_h_last)
    if args.mode == "step":
        nbytes = step_bytes(inp)
    gbs = nbytes / (ms * 1e-3) / 1e9
    traffic = None if out_bf16 else measured_traffic(args.workload)   # the record is of the fp32-output kernel

    line = {
        "metric": METRIC, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "warmup_extra_steps": extra_warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "mode": args.mode, "arithmetic": "f32",
                   **{k: v for k, v in WORKLOADS[args.workload].items()},
                   "gated": inp.z is not None, "h0": inp.h0 is not None, "h_last": want_h_last,
                   "out_dtype": "bf16" if out_bf16 else "f32", "parallelism": "single GPU",
                   "hip_graph": bool(args.graph)},
        "elems_per_s": round(E / (ms * 1e-3), 1),
        "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
        "ms_per_launch": per_launch,
        "copy_gbs": round(copy_gbs, 1), "frac_of_copy": round(gbs / copy_gbs, 4),
        # algorithmic bytes per step over the step's event-timed duration on the
        # launch stream (every kernel of the step: one scan launch, or the segment
        # pre-pass and the scan)
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic, "algorithmic_bytes": nbytes,
                     "scope": "whole step (all kernels of one call)"},
        # secondary: the same step against the issue model (VALU 4.1, transcendental
        # 8.6 SIMD-cycles per wave64 instruction; 76 + 20 per element; 2.4 GHz)
        "alu_model": {"achieved": round(E / (ms * 1e-3) / 1e9, 2), "peak": round(ALU_PEAK_GELEMS, 1),
                      "unit": "Gelem/s", "frac": round(E / (ms * 1e-3) / 1e9 / ALU_PEAK_GELEMS, 4)},
    }
    if args.mode == "step":
        # one-byte steps are bound by moving the state: report against HBM
        line["roofline"] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                            "note": "one HIP graph of the per-byte calls" if args.graph
                            else "includes host launch gaps between the per-byte calls"}
    if not args.no_cpu_baseline:
        if args.mode == "fwd":
            cb = cpu_baseline(inp, y, h_last)
            what = f"whole workload: {inp.batch} x {inp.dim} rows of L={inp.seqlen}, fp64"
        else:
            # the timed runs advanced the state many times: run the 16 steps once more
            # from h0 for the parity check
            state.copy_(g["h0"]) if g.get("h0") is not None else state.zero_()
            step()
            torch.cuda.synchronize()
            cb = cpu_baseline_steps(inp, ycols, state)
            what = f"{inp.seqlen} one-byte steps of {inp.batch} x {inp.dim} rows, fp64"
        line["cpu_baseline"] = {
            "value": round(cb["elems_per_s"] * nbytes / E / 1e9, 3), "unit": "GB/s",
            "elems_per_s": round(cb["elems_per_s"], 1), "cores": cb["threads"], "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{what}, best of {CPU_REPEATS}: {cb['elapsed']:.3f} s "
                      f"(runs {', '.join(f'{r:.3f}' for r in cb['runs'])} s)",
            "gpu_over_oracle": round((E / (ms * 1e-3)) / cb["elems_per_s"], 1),
        }
        if "single_thread" in cb:
            st1 = cb["single_thread"]
            line["cpu_baseline"]["single_thread"] = {
                "elems_per_s": round(st1["elems_per_s"], 1), "cores": 1,
                "sample": f"{what}, one core, best of {CPU_REPEATS}: {st1['elapsed']:.4f} s"}
        line["parity"] = {"y_rel_err_vs_oracle": cb["y_err"], "h_rel_err_vs_oracle": cb["h_err"],
                          "ok": cb["parity_ok"]}
        if not cb["parity_ok"]:
            print(json.dumps(line))
            print("parity gate failed: GPU output disagrees with the oracle", file=sys.stderr)
            sys.exit(1)
    print(json.dumps(line))


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the KAN-layer forward hot path on one MI355X.

One step = the whole hot path over one batch of synthetic input of the
3-layer KAN MLP workload (784 -> 256 -> 256 -> 10, G = 10, cubic, grid [-1, 1],
batch 65536):
    kan_basis_eval(x)                      basis-only tensor of the input
    3 x kan_layer_forward                  fused basis + MFMA contraction + SiLU
Inputs and weights are resident in HBM before timing starts; every launch goes
through the C ABI onto torch's current stream.

Prints ONE JSON line: samples/s (value), Gbasis/s, the roofline of the
dominant kernel (its duration from HIP events around it in every timed step,
the other kernels' from an untimed pass with an event between consecutive
launches, all on the launch stream),
per-layer parity of the run's output against the float64 oracle, the same
step in the other dtype (bf16 and fp32 are both measured) and the float64
CPU oracle timed on a bounded row sample of the same step.

    python bench.py [--steps K] [--warmup W] [--dtype bf16|f32]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

WORKLOAD = "c5_mlp_784_256_256_10_g10"
METRIC = "KAN layer fwd samples/s + Gbasis/s; % of HBM / MFMA peak on MI355X"
# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}
# VALU peak in G lane-ops/s: MI355X's 256 CUs x 4 SIMDs x 32 fp32 lanes x
# 2.4 GHz = 78.6 T lane-ops/s, the published 157.3 TFLOP/s fp32 vector rate
# with an fma counted as one lane-op (two flops).  Two counts of the VALU work
# of one (row, input feature) are reported against it:
#  * the least the kernels do (the headline "alu" figure): of the G + 3 basis
#    columns at most four consecutive ones are nonzero, each 7 lane-ops in the
#    truncated power form (v 1, P and Q 2 clamped fmas, P^2, Q^2, Q^3 3, the
#    final fma 1); the coordinate and the interval 4 (fma, add, floor,
#    fraction); SiLU 4 (exp, fma, reciprocal, multiply); in bf16 2 packed
#    conversions;
#  * the dense count of the method (every one of the G + 3 values evaluated,
#    no span lookup): 10 lane-ops per basis value (coordinate, clamp and the
#    two-term form) plus the SiLU's 4.
PEAK_VALU_GOPS = 256 * 4 * 32 * 2.4
VALU_OPS_PER_FEATURE = {"bf16": 38.0, "f32": 36.0}
VALU_OPS_PER_VALUE_DENSE = 10.0


def parse():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--clock-warmup-s", type=float, default=2.0,
                   help="seconds of untimed steps run before the --warmup steps, so the timed "
                        "steps run at the clock of a continuous job rather than the ramp out "
                        "of idle")
    p.add_argument("--dtype", choices=["bf16", "f32"], default="bf16")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target wall time of the CPU oracle sample (three runs)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--configs", action="store_true",
                   help="only time the fused layer and the basis kernel on every configured "
                        "workload (one JSON line each, with the partition-of-unity error of "
                        "the grid-size sweep) and exit")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                   help="only run a plain device copy of BYTES bytes 10 times (HBM counter "
                        "calibration under rocprofv3) and exit")
    return p.parse_args()


def copy_calibration(nbytes: int) -> None:
    import torch
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "launches": 10}), flush=True)


def layer_roofline(dtype: str, batch: int, n_in: int, n_out: int, nb: int,
                   narrow: bool = False) -> dict:
    """Roofline of one fused layer: bound by the matrix cores (dense flops,
    all nb bases plus the SiLU column per input) unless generating its basis
    values (the least VALU work, four nonzero columns per input) takes longer
    at the VALU peak than the contraction at the MFMA peak (narrow outputs);
    then it is reported against the VALU.  A layer that runs on the
    vector-ALU kernel of narrow fp32 layers (`narrow`) is reported against the
    VALU with that kernel's least work: the basis generation plus one fma per
    output for each of the five nonzero columns (SiLU and four bases)."""
    flop = 2.0 * batch * n_out * n_in * (nb + 1)
    valu = VALU_OPS_PER_FEATURE[dtype] * batch * n_in
    if narrow:
        k = {"bound": "alu", "unit": "Gop/s", "peak": PEAK_VALU_GOPS,
             "algorithmic": (VALU_OPS_PER_FEATURE[dtype] + 5.0 * n_out) * batch * n_in / 1e9,
             "kernel": "vector ALU (narrow layer)"}
    elif valu / (PEAK_VALU_GOPS * 1e9) > flop / (PEAK_TFLOPS[dtype] * 1e12):
        k = {"bound": "alu", "unit": "Gop/s", "peak": PEAK_VALU_GOPS,
             "algorithmic": valu / 1e9}  # G lane-ops
    else:
        k = {"bound": "mfma", "unit": "TFLOP/s", "peak": PEAK_TFLOPS[dtype],
             "algorithmic": flop / 1e12}  # dense TFLOP
    k["valu_gops"] = valu / 1e9
    k["valu_gops_dense"] = (VALU_OPS_PER_VALUE_DENSE * nb + 4.0) * batch * n_in / 1e9
    return k


def planned_narrow(kb, dtype: str, G: int, lo: float, hi: float, batch: int, n_in: int,
                   n_out: int) -> bool:
    """Whether the library plans the vector-ALU kernel of narrow layers
    (kan_layer_plan's shape {0, 4, 4, 1}) for this layer and batch."""
    code = kb.KAN_BF16 if dtype == "bf16" else kb.KAN_F32
    st, plan = kb.kan_layer_plan(kb.make_grid(G, lo, hi), code, batch, n_in, n_out)
    kb.check(st)
    return plan[0] == 0


KERNEL_SOURCES = ["kan_layer_kernel.h", "kan_layer.hip", "kan_internal.h", "kan_device.h"]


def traffic_record(dtype: str, kernel: str, root: str = ROOT):
    """HBM bytes per launch of `kernel`, from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE, each scaled by its plain-copy
    calibration factor), or None when there is no record for this dtype and
    kernel or the kernel sources have changed since the counters were taken."""
    import hashlib

    path = os.path.join(root, "profiles", f"kan_mlp_c5_{dtype}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    lines = open(path).read().splitlines()
    if "traffic-record" not in lines:
        return None
    rec = {}
    for ln in lines[lines.index("traffic-record") + 1:]:
        if ":" not in ln:
            break
        k, v = ln.split(":", 1)
        rec[k.strip()] = v.strip()
    h = hashlib.md5()
    for f in KERNEL_SOURCES:
        with open(os.path.join(root, "paper_2609_01956_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if (rec.get("kernel_sources_md5") != h.hexdigest() or rec.get("dtype") != dtype
            or rec.get("kernel") != kernel):
        return None
    kib = (float(rec["fetch_kib"]) * float(rec["fetch_factor"]) +
           float(rec["write_kib"]) * float(rec["write_factor"]))
    return kib * 1024.0


def _time_us(fn, warmup: int = 5, reps: int = 20, warm_s: float = 0.0) -> float:
    """Median over `reps` launches of fn, each between two HIP events on
    torch's current stream, after `warm_s` seconds of untimed calls (bringing
    an idle GPU to its working clock) and `warmup` more (microseconds)."""
    import numpy as np
    import torch
    t_end = time.perf_counter() + warm_s
    while time.perf_counter() < t_end:
        fn()
        torch.cuda.synchronize()
    for _ in range(warmup):
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return float(np.median([e0.elapsed_time(e1) * 1e3 for e0, e1 in ev]))


def _graph_time_us(fn, check=None, calls: int = 20, reps: int = 15) -> tuple:
    """Per-call GPU time of fn with no host time between its kernels: `calls`
    calls captured in one graph (torch.cuda.graph on its capture stream), the
    graph replayed `reps` times, each replay between two HIP events on
    torch's current stream; the median replay over `calls` (microseconds).
    check() runs after every replay (outside the timed region); returns
    (us, all checks true)."""
    import numpy as np
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(3):
            fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(calls):
            fn()
    ok = True
    ts = []
    for i in range(reps + 3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        if i >= 3:
            ts.append(e0.elapsed_time(e1) * 1e3 / calls)
        if check is not None:
            ok = ok and bool(check())
    return float(np.median(ts)), ok


SMALL_BATCHES = (1, 64, 1024)


def small_batch_block(W) -> dict:
    """The MLP's three layers (the workload's weights, seeded uniform inputs
    on the grid interval) at small batches in both dtypes: per-call time of
    kan_layer_forward_packed with its workspace, where the contraction splits
    across workgroups (kan_layer_plan's plan[5] splits), and without it
    (unsplit), timed by graph replay.  Every replay's output is compared
    with an eager call's (bitwise: same kernels, same summation order)."""
    import numpy as np
    import torch

    from paper_2609_01956_amd import binding as kb
    from paper_2609_01956_amd import workloads as wl

    G, lo, hi = W["G"], W["lo"], W["hi"]
    rng = np.random.default_rng(17)
    out = {}
    for dtype in ("bf16", "f32"):
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        code = kb.KAN_BF16 if dtype == "bf16" else kb.KAN_F32
        prep = (lambda a: wl.round_to_bf16_f32(a)) if dtype == "bf16" else (lambda a: a)
        rows = {}
        for li, (C, Wb) in enumerate(W["layers"]):
            n_out, n_in = Wb.shape
            Ct = torch.from_numpy(prep(C)).to("cuda").to(tdt).contiguous()
            Wt = torch.from_numpy(prep(Wb)).to("cuda").to(tdt).contiguous()
            pk = kb.pack_layer(Ct, Wt, G, lo, hi)
            for B in SMALL_BATCHES:
                x = torch.from_numpy(rng.uniform(lo, hi, (B, n_in)).astype(np.float32))
                x = x.to("cuda").to(tdt).contiguous()
                st, plan = kb.kan_layer_plan(kb.make_grid(G, lo, hi), code, B, n_in, n_out)
                kb.check(st)
                st, nbytes = kb.kan_layer_forward_packed_workspace_bytes(
                    kb.make_grid(G, lo, hi), code, B, n_in, n_out)
                kb.check(st)
                ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")
                y = torch.empty((B, n_out), dtype=tdt, device="cuda")
                ref_split = kb.layer_forward_packed(x, pk, workspace=ws)
                ref_plain = kb.layer_forward_packed(x, pk, split=False)
                split_us, ok1 = _graph_time_us(
                    lambda: kb.layer_forward_packed(x, pk, out=y, workspace=ws),
                    check=lambda: torch.equal(y, ref_split))
                plain_us, ok2 = _graph_time_us(
                    lambda: kb.layer_forward_packed(x, pk, out=y, split=False),
                    check=lambda: torch.equal(y, ref_plain))
                rows[f"layer{li + 1}_{n_in}x{n_out}_b{B}"] = {
                    "splits": plan[5], "split_us": split_us, "unsplit_us": plain_us,
                    "replays_match_eager": ok1 and ok2}
        out[dtype] = rows
    return {"timing": "per call, 20 calls per graph replay, median of 15 replays",
            "layers": out}


# Seconds of untimed calls before each timing of the configs sweep (the
# inputs of the next workload are generated on the host in between).
CONFIG_WARM_S = 0.5


def configs_sweep(dtype: str) -> None:
    """Every configured workload, one JSON line each (each kernel the median of
    200 launches after 0.5 s of calls and 50 more): the fused layer (packed weights, per layer of the
    MLP) against its roofline, the basis-only kernel
    of its input, and for the grid-size sweep the partition-of-unity error of
    the basis kernel on the same x plus 2001 points spread over the grid and
    the span-sparse layer (kan_layer_forward_span, weight transposition
    included) beside the dense one."""
    import numpy as np
    import torch

    from paper_2609_01956_amd import binding as kb
    from paper_2609_01956_amd import workloads as wl

    kb.load_library()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    es = 2 if dtype == "bf16" else 4
    prep = (lambda a: wl.round_to_bf16_f32(a)) if dtype == "bf16" else (lambda a: a)
    for name in wl.WORKLOADS:
        W = wl.make_workload(name)
        G, lo, hi = W["G"], W["lo"], W["hi"]
        nb = G + 3
        x = torch.from_numpy(prep(W["x"])).to("cuda").to(tdt).contiguous()
        B, n_in0 = x.shape
        phi = torch.empty((B, n_in0, nb), dtype=tdt, device="cuda")
        us = _time_us(lambda: kb.basis(x, G, lo, hi, out=phi), 50, 200, CONFIG_WARM_S)
        line = {"workload": name, "dtype": dtype, "batch": B, "grid_size": G,
                "basis_eval": {"us": us, "gbasis_per_s": B * n_in0 * nb / us / 1e3,
                               "hbm_frac": B * n_in0 * (nb + 1) * es / us / 1e3 / PEAK_HBM_GBS}}
        if name.startswith("c4_"):
            xs = np.concatenate([W["x"].reshape(-1), np.linspace(lo, hi, 2001)]).astype(np.float32)
            pu = kb.basis(torch.from_numpy(xs).to("cuda"), G, lo, hi).double().sum(dim=1)
            line["pu_max_err"] = float((pu - 1.0).abs().max())
        h = x
        layers = []
        for C, Wb in W["layers"]:
            Ct = torch.from_numpy(prep(C)).to("cuda").to(tdt).contiguous()
            Wt = torch.from_numpy(prep(Wb)).to("cuda").to(tdt).contiguous()
            pk = kb.pack_layer(Ct, Wt, G, lo, hi)
            out = torch.empty((B, C.shape[0]), dtype=tdt, device="cuda")
            lus = _time_us(lambda: kb.layer_forward_packed(h, pk, out=out), 50, 200,
                           CONFIG_WARM_S)
            k = layer_roofline(dtype, B, C.shape[1], C.shape[0], nb,
                               planned_narrow(kb, dtype, G, lo, hi, B, C.shape[1], C.shape[0]))
            k.pop("valu_gops")
            k.pop("valu_gops_dense")
            k.update(us=lus, samples_per_s=B / lus * 1e6, achieved=k["algorithmic"] / (lus * 1e-6))
            k["frac"] = k["achieved"] / k["peak"]
            layers.append({"in": C.shape[1], "out": C.shape[0], **k})
            h = out
        line["layers"] = layers
        if name in SPAN_GRIDS:
            (C, Wb), = W["layers"]
            Ct = torch.from_numpy(prep(C)).to("cuda").to(tdt).contiguous()
            Wt = torch.from_numpy(prep(Wb)).to("cuda").to(tdt).contiguous()
            n_out, n_in = Wb.shape
            st, nbytes = kb.kan_layer_forward_span_workspace_bytes(
                kb.make_grid(G, lo, hi), kb.KAN_BF16 if dtype == "bf16" else kb.KAN_F32, B,
                n_in, n_out)
            kb.check(st)
            ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
            y = torch.empty((B, n_out), dtype=tdt, device="cuda")
            sus = _time_us(lambda: kb.layer_forward_span(x, Ct, Wt, G, lo, hi, out=y, workspace=ws),
                           50, 200, CONFIG_WARM_S)
            line["span_sparse_layer"] = {
                "us": sus, "samples_per_s": B / sus * 1e6,
                "valu_frac": B * n_in * (5.0 * n_out + 38.0) / (sus * 1e-6) / 1e9 / PEAK_VALU_GOPS}
        print(json.dumps(line), flush=True)


def cpu_baseline(W, target_s: float):
    """The float64 oracle, untuned, on a row sample of the same step: the
    basis of the input and the 3-layer forward of its first rows.  A 64-row
    warm-up, then a sizing run of about a second (the warm-up's time is
    mostly fixed cost), size the sample so that one run takes about
    target_s / 3; three runs follow and their median is reported (cost is
    linear in rows)."""
    import numpy as np
    import oracle

    oracle.build()
    threads = oracle.num_threads()
    G = W["G"]
    x = W["x"]
    layers = W["layers"]

    def step(rows):
        xs = x[:rows].astype(np.float64)
        oracle.basis_tp(xs, G)
        oracle.mlp(xs, layers, G)

    t0 = time.perf_counter()
    step(64)
    dt64 = time.perf_counter() - t0
    n1 = int(max(64, min(x.shape[0], 64 * 1.0 / max(dt64, 1e-6))))
    t0 = time.perf_counter()
    step(n1)
    dt1 = time.perf_counter() - t0
    rows = int(max(64, min(x.shape[0], n1 * (target_s / 3.0) / max(dt1, 1e-6))))
    runs = []
    for _ in range(3):
        t0 = time.perf_counter()
        step(rows)
        runs.append(time.perf_counter() - t0)
    dt = float(np.median(runs))
    return {"value": rows / dt, "unit": "samples/s", "cores": threads, "kind": "oracle",
            "sample": f"first {rows} rows of the {x.shape[0]}-row batch: float64 basis of the "
                      f"input + 3-layer forward; median of 3 runs ({', '.join(f'{r:.2f}' for r in runs)} s) "
                      f"after a 64-row warm-up and a {n1}-row sizing run, on {threads} threads"}


def measure_step(dtype: str, W, steps: int, warmup: int, clock_warmup_s: float = 0.0) -> dict:
    """Times `steps` steps of the hot path in `dtype` (after `clock_warmup_s`
    seconds of untimed steps, then `warmup` more).  Per-kernel durations come
    from `steps` untimed steps with a HIP event between consecutive kernels on
    torch's current stream (the stream every kernel is launched on); the
    timed steps then carry only a pair of events around the dominant kernel,
    whose duration (the roofline's) is taken from them.  Returns the step
    time, per-kernel averages and rooflines, and the outputs of the last
    step."""
    import numpy as np
    import torch

    from paper_2609_01956_amd import binding as kb
    from paper_2609_01956_amd import workloads as wl

    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    es = 2 if dtype == "bf16" else 4
    G, lo, hi = W["G"], W["lo"], W["hi"]
    nb = G + 3
    x_np = W["x"]
    B, n_in0 = x_np.shape
    prep = (lambda a: wl.round_to_bf16_f32(a)) if dtype == "bf16" else (lambda a: a)
    x = torch.from_numpy(prep(x_np)).to(dev).to(tdt).contiguous()
    layers = [(torch.from_numpy(prep(C)).to(dev).to(tdt).contiguous(),
               torch.from_numpy(prep(Wb)).to(dev).to(tdt).contiguous()) for C, Wb in W["layers"]]
    shapes = [(C.shape[1], C.shape[0]) for C, _ in layers]  # (in, out)
    phi = torch.empty((B, n_in0, nb), dtype=tdt, device=dev)
    hs = [torch.empty((B, o), dtype=tdt, device=dev) for _, o in shapes]

    packs = [kb.pack_layer(C, Wb, G, lo, hi) for C, Wb in layers]
    names = ["basis_eval"]
    for i, (i_, o) in enumerate(shapes):
        names += [f"pack{i + 1}_{i_}x{o}", f"layer{i + 1}_{i_}x{o}"]

    # The step's launches in order: kan_basis_eval of the input, then per
    # layer kan_layer_pack + kan_layer_forward_packed (the weights are
    # re-packed every step).
    launches = [lambda: kb.basis(x, G, lo, hi, out=phi)]
    h = x
    for (C, Wb), pk, out in zip(layers, packs, hs):
        launches.append(lambda C=C, Wb=Wb, pk=pk: kb.pack_layer(C, Wb, G, lo, hi, out=pk))
        launches.append(lambda h=h, pk=pk, out=out: kb.layer_forward_packed(h, pk, out=out))
        h = out

    def step(events=None, only=None):
        """One step.  events: with only=None an event before every launch and
        one after the last; else a pair around launch `only`."""
        for k, f in enumerate(launches):
            if events is not None:
                if only is None:
                    events[k].record()
                elif k == only:
                    events[0].record()
            f()
            if events is not None and k == only:
                events[1].record()
        if events is not None and only is None:
            events[len(launches)].record()

    # Out of idle the GPU takes tens of milliseconds to reach its working
    # clock: with 5 warm-up steps alone the bf16 step measured 0.744 ms, after
    # 0.5, 2 or 5 s of continuous steps 0.662, 0.661 and 0.669 ms on the same
    # box.  A continuous job runs at the latter.
    t_end = time.perf_counter() + clock_warmup_s
    while time.perf_counter() < t_end:
        step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()

    # Per-kernel durations: `steps` untimed steps with an event between
    # consecutive launches (each event costs the step a few us, so the timed
    # region below brackets only the dominant kernel).
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
          for _ in range(steps)]
    for k in range(steps):
        step(ev[k])
    torch.cuda.synchronize()
    per_kernel_ms = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev]))
                     for i in range(len(names))]
    dom_i = int(np.argmax(per_kernel_ms))

    # Timed region: exactly `steps` steps, bracketed by synchronisations, with
    # a pair of events around the dominant kernel in every step.
    evd = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step(evd[k], only=dom_i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / steps
    per_kernel_ms[dom_i] = float(np.mean([e[0].elapsed_time(e[1]) for e in evd]))

    # Algorithmic work per launch.
    basis_values = B * n_in0 * nb
    kern = {}
    kern["basis_eval"] = {
        "bound": "hbm", "unit": "GB/s", "peak": PEAK_HBM_GBS,
        "algorithmic": (B * n_in0 * es + basis_values * es) / 1e9,  # GB: read x, write phi
    }
    for li, (i_, o) in enumerate(shapes):
        # pack: read coef + base_w, write the packed buffer
        kern[names[1 + 2 * li]] = {
            "bound": "hbm", "unit": "GB/s", "peak": PEAK_HBM_GBS,
            "algorithmic": (o * i_ * (nb + 1) * es + packs[li].nbytes) / 1e9}
        kern[names[2 + 2 * li]] = layer_roofline(dtype, B, i_, o, nb,
                                                 planned_narrow(kb, dtype, G, lo, hi, B, i_, o))
        # HBM bytes the layer must move: x, the packed weights once, y
        kern[names[2 + 2 * li]]["algorithmic_bytes"] = (B * (i_ + o) * es + packs[li].nbytes)
    for name, ms in zip(names, per_kernel_ms):
        k = kern[name]
        k["avg_us"] = ms * 1e3
        k["achieved"] = k["algorithmic"] / (ms * 1e-3)
        k["frac"] = k["achieved"] / k["peak"]
        if "valu_gops" in k:  # the basis generation's share of the VALU peak
            k["valu_frac"] = k.pop("valu_gops") / (ms * 1e-3) / PEAK_VALU_GOPS
            k["valu_frac_dense_count"] = k.pop("valu_gops_dense") / (ms * 1e-3) / PEAK_VALU_GOPS
    dom = names[dom_i]
    dk = kern[dom]
    traffic = traffic_record(dtype, dom)
    roof = {"kernel": dom, "bound": dk["bound"], "achieved": dk["achieved"], "peak": dk["peak"],
            "unit": dk["unit"], "frac": dk["frac"], "traffic": traffic}
    if traffic is not None and "algorithmic_bytes" in dk:
        # HBM bytes measured per launch over the bytes the layer must move
        roof["traffic_over_algorithmic_bytes"] = traffic / dk["algorithmic_bytes"]
    basis_total = B * nb * (n_in0 + sum(i_ for i_, _ in shapes))
    return {"ms_per_step": ms_per_step, "samples_per_s": B / (ms_per_step * 1e-3),
            "gbasis_per_s": basis_total / (ms_per_step * 1e-3) / 1e9, "roofline": roof,
            "kernels": kern, "shapes": shapes, "x": x, "outs": hs, "prep": prep}


def backward_block(dtype: str, W, r: dict, reps: int = 10) -> dict:
    """kan_layer_backward of each MLP layer (dx, dcoef and dbase_w) on that
    layer's own input from the timed forward and a seeded N(0, 1) dy, timed
    with HIP events on torch's current stream.  Work: the two contractions
    dx = dy W^T and [dcoef dbase_w] = A^T dy over all G + 4 columns of the
    layer (A: SiLU and basis values of x), 2 B out in (G + 4) dense flops
    each, against the MFMA peak of the dtype."""
    import torch

    from paper_2609_01956_amd import binding as kb

    G, lo, hi = W["G"], W["lo"], W["hi"]
    nb = G + 3
    tdt = r["x"].dtype
    prep = r["prep"]
    ins = [r["x"]] + r["outs"][:-1]
    gen = torch.Generator(device=r["x"].device).manual_seed(11)
    layers = {}
    total = 0.0
    for li, ((C, Wb), h) in enumerate(zip(W["layers"], ins)):
        Ct = torch.from_numpy(prep(C)).to(h.device).to(tdt).contiguous()
        Wt = torch.from_numpy(prep(Wb)).to(h.device).to(tdt).contiguous()
        B, n_in = h.shape
        n_out = C.shape[0]
        dy = torch.randn((B, n_out), generator=gen, device=h.device).to(tdt)
        st, nbytes = kb.kan_layer_backward_workspace_bytes(
            kb.make_grid(G, lo, hi), kb.KAN_BF16 if dtype == "bf16" else kb.KAN_F32, B, n_in,
            n_out)
        kb.check(st)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=h.device)
        outs = (torch.empty_like(h), torch.empty_like(Ct), torch.empty_like(Wt))
        us = _time_us(lambda: kb.layer_backward(h, Ct, Wt, dy, G, lo, hi, workspace=ws, out=outs),
                      warmup=2, reps=reps)
        flop = 2 * 2.0 * B * n_out * n_in * (nb + 1)
        layers[f"layer{li + 1}_{n_in}x{n_out}"] = {
            "avg_us": us, "bound": "mfma", "unit": "TFLOP/s", "peak": PEAK_TFLOPS[dtype],
            "achieved": flop / (us * 1e-6) / 1e12,
            "frac": flop / (us * 1e-6) / 1e12 / PEAK_TFLOPS[dtype]}
        total += us
    return {"ms_all_layers": total * 1e-3, "layers": layers,
            "step": "kan_layer_backward (dx, dcoef, dbase_w) per layer"}


SPAN_GRIDS = ("c4_layer_128x128_g50", "c4_layer_128x128_g100", "c4_layer_128x128_g200")


def grid_sweep_block(dtype: str = "f32") -> dict:
    """The grid-size sweep layer (batch 8192, 128 -> 128, G = 50, 100, 200)
    through both forward paths: the dense fused layer (kan_layer_forward_packed,
    MFMA over all G + 4 columns) and the span-sparse one (kan_layer_forward_span,
    its weight transposition included: only the k + 1 nonzero bases and SiLU
    per input, on the vector ALUs), with the partition-of-unity error of the
    basis kernel on the same inputs.  Dense work against the MFMA peak; the
    span path's multiply-adds (B in out (k + 2)) and its least basis work (38
    lane-ops per input) against the VALU peak."""
    import numpy as np
    import torch

    from paper_2609_01956_amd import binding as kb
    from paper_2609_01956_amd import workloads as wl

    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    prep = (lambda a: wl.round_to_bf16_f32(a)) if dtype == "bf16" else (lambda a: a)
    out = {}
    for name in SPAN_GRIDS:
        W = wl.make_workload(name)
        G, lo, hi = W["G"], W["lo"], W["hi"]
        (C, Wb), = W["layers"]
        x = torch.from_numpy(prep(W["x"])).to("cuda").to(tdt).contiguous()
        Ct = torch.from_numpy(prep(C)).to("cuda").to(tdt).contiguous()
        Wt = torch.from_numpy(prep(Wb)).to("cuda").to(tdt).contiguous()
        B, n_in = x.shape
        n_out = C.shape[0]
        y = torch.empty((B, n_out), dtype=tdt, device="cuda")
        pk = kb.pack_layer(Ct, Wt, G, lo, hi)
        dense = _time_us(lambda: kb.layer_forward_packed(x, pk, out=y))
        st, nbytes = kb.kan_layer_forward_span_workspace_bytes(
            kb.make_grid(G, lo, hi), kb.KAN_BF16 if dtype == "bf16" else kb.KAN_F32, B, n_in,
            n_out)
        kb.check(st)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        span = _time_us(lambda: kb.layer_forward_span(x, Ct, Wt, G, lo, hi, out=y, workspace=ws))
        xs = torch.from_numpy(np.concatenate([W["x"].reshape(-1),
                                              np.linspace(lo, hi, 2001)]).astype(np.float32))
        pu = kb.basis(xs.to("cuda"), G, lo, hi).double().sum(dim=1)
        flop = 2.0 * B * n_out * n_in * (G + 4)
        lane_ops = B * n_in * (5.0 * n_out + 38.0)
        out[name] = {"grid_size": G, "dense_us": dense, "span_us": span,
                     "samples_per_s": B / (min(dense, span) * 1e-6),
                     "dense_mfma_frac": flop / (dense * 1e-6) / 1e12 / PEAK_TFLOPS[dtype],
                     "span_valu_frac": lane_ops / (span * 1e-6) / 1e9 / PEAK_VALU_GOPS,
                     "pu_max_err": float((pu - 1.0).abs().max())}
    return {"dtype": dtype, "grids": out}


def cdb_context() -> dict:
    """The truncated-power basis kernel against our Cox-de Boor kernel (the
    recursion over every knot interval that the paper measures against), fp32
    storage, on the inputs of: the MLP's first layer (65536 x 784, G = 10), the
    paper's basis-timing layer (256 x 784, G = 5), and the grid-size sweep's
    largest grid (8192 x 128, G = 200).  Context, not a target: both kernels
    write the same basis tensor, so on large inputs both are bound by its HBM
    write and the ratio stays near 1."""
    import numpy as np
    import torch

    from paper_2609_01956_amd import binding as kb

    out = {}
    rng = np.random.default_rng(7)
    for name, (B, n, G) in {"mlp_layer1_65536x784_g10": (65536, 784, 10),
                            "basis_timing_layer_256x784_g5": (256, 784, 5),
                            "grid_sweep_8192x128_g200": (8192, 128, 200)}.items():
        x = torch.from_numpy(rng.uniform(-1, 1, (B, n)).astype(np.float32)).to("cuda")
        phi = torch.empty((B, n, G + 3), dtype=torch.float32, device="cuda")
        tp = _time_us(lambda: kb.basis(x, G, out=phi))
        cdb = _time_us(lambda: kb.basis(x, G, out=phi, method="cdb"))
        out[name] = {"tp_us": tp, "cdb_us": cdb, "cdb_over_tp": cdb / tp,
                     "tp_gbasis_per_s": B * n * (G + 3) / tp / 1e3}
    return out


def table1_context() -> dict:
    """The paper's forward-cost breakdown (Table 1: a 256 x 784 -> 64 layer,
    the basis materialised by the Cox-de Boor recursion, then the spline
    einsum and the SiLU branch) taken on MI355X, fp32, G = 5, as context: the
    basis tensor from our Cox-de Boor kernel (and from the truncated-power
    kernel), the two contractions by the vendor GEMM through torch (context
    only, not part of the library), and the library's fused layer, which
    never materialises the basis, on the same inputs.  Median of 200
    launches after 50, each between HIP events (host time of the call
    included where it exceeds the kernel's); the fused layer also per call
    under graph replay."""
    import numpy as np
    import torch
    import torch.nn.functional as F

    from paper_2609_01956_amd import binding as kb

    B, n_in, n_out, G = 256, 784, 64, 5
    rng = np.random.default_rng(9)
    x = torch.from_numpy(rng.uniform(-1, 1, (B, n_in)).astype(np.float32)).to("cuda")
    C = torch.from_numpy(rng.normal(0, 0.1, (n_out, n_in, G + 3)).astype(np.float32)).to("cuda")
    Wb = torch.from_numpy(rng.normal(0, 1 / np.sqrt(n_in), (n_out, n_in)).astype(np.float32)).to("cuda")
    phi = torch.empty((B, n_in, G + 3), dtype=torch.float32, device="cuda")
    Ct = C.reshape(n_out, -1).t().contiguous()
    Wt = Wb.t().contiguous()
    y = torch.empty((B, n_out), dtype=torch.float32, device="cuda")
    pk = kb.pack_layer(C, Wb, G)

    med = lambda fn: _time_us(fn, 50, 200)

    cdb = med(lambda: kb.basis(x, G, out=phi, method="cdb"))
    tp = med(lambda: kb.basis(x, G, out=phi))
    spline = med(lambda: torch.matmul(phi.view(B, -1), Ct))
    base = med(lambda: torch.matmul(F.silu(x), Wt))
    fused = med(lambda: kb.layer_forward_packed(x, pk, out=y))
    fused_graph, _ = _graph_time_us(lambda: kb.layer_forward_packed(x, pk, out=y))
    total = cdb + spline + base
    return {"layer": "256 x 784 -> 64, G = 5, fp32",
            "basis_cox_de_boor_us": cdb, "basis_truncated_power_us": tp,
            "spline_contraction_gemm_us": spline, "silu_branch_us": base,
            "unfused_total_us": total, "basis_share": cdb / total,
            "fused_layer_us": fused, "fused_layer_graph_replay_us": fused_graph,
            "paper_context": "Table 1: basis 91% of 1.58 ms on an Apple MPS GPU; Table 3: "
                             "2.8-3.5x forward latency of the truncated-power form over Cox-de "
                             "Boor on its own hardware"}


def layer_parity(dtype: str, W, r: dict, n_rows: int = 64) -> dict:
    """Per layer, the sampled rows of this run's GPU output against the plain
    float64 oracle (eq. kan_forward) fed the GPU's own input rows of that
    layer (rounded to bf16 in bf16 mode): normwise errors, gated at 1e-5
    (fp32) and 2e-2 (bf16).  End-to-end errors against the oracle's own chain
    (and, in bf16, against the chain that also rounds the contraction
    operands to bf16) are information only."""
    import numpy as np
    import torch

    import oracle

    G = W["G"]
    prep = r["prep"]
    B = W["x"].shape[0]
    rows = np.arange(0, B, max(1, B // n_rows))[:n_rows]
    ridx = torch.from_numpy(rows).to(r["x"].device)
    host = lambda t: t[ridx].float().cpu().numpy().astype(np.float64)
    ins = [r["x"]] + r["outs"][:-1]
    bf = dtype == "bf16"
    per_layer = []
    for (C, Wb), h_in, h_out in zip(W["layers"], ins, r["outs"]):
        ref = oracle.layer(host(h_in), prep(C), prep(Wb), G)
        if bf:
            ref = oracle.round_bf16(ref)
        got = host(h_out)
        per_layer.append(float(np.abs(got - ref).max() / np.abs(ref).max()))
    tol = 2e-2 if bf else 1e-5
    layers = [(prep(C), prep(Wb)) for C, Wb in W["layers"]]
    got = host(r["outs"][-1])
    chain = oracle.mlp(prep(W["x"])[rows], layers, G, bf16=bf)
    out = {"rows": int(rows.size), "per_layer_normwise": per_layer, "tolerance": tol,
           "ok": bool(max(per_layer) <= tol),
           "e2e_vs_oracle_chain_info": float(np.abs(got - chain).max() / np.abs(chain).max())}
    if bf:
        ops = oracle.mlp(prep(W["x"])[rows], layers, G, bf16=True, bf16_operands=True)
        out["e2e_vs_bf16_operand_chain_info"] = float(np.abs(got - ops).max() / np.abs(ops).max())
    return out


def main() -> int:
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not run (rows are "
              "independent: the batch would shard across GPUs with the weights replicated "
              "and no communication inside a layer)", file=sys.stderr)
        return 2
    import torch

    from paper_2609_01956_amd import binding as kb
    from paper_2609_01956_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return 0
    if args.configs:
        configs_sweep(args.dtype)
        return 0
    kb.load_library()
    W = wl.make_workload(WORKLOAD)
    other = "f32" if args.dtype == "bf16" else "bf16"
    res = {}
    for dt in (args.dtype, other):
        res[dt] = measure_step(dt, W, args.steps, args.warmup, args.clock_warmup_s)
        try:
            res[dt]["parity"] = layer_parity(dt, W, res[dt])
        except Exception as e:  # the oracle is optional for timing
            res[dt]["parity"] = f"unavailable: {e}"
    r = res[args.dtype]
    B, n_in0 = W["x"].shape
    G = W["G"]
    line = {
        "metric": METRIC,
        "value": r["samples_per_s"],
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "clock_warmup_s": args.clock_warmup_s,
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "global_batch": B,
                   "layers": [n_in0] + [o for _, o in r["shapes"]],
                   "grid_size": G, "spline_order": 3, "grid": [W["lo"], W["hi"]],
                   "step": "kan_basis_eval(x) + 3 x (kan_layer_pack + kan_layer_forward_packed)"},
        "gbasis_per_s": r["gbasis_per_s"],
        "roofline": r["roofline"],
        "kernel_timing": ("dominant kernel: HIP events around it in every timed step; the "
                          "others: an untimed pass of as many steps with an event between "
                          "consecutive launches"),
        "kernels": r["kernels"],
        "parity": r["parity"],
    }
    o = res[other]
    line[other] = {"ms_per_step": o["ms_per_step"], "samples_per_s": o["samples_per_s"],
                   "gbasis_per_s": o["gbasis_per_s"], "roofline": o["roofline"],
                   "kernels": {n: {k: v for k, v in kk.items() if k in
                                   ("avg_us", "frac", "bound", "achieved", "unit", "valu_frac",
                                    "valu_frac_dense_count")}
                               for n, kk in o["kernels"].items()},
                   "parity": o["parity"]}
    # The blocks below add to the line; a failure in one is recorded in its
    # place rather than losing the measured step.
    def optional(fn, *a):
        try:
            return fn(*a)
        except Exception as e:  # noqa: BLE001 (reported in the line)
            return {"error": f"{type(e).__name__}: {e}"}

    line["backward"] = optional(backward_block, args.dtype, W, r)
    line[other]["backward"] = optional(backward_block, other, W, o)
    line["grid_sweep"] = optional(grid_sweep_block, "f32")
    line["cox_de_boor_context"] = optional(cdb_context)
    line["table1_cost_breakdown_context"] = optional(table1_context)
    line["small_batch"] = optional(small_batch_block, W)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = optional(cpu_baseline, W, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

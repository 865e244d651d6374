#!/usr/bin/env python3
"""Benchmark of the FLARE++ mixer forward on one MI355X (gfx950).

One step = one complete mixer forward (project; query synthesis, encode and
decode routing calls; merge) over one batch of synthetic inputs already
resident in HBM.  Default workload: the large 3D-mesh layer, the largest
configuration that fits one GPU (B=1, N=2^20, C=128, H=8, D=16, M=512, bf16
storage, fp32 accumulation).

Prints one JSON line with tokens/s, the per-stage device times measured with
HIP events, the roofline of the dominant kernel and the float64 oracle timed
on the host cores as a CPU baseline.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
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

METRIC = "FLARE++ mixer fwd tokens/sec (B·N/s) at 1 GPU + % bf16 MFMA peak"

# MI355X published peaks
PEAK_MFMA_BF16_TFLOPS = 2500.0
PEAK_MFMA_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
# v_exp_f32 issue rate: 256 CUs x 2.4 GHz x 32 lanes per clock per CU, half
# the fp32 FMA rate (a wave64 v_exp_f32 occupies a 16-lane SIMD for 8 clocks)
PEAK_EXP_TPS = 256 * 2.4e9 * 32 / 1e12  # Texp/s


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mesh3d")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-graph", action="store_true", help="launch every step eagerly")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-backward", action="store_true", help="skip the mixer-backward timing")
    ap.add_argument("--no-block", action="store_true", help="skip the pre-norm residual block timing")
    ap.add_argument("--no-train-pair", action="store_true",
                    help="skip the training forward + backward-from-saved timing")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum host seconds spent timing the oracle")
    ap.add_argument("--stage-reps", type=int, default=20,
                    help="back-to-back launches per stage when timing stages alone")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (for counter scaling)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this "
                         "script into profiles/traffic_<workload>.json and exit")
    ap.add_argument("--pmc-command", default="", help="the profiled command, recorded in the summary")
    return ap.parse_args(argv)


def stage_work(w, fused):
    """Algorithmic flops, HBM bytes and exponentials per launch of each stage.

    Flops: 4*T*M*C per routing call (scores and values over all heads) plus
    2*T*C*C for each C x C projection the stage owns (the fused decode's
    recompute of K is not counted).  Bytes: what the stage must move at its
    boundary (X read once, O written once, the route operands it produces);
    the split-key partials are not counted, they exist only because of the
    split."""
    T, C, M, H, D = w.B * w.N, w.C, w.M, w.H, w.D
    bs = 2 if w.dtype == "bf16" else 4
    route = 4.0 * T * M * C
    gemm = 2.0 * T * C * C
    exps = 1.0 * T * H * M
    prep = 10.0 * C * C * bs + 2.0 * H * M * D * bs
    comb = w.B * H * M * D * (4.0 + bs)
    zero = dict(flops=0.0, bytes=0.0, exps=0.0)
    if fused:  # the first encode call converts the weights (stage 1 is empty)
        return {
            "prep": zero,
            "project": zero,
            "call1_encode": dict(flops=route + 2 * gemm, bytes=T * C * bs, exps=exps),
            "call1_combine": dict(flops=0.0, bytes=comb, exps=0.0),
            "call2_encode": dict(flops=route + 2 * gemm, bytes=T * C * bs, exps=exps),
            "call2_combine": dict(flops=0.0, bytes=comb, exps=0.0),
            "call3_decode": dict(flops=route + gemm, bytes=2.0 * T * C * bs, exps=exps),
            "merge": zero,
        }
    return {
        "prep": dict(flops=0.0, bytes=prep, exps=0.0),
        "project": dict(flops=4 * gemm, bytes=5.0 * T * C * bs, exps=0.0),
        "call1_encode": dict(flops=route, bytes=2.0 * T * C * bs, exps=exps),
        "call1_combine": dict(flops=0.0, bytes=comb, exps=0.0),
        "call2_encode": dict(flops=route, bytes=2.0 * T * C * bs, exps=exps),
        "call2_combine": dict(flops=0.0, bytes=comb, exps=0.0),
        "call3_decode": dict(flops=route, bytes=2.0 * T * C * bs, exps=exps),
        "merge": dict(flops=gemm, bytes=2.0 * T * C * bs, exps=0.0),
    }


def roofline(work, ms, dtype):
    """Binding resource of one kernel under the roofline model and the
    achieved rate on it."""
    s = ms * 1e-3
    peak_mfma = PEAK_MFMA_BF16_TFLOPS if dtype == "bf16" else PEAK_MFMA_F32_TFLOPS
    ideal = {
        "mfma": work["flops"] / (peak_mfma * 1e12),
        "hbm": work["bytes"] / (PEAK_HBM_GBS * 1e9),
        "alu": work["exps"] / (PEAK_EXP_TPS * 1e12),
    }
    bound = max(ideal, key=ideal.get)
    if bound == "mfma":
        a, p, unit = work["flops"] / s / 1e12, peak_mfma, "TFLOP/s"
    elif bound == "hbm":
        a, p, unit = work["bytes"] / s / 1e9, PEAK_HBM_GBS, "GB/s"
    else:
        a, p, unit = work["exps"] / s / 1e12, PEAK_EXP_TPS, "Texp/s"
    return {"bound": bound, "achieved": round(a, 3), "peak": p, "unit": unit,
            "frac": round(a / p, 4), "traffic": None}


# Kernels (symbol substrings) that can carry each stage on the fused path, for
# the counter tables; for C <= 128 the decode is k_decode3 or k_decode2 when
# the head-group stages fit, else k_decode_persist when one head's route
# operands fit beside the weights, otherwise k_decode_fused.
STAGE_KERNELS_FUSED = {"call1_encode": ("k_encode_fused",),
                       "call1_combine": ("k_combine_par",), "call2_encode": ("k_encode_fused",),
                       "call2_combine": ("k_combine_par",),
                       "call3_decode": ("k_decode3", "k_decode2", "k_decode_persist", "k_decode_fused")}


def sources_digest():
    """SHA-256 over the kernel sources (comments and layout removed) and the
    build command: counters taken for other kernels are not reported."""
    import hashlib
    import re
    from paper_2608_11519_amd import build

    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_11519_amd", "csrc")
    for name in sorted(os.listdir(csrc)) + ["../../include/flarepp.h"]:
        with open(os.path.join(csrc, name)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(os.path.basename(name).encode() + b"\0" + " ".join(text.split()).encode())
    h.update(" ".join(os.path.basename(a) for a in build.command("lib")).encode())
    return h.hexdigest()


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.json")


def measured_traffic(w, stage):
    """HBM bytes per launch of the stage's kernel from the committed counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by the plain-copy calibration),
    or None when there is none for the current kernel sources."""
    path = traffic_file(w.name)
    if stage not in STAGE_KERNELS_FUSED or not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("sources_sha256") != sources_digest():
        return None
    for kern in STAGE_KERNELS_FUSED[stage]:
        if kern in t.get("kernels", {}):
            return t["kernels"][kern]["bytes_per_dispatch"]
    return None


def pmc_summary(fetch_dir, write_dir, workload, copy_mib, command):
    """Average FETCH_SIZE / WRITE_SIZE per dispatch of every flarepp kernel
    in two rocprofv3 --pmc runs, scaled by the counters of the plain device
    copy of copy_mib MiB that bench.py ran in the same process."""
    import csv
    import glob

    def read(d, counter):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                rows += [r for r in csv.DictReader(fh) if r["Counter_Name"] == counter]
        if not rows:
            raise SystemExit(f"no {counter} rows under {d}")
        return rows

    fetch, write = read(fetch_dir, "FETCH_SIZE"), read(write_dir, "WRITE_SIZE")
    copy_kib = copy_mib * 1024.0
    # the copy: the non-flarepp dispatch that fetched the most / wrote the most
    cf = max((r for r in fetch if "flarepp" not in r["Kernel_Name"]), key=lambda r: float(r["Counter_Value"]))
    copy_name = cf["Kernel_Name"]
    cw = max((r for r in write if r["Kernel_Name"] == copy_name), key=lambda r: float(r["Counter_Value"]))
    f_fac = copy_kib / float(cf["Counter_Value"])
    w_fac = copy_kib / float(cw["Counter_Value"])
    kernels = {}
    for kern in sorted({k for ks in STAGE_KERNELS_FUSED.values() for k in ks}):
        fv = [float(r["Counter_Value"]) for r in fetch if kern in r["Kernel_Name"]]
        wv = [float(r["Counter_Value"]) for r in write if kern in r["Kernel_Name"]]
        if not fv or not wv:
            continue
        fk, wk = sum(fv) / len(fv), sum(wv) / len(wv)
        kernels[kern] = {"dispatches": len(fv), "fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
                         "bytes_per_dispatch": round((fk * f_fac + wk * w_fac) * 1024.0)}
    out = {"workload": workload, "sources_sha256": sources_digest(), "command": command,
           "copy": {"mib": copy_mib, "kernel": copy_name[:80], "fetch_kib": float(cf["Counter_Value"]),
                    "write_kib": float(cw["Counter_Value"]), "fetch_factor": round(f_fac, 4),
                    "write_factor": round(w_fac, 4)},
           "kernels": kernels}
    with open(traffic_file(workload), "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


def cpu_sample_tokens(N, call_seconds, min_seconds, start=4096):
    """Token count of the oracle's bounded sample: doubles from `start` while
    a call at the current count took under a quarter of min_seconds (given
    the time call_seconds(n) of one call over n tokens), up to N."""
    n = min(start, N)
    while n < N and call_seconds(n) < min_seconds / 4:
        n = min(2 * n, N)
    return n


def cpu_baseline(w, d, min_seconds):
    """Time the float64 oracle on the host on a bounded sample of the
    workload: the mixer over the first n tokens of every batch entry (the
    same C, H, M, weights and seeds), with n the whole sequence when one call
    over it fits in a quarter of min_seconds, and calls repeated until
    min_seconds have passed.  The oracle's work per token is the same at any
    n (every token enters each routing call and projection once), so tokens/s
    over the sample is the oracle's rate on the workload."""
    from oracle import flarepp_oracle as orc

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - optional dependency
        threads = os.cpu_count() or 1

    def call(n):
        X = d["X"][:, :n]
        t0 = time.perf_counter()
        orc.mixer_forward(X, d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H)
        return time.perf_counter() - t0

    n = cpu_sample_tokens(w.N, call, min_seconds)
    reps, el = 0, 0.0
    while el < min_seconds:
        el += call(n)
        reps += 1
    what = "full batch" if n == w.N else f"first {n} of the {w.N} tokens of every batch entry"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "unknown")
    except OSError:
        model = "unknown"
    return {"value": round(w.B * n * reps / el, 1), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{w.name} (B={w.B}, N={w.N}, C={w.C}, H={w.H}, M={w.M}): {what} x {reps} calls, "
                      f"float64 NumPy, {el:.1f} s on {len(os.sched_getaffinity(0))} host cores ({model}), "
                      f"{threads} BLAS threads"}


def _time_steps(args, step, use_graph):
    """Mean ms of `step` over args.steps runs after args.warmup, replayed from
    a HIP graph when use_graph."""
    import torch

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    graph = None
    if use_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(args.warmup):
            graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        if graph is not None:
            graph.replay()
        else:
            step()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / args.steps


def backward_flops(w):
    """Algorithmic flops of the mixer backward (App. A.5), per token: the
    merge (dY, dW_O: 4 C^2), each routing call's recomputed scores and its
    four gradient products (5 x 2 M C, three calls), and the projections
    (dX, dW over four weights: 16 C^2).  The forward that the entry point
    runs again to recover its statistics is not counted."""
    return (20.0 * w.C * w.C + 30.0 * w.M * w.C) * w.B * w.N


def time_backward(args, w, t, use_graph):
    """The mixer backward on the same workload: gradients of <O, dO> for a
    seeded dO, one complete call (forward again, then the reverse pass)."""
    import torch

    from paper_2608_11519_amd import flarepp as fp
    from paper_2608_11519_amd import inputs as inp

    dcode = fp.BF16 if w.dtype == "bf16" else fp.F32
    dev = t["X"].device
    dO = torch.from_numpy(inp.make_tensor((w.B, w.N, w.C), 100, w.dtype)).to(dev, t["X"].dtype)
    ws = torch.empty(fp.flarepp_mixer_backward_workspace_bytes(dcode, w.B, w.N, w.C, w.H, w.M),
                     dtype=torch.uint8, device=dev)
    f32 = dict(dtype=torch.float32, device=dev)
    out = {"dX": torch.empty((w.B, w.N, w.C), **f32), "dseeds": torch.empty((w.H, w.M, w.D), **f32)}
    for k in ("dWk", "dWv", "dWkt", "dWvt", "dWo"):
        out[k] = torch.empty((w.C, w.C), **f32)
    args6 = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"], dO)

    def step():
        fp.flarepp_mixer_backward(*args6, H=w.H, ws=ws, out=out)

    ms = _time_steps(args, step, use_graph)
    fl = backward_flops(w)
    peak = PEAK_MFMA_BF16_TFLOPS if w.dtype == "bf16" else PEAK_MFMA_F32_TFLOPS
    tf = fl / (ms * 1e-3) / 1e12
    # the training pair: a forward that keeps its statistics, then the
    # backward from them (no second forward)
    O = torch.empty_like(t["X"])
    args7 = args6[:7]

    def train_step():
        fp.flarepp_mixer_forward_train(*args7, H=w.H, ws=ws, out=O)
        fp.flarepp_mixer_backward_from_saved(*args6, H=w.H, ws=ws, out=out)

    ms_train = None if args.no_train_pair else _time_steps(args, train_step, use_graph)
    return {"ms_per_step": round(ms, 5), "tokens_per_s": round(w.B * w.N / (ms * 1e-3), 1),
            "algorithmic_tflop": round(fl / 1e12, 4), "achieved_tflops": round(tf, 2),
            "mfma_frac": round(tf / peak, 4),
            "train_pair_ms": None if ms_train is None else round(ms_train, 5)}


def time_flare(args, w, t, use_graph):
    """The fixed-query FLARE mixer (Sec. 3.1) on the same workload and
    weights (its learned queries: the seeds), timed like the FLARE++ step:
    the paper's cost comparison of the two mixers (Sec. 3.2 end; App. C.3)."""
    import torch

    from paper_2608_11519_amd import flarepp as fp

    dcode = fp.BF16 if w.dtype == "bf16" else fp.F32
    O = torch.empty_like(t["X"])
    ws = torch.empty(fp.flarepp_flare_workspace_bytes(dcode, w.B, w.N, w.C, w.H, w.M),
                     dtype=torch.uint8, device=t["X"].device)

    def step():
        fp.flarepp_flare_forward(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H, out=O, ws=ws)

    ms = _time_steps(args, step, use_graph)
    return {"ms_per_step": round(ms, 5), "tokens_per_s": round(w.B * w.N / (ms * 1e-3), 1)}


def time_block(args, w, t, use_graph, mixer_ms):
    """The pre-norm residual block X + mixer(LayerNorm(X)) on the same workload
    and weights: what the layer-norm pass and the fused residual add to the
    mixer step."""
    import torch

    from paper_2608_11519_amd import flarepp as fp

    dcode = fp.BF16 if w.dtype == "bf16" else fp.F32
    dev = t["X"].device
    O = torch.empty_like(t["X"])
    gamma = torch.ones(w.C, dtype=t["X"].dtype, device=dev)
    beta = torch.zeros_like(gamma)
    ws = torch.empty(fp.flarepp_block_workspace_bytes(dcode, w.B, w.N, w.C, w.H, w.M),
                     dtype=torch.uint8, device=dev)

    def step():
        fp.flarepp_block_forward(t["X"], gamma, beta, t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"],
                                 H=w.H, out=O, ws=ws)

    ms = _time_steps(args, step, use_graph)
    return {"ms_per_step": round(ms, 5), "tokens_per_s": round(w.B * w.N / (ms * 1e-3), 1),
            "over_mixer_ms": round(ms - mixer_ms, 5)}


def main(argv=None):
    args = parse_args(argv)
    if args.pmc_summary:
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.workload,
                    args.copy_calibration_mib or 256, args.pmc_command)
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the mixer forward is benchmarked on a single MI355X)", file=sys.stderr)
        return 2
    import numpy as np
    import torch

    from paper_2608_11519_amd import flarepp as fp
    from paper_2608_11519_amd import inputs as inp

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    fp.load()
    w = inp.workload(args.workload)
    d = inp.make_inputs(w, args.seed)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dev = torch.device("cuda:0")
    t = {k: torch.from_numpy(v).to(dev, tdt) for k, v in d.items()}
    O = torch.empty_like(t["X"])
    dcode = fp.BF16 if w.dtype == "bf16" else fp.F32
    ws = torch.empty(fp.flarepp_mixer_workspace_bytes(dcode, w.B, w.N, w.C, w.H, w.M),
                     dtype=torch.uint8, device=dev)
    margs = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])

    def step():
        fp.flarepp_mixer_forward(*margs, H=w.H, out=O, ws=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
    print(f"[bench] {inp.describe(w)} warmup done", file=sys.stderr, flush=True)

    # ---- timed region: K whole-mixer steps ----
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        if graph is not None:
            graph.replay()
        else:
            step()
    ev1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    dev_ms = ev0.elapsed_time(ev1)
    ms_per_step = max(dev_ms, 1e-9) / args.steps
    tokens = w.B * w.N
    value = tokens / (ms_per_step * 1e-3)
    print(f"[bench] timed {args.steps} steps: {ms_per_step * 1e3:.1f} us/step", file=sys.stderr, flush=True)

    # ---- per-stage device times: each stage launched alone, back to back ----
    fused = fp.flarepp_mixer_path(dcode, w.B, w.N, w.C, w.H, w.M) == fp.PATH_FUSED
    empty = {"prep", "project", "merge"} if fused else set()
    reps = max(args.stage_reps, 1)
    stage_ms = {}
    for k, name in enumerate(fp.PROFILE_STAGES, start=1):
        if name in empty:
            stage_ms[name] = 0.0
            continue

        def run_stage(k=k):
            for _ in range(reps):
                fp.flarepp_mixer_stage(k, *margs, H=w.H, out=O, ws=ws)

        sg = None
        if graph is not None:
            sg = torch.cuda.CUDAGraph()
            with torch.cuda.graph(sg):
                run_stage()
            sg.replay()
        else:
            run_stage()
        torch.cuda.synchronize()
        # the median of five timed regions of `reps` launches each (a single
        # region varies by a few microseconds per launch from run to run)
        region_ms = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            if sg is not None:
                sg.replay()
            else:
                run_stage()
            e1.record()
            torch.cuda.synchronize()
            region_ms.append(e0.elapsed_time(e1) / reps)
        stage_ms[name] = sorted(region_ms)[2]
    step()  # leave the workspace and O as one complete step wrote them
    torch.cuda.synchronize()
    flare = time_flare(args, w, t, graph is not None)
    backward = None if args.no_backward else time_backward(args, w, t, graph is not None)
    block = None if args.no_block else time_block(args, w, t, graph is not None, ms_per_step)
    work = stage_work(w, fused)
    stages = {n: {"ms": round(stage_ms[n], 5), **roofline(work[n], stage_ms[n], w.dtype)}
              for n in fp.PROFILE_STAGES if n not in empty}
    dominant = max(stage_ms, key=stage_ms.get)
    roof = dict(roofline(work[dominant], stage_ms[dominant], w.dtype))
    roof["kernel"] = dominant
    roof["traffic"] = measured_traffic(w, dominant)
    route_names = ("call1_encode", "call1_combine", "call2_encode", "call2_combine", "call3_decode")
    route_ms = sum(stage_ms[n] for n in route_names)
    route_flops = 3 * 4.0 * tokens * w.M * w.C
    total_flops = route_flops + 10.0 * tokens * w.C * w.C
    peak = PEAK_MFMA_BF16_TFLOPS if w.dtype == "bf16" else PEAK_MFMA_F32_TFLOPS

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "N": w.N, "C": w.C, "H": w.H, "D": w.D, "M": w.M,
                   "storage": w.dtype, "accumulate": "f32", "launch": "hip-graph" if graph else "eager"},
        "roofline": roof,
        "mfma_frac_routing_calls": round(route_flops / (route_ms * 1e-3) / (peak * 1e12), 4),
        "mfma_frac_mixer": round(total_flops / (ms_per_step * 1e-3) / (peak * 1e12), 4),
        "stages": stages,
        "wall_ms_timed_region": round(wall_ms, 3),
        "flare": {**flare, "flarepp_over_flare_time": round(ms_per_step / flare["ms_per_step"], 3)},
    }
    if block is not None:
        out["block"] = block
    if backward is not None:
        out["backward"] = backward
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, d, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

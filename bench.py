#!/usr/bin/env python3
"""Benchmark of the FLARE++ mixer forward on one MI355X (gfx950).

One step = one complete mixer forward (project; query synthesis, encode and
decode routing calls; merge) over one batch of synthetic inputs already
resident in HBM.  Default workload: the 2D structured-grid surrogate layer
(B=4, N=16384, C=128, H=8, D=16, M=128, bf16 storage, fp32 accumulation).

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
# v_exp_f32 issue rate: 256 CUs x 2.4 GHz x 32 per clock per CU (half the
# 64-lane fp32 vector rate; see the derivation in the design notes)
PEAK_EXP_TPS = 256 * 2.4e9 * 32 / 1e12  # Texp/s


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="grid2d")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-graph", action="store_true", help="launch every step eagerly")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum host seconds spent timing the oracle")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (for counter scaling)")
    return ap.parse_args(argv)


def stage_work(w):
    """Algorithmic flops, HBM bytes and exponentials per launch of each stage.

    Bytes count only what the method must move at this stage boundary
    (inputs read once, outputs written once), not re-reads."""
    T, C, M, H = w.B * w.N, w.C, w.M, w.H
    bs = 2 if w.dtype == "bf16" else 4
    enc_flops = 4.0 * T * M * C
    return {
        "prep": dict(flops=0.0, bytes=5.0 * C * C * bs, exps=0.0),
        "project": dict(flops=8.0 * T * C * C, bytes=5.0 * T * C * bs, exps=0.0),
        "call1_encode": dict(flops=enc_flops, bytes=2.0 * T * C * bs, exps=1.0 * T * H * M),
        "call1_combine": dict(flops=0.0, bytes=4.0 * w.B * H * M * w.D, exps=0.0),
        "call2_encode": dict(flops=enc_flops, bytes=2.0 * T * C * bs, exps=1.0 * T * H * M),
        "call2_combine": dict(flops=0.0, bytes=4.0 * w.B * H * M * w.D, exps=0.0),
        "call3_decode": dict(flops=enc_flops, bytes=2.0 * T * C * bs, exps=1.0 * T * H * M),
        "merge": dict(flops=2.0 * T * C * C, bytes=2.0 * T * C * bs, exps=0.0),
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


def cpu_baseline(w, d, min_seconds):
    """Time the float64 oracle on the host (the full batch, repeated until
    min_seconds have passed)."""
    from oracle import flarepp_oracle as orc

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - optional dependency
        threads = os.cpu_count() or 1
    reps, t0 = 0, time.perf_counter()
    while True:
        orc.mixer_forward(d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    return {"value": round(w.B * w.N * reps / el, 1), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"full {w.name} batch (B={w.B}, N={w.N}) x {reps}, float64 NumPy, "
                      f"{el:.1f} s on {len(os.sched_getaffinity(0))} host cores"}


def main(argv=None):
    args = parse_args(argv)
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

    # ---- per-stage device times (HIP events around each stage) ----
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(fp.PROFILE_EVENTS)]
           for _ in range(args.steps)]
    for k in range(args.steps):
        fp.flarepp_mixer_forward_profiled(*margs, H=w.H, events=evs[k], out=O, ws=ws)
    torch.cuda.synchronize()
    stage_ms = {}
    for i, name in enumerate(fp.PROFILE_STAGES):
        stage_ms[name] = float(np.mean([evs[k][i].elapsed_time(evs[k][i + 1]) for k in range(args.steps)]))
    work = stage_work(w)
    stages = {n: {"ms": round(stage_ms[n], 5), **roofline(work[n], stage_ms[n], w.dtype)}
              for n in fp.PROFILE_STAGES}
    dominant = max(stage_ms, key=stage_ms.get)
    roof = dict(roofline(work[dominant], stage_ms[dominant], w.dtype))
    roof["kernel"] = dominant
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
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, d, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

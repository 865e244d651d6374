"""Host-side logic of bench.py (no GPU): the one-GPU contract, the counter
summary that feeds roofline.traffic, and the algorithmic work figures."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_11519_amd import inputs as inp  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)


def test_traffic_is_reported_only_for_the_sources_it_was_taken_on(monkeypatch):
    # counters taken for other kernel sources are never reported
    w = inp.workload("grid2d")
    monkeypatch.setattr(bench, "sources_digest", lambda: "not-the-digest-of-any-counter-file")
    assert bench.measured_traffic(w, "call3_decode") is None


def test_decode_algorithmic_bytes_and_flops():
    # per launch at grid2d: X read and O written once (bf16), 4 T M C + 2 T C^2
    # flops, T H M exponentials
    w = inp.workload("grid2d")
    work = bench.stage_work(w, True)["call3_decode"]
    T = w.B * w.N
    assert work["bytes"] == 2 * T * w.C * 2
    assert work["flops"] == 4 * T * w.M * w.C + 2 * T * w.C * w.C
    assert work["exps"] == T * w.H * w.M


def test_backward_flops_formula():
    w = inp.workload("grid2d")
    assert bench.backward_flops(w) == (20.0 * w.C ** 2 + 30.0 * w.M * w.C) * w.B * w.N


def test_default_workload_is_the_largest_single_gpu_configuration():
    args = bench.parse_args([])
    w = inp.workload(args.workload)
    assert w.name == "mesh3d" and w.B * w.N == max(v.B * v.N for v in inp.WORKLOADS.values())


def test_cpu_sample_grows_until_a_call_takes_a_quarter_of_the_budget():
    # a call over n tokens takes n / 1e4 seconds: with 12 s of budget the
    # sample doubles from 4096 while a call is under 3 s
    assert bench.cpu_sample_tokens(1 << 20, lambda n: n / 1e4, 12.0) == 32768
    assert bench.cpu_sample_tokens(1000, lambda n: n / 1e4, 12.0) == 1000
    assert bench.cpu_sample_tokens(20000, lambda n: n / 1e4, 1e9) == 20000

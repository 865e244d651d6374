"""GPU parity of the pre-norm residual block, X + mixer(LayerNorm(X)), against
the float64 oracle, through the C ABI.

The layer norm runs as its own pass; the residual is added in the store of
the mixer's output projection, on every path that writes O (the fused decode
kernels and the unfused merge projection).  Gates as for the mixer: max |err|
within 1e-4 (fp32) or 2e-2 (bf16) of the reference's max |O|.  Every case also
checks that the gate would reject a block that dropped the mixer (O = X), so
the residual cannot pass the test on its own.  The workloads' X is scaled by
1/4 (exact in both storage types): the layer norm removes the scale, so the
mixer sees the workload's inputs, and its share of O grows from ~10% to ~30%.
"""

import numpy as np
import pytest
import torch

from oracle import flarepp_oracle as orc
from paper_2608_11519_amd import flarepp as fp
from paper_2608_11519_amd import inputs as inp

from gpu_util import TOL, assert_close, rel_err, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp.load()
    yield


def _check_block(w, d, label, seed=40, eps=1e-5):
    print(f"[case] block {label} {inp.describe(w)}", flush=True)
    d = dict(d, X=np.asarray(d["X"], dtype=np.float32) * 0.25)
    gamma = 1.0 + inp.make_tensor((w.C,), seed, w.dtype, scale=0.2)
    gamma = inp.round_to_bf16(gamma.astype(np.float32)) if w.dtype == "bf16" else gamma.astype(np.float32)
    beta = inp.make_tensor((w.C,), seed + 1, w.dtype, scale=0.2)
    t = upload(dict(d, gamma=gamma, beta=beta), w)
    O = fp.flarepp_block_forward(t["X"], t["gamma"], t["beta"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"],
                                 t["seeds"], H=w.H, eps=eps)
    torch.cuda.synchronize()
    got = O.float().cpu().numpy()
    ref = orc.block_forward(d["X"], gamma, beta, eps, d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H)
    tol = TOL[w.dtype]
    assert rel_err(np.asarray(d["X"], dtype=np.float64), ref) > 5 * tol, "the mixer term is too small to test"
    assert_close("O", got, ref, tol, label)
    # the mixer's share on its own, O - X against mixer(LN(X)), at the same
    # gate relative to max |mixer(LN(X))| (with bf16 the difference also
    # carries the rounding of O to its storage type, ~0.2% of max |O|)
    assert_close("O-X", got - np.asarray(d["X"], dtype=np.float64), ref - np.asarray(d["X"], dtype=np.float64),
                 tol, label)
    return got


def test_block_tiny_fp32():
    w = inp.workload("tiny")
    _check_block(w, inp.make_inputs(w, 0, seed_scale=4.0), "tiny")


@pytest.mark.parametrize("name", ["grid2d", "mesh"])
def test_block_bf16_workloads_full_size(name):
    w = inp.workload(name)
    _check_block(w, inp.make_inputs(w, 0), name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_block_unfused_path(monkeypatch, dtype):
    monkeypatch.setenv("FLAREPP_UNFUSED", "1")
    w = inp.Workload("block-unfused", 2, 900, 64, 4, 48, dtype, "normal")
    dt = fp.F32 if dtype == "f32" else fp.BF16
    assert fp.flarepp_mixer_path(dt, w.B, w.N, w.C, w.H, w.M) == fp.PATH_UNFUSED
    _check_block(w, inp.make_inputs(w, 15, seed_scale=4.0), f"unfused-{dtype}")


@pytest.mark.parametrize("kind", [0, 1, 2, 3])
def test_block_every_decode_kernel(monkeypatch, kind):
    monkeypatch.setenv("FLAREPP_DECODE_KIND", str(kind))
    w = inp.Workload("block-deckind", 2, 1500, 128, 8, 64, "bf16", "normal")
    _check_block(w, inp.make_inputs(w, 16, seed_scale=4.0), f"decode-kind{kind}")


@pytest.mark.parametrize("C,H,dtype", [(96, 3, "f32"), (32, 2, "bf16"), (512, 8, "bf16"), (1024, 16, "bf16"), (2048, 32, "f32")])
def test_block_widths(C, H, dtype):
    # the layer norm's kernels: C = 96 takes the one-wave-per-token kernel,
    # C = 32 and 512 a single run of 8 channels per lane (16 and 1 tokens per
    # wave), C = 1024 and 2048 two and four runs per lane
    w = inp.Workload("block-width", 1, 300, C, H, 32, dtype, "normal")
    _check_block(w, inp.make_inputs(w, 17, seed_scale=4.0), f"C{C}")


def test_block_large_eps_and_token_tail():
    w = inp.Workload("block-eps", 1, 33, 64, 2, 5, "f32", "normal")
    _check_block(w, inp.make_inputs(w, 18, seed_scale=4.0), "eps", eps=0.5)


def test_block_workspace_and_output_reuse():
    w = inp.Workload("block-reuse", 1, 700, 128, 4, 32, "bf16", "normal")
    d = inp.make_inputs(w, 19, seed_scale=4.0)
    t = upload(d, w)
    gamma = torch.ones(w.C, dtype=torch.bfloat16, device="cuda")
    beta = torch.zeros_like(gamma)
    n = fp.flarepp_block_workspace_bytes(fp.BF16, w.B, w.N, w.C, w.H, w.M)
    assert n > fp.flarepp_mixer_workspace_bytes(fp.BF16, w.B, w.N, w.C, w.H, w.M)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    out = torch.empty_like(t["X"])
    args = (t["X"], gamma, beta, t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])
    a = fp.flarepp_block_forward(*args, H=w.H, ws=ws, out=out).clone()
    b = fp.flarepp_block_forward(*args, H=w.H, ws=ws, out=out)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


BWD = ("dX", "dgamma", "dbeta", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dseeds")


@pytest.mark.parametrize("name,C,H", [("tiny", None, None), ("grid2d", None, None), ("widths", 96, 3)])
def test_block_backward(name, C, H):
    # the layer norm's backward (both layer-norm kernel shapes: C = 64, 128
    # take the vector kernel's statistics, C = 96 the one-wave-per-token one)
    # and the residual on top of the mixer backward
    w = inp.workload(name) if C is None else inp.Workload("block-bwd", 1, 300, C, H, 32, "f32", "normal")
    d = inp.make_inputs(w, 27, seed_scale=4.0)
    d = dict(d, X=np.asarray(d["X"], dtype=np.float32) * 0.25)
    print(f"[case] block backward {name} {inp.describe(w)}", flush=True)
    gamma = 1.0 + inp.make_tensor((w.C,), 28, w.dtype, scale=0.2)
    gamma = inp.round_to_bf16(gamma.astype(np.float32)) if w.dtype == "bf16" else gamma.astype(np.float32)
    beta = inp.make_tensor((w.C,), 29, w.dtype, scale=0.2)
    dO = inp.make_tensor((w.B, w.N, w.C), 30, w.dtype)
    t = upload(dict(d, gamma=gamma, beta=beta, dO=dO), w)
    g = fp.flarepp_block_backward(t["X"], t["gamma"], t["beta"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"],
                                  t["seeds"], t["dO"], H=w.H)
    torch.cuda.synchronize()
    ref = orc.block_backward(d["X"], gamma, beta, 1e-5, d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"],
                             w.H, dO)
    for k in BWD:
        assert_close(k, g[k].cpu().numpy(), ref[k], TOL[w.dtype], f"block-bwd-{name}")


@pytest.mark.parametrize("B,N,C,H,M,dtype", [(2, 33, 64, 4, 100, "f32"), (1, 1500, 256, 8, 64, "bf16")])
def test_block_backward_tail_and_wide(B, N, C, H, M, dtype):
    w = inp.Workload("block-bwd-shapes", B, N, C, H, M, dtype, "normal")
    d = inp.make_inputs(w, 33, seed_scale=4.0)
    d = dict(d, X=np.asarray(d["X"], dtype=np.float32) * 0.25)
    print(f"[case] block backward {inp.describe(w)}", flush=True)
    gamma = 1.0 + inp.make_tensor((w.C,), 34, w.dtype, scale=0.2)
    gamma = inp.round_to_bf16(gamma.astype(np.float32)) if w.dtype == "bf16" else gamma.astype(np.float32)
    beta = inp.make_tensor((w.C,), 35, w.dtype, scale=0.2)
    dO = inp.make_tensor((w.B, w.N, w.C), 36, w.dtype)
    t = upload(dict(d, gamma=gamma, beta=beta, dO=dO), w)
    g = fp.flarepp_block_backward(t["X"], t["gamma"], t["beta"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"],
                                  t["seeds"], t["dO"], H=w.H)
    torch.cuda.synchronize()
    ref = orc.block_backward(d["X"], gamma, beta, 1e-5, d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"],
                             w.H, dO)
    for k in BWD:
        assert_close(k, g[k].cpu().numpy(), ref[k], TOL[w.dtype], "block-bwd-shapes")

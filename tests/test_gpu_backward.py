"""GPU parity of the mixer backward (App. A.5) against the float64 oracle,
through the C ABI.

The output gradient dO is a seeded N(0, 1) tensor in the storage type; both
sides see the same rounded values.  Gates as for the forward: every gradient
(dX, the five weight gradients, the seed gradient) and the summed latent and
query gradients dZ, dQ within 1e-4 (fp32) or 2e-2 (bf16) of the reference's
max |.|.
"""

import numpy as np
import pytest
import torch

from oracle import flarepp_oracle as orc
from paper_2608_11519_amd import flarepp as fp
from paper_2608_11519_amd import inputs as inp

from gpu_util import TOL, assert_close, rel_err, upload

pytestmark = pytest.mark.gpu

GRADS = ("dX", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dseeds")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp.load()
    yield


def _run(w, d, dO, debug=True):
    t = upload(d, w)
    dOt = torch.from_numpy(dO).to("cuda", t["X"].dtype)
    args = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"], dOt)
    g = fp.flarepp_mixer_backward_debug(*args, H=w.H) if debug else fp.flarepp_mixer_backward(*args, H=w.H)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in g.items()}


def _check(w, d, label, dO_seed=100, tol=None):
    print(f"[case] backward {label} {inp.describe(w)}", flush=True)
    dO = inp.make_tensor((w.B, w.N, w.C), dO_seed, w.dtype)
    got = _run(w, d, dO)
    ref = orc.mixer_backward(d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H, dO)
    tol = TOL[w.dtype] if tol is None else tol
    for k in GRADS + ("dZ", "dQ"):
        assert_close(k, got[k], ref[k], tol, label)
    return got, ref


def test_backward_tiny_fp32():
    w = inp.workload("tiny")
    _check(w, inp.make_inputs(w, 0, seed_scale=4.0), "tiny")


def test_backward_grid2d_full_size():
    w = inp.workload("grid2d")
    _check(w, inp.make_inputs(w, 0), "grid2d")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_sharp_seeds(dtype):
    # seeds x8: far-from-uniform routing weights, so dS = P (dP - c) is not
    # dominated by the mean-field term
    w = inp.Workload("bwd-sharp", 2, 1500, 64, 4, 64, dtype, "normal")
    _check(w, inp.make_inputs(w, 2, seed_scale=8.0), "sharp")


@pytest.mark.parametrize("N,M", [(33, 100), (1000, 1), (777, 48), (5, 3)])
def test_backward_tails_and_route_counts(N, M):
    w = inp.Workload("bwd-tail", 2, N, 64, 4, M, "f32", "normal")
    _check(w, inp.make_inputs(w, 3, seed_scale=4.0), f"N{N}-M{M}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_backward_several_tiles_per_wave_with_tail(dtype):
    # two heads over 40,013 tokens: 1,251 position tiles per (b, h), so each
    # wave of the SDPA backward walks two of them (in bf16 at D = 16 the
    # second tile's rows are staged through LDS during the first), and the
    # last tile holds 13 positions
    w = inp.Workload("bwd-tiles", 1, 40013, 32, 2, 40, dtype, "normal")
    _check(w, inp.make_inputs(w, 11, seed_scale=4.0), "tiles-tail")


@pytest.mark.parametrize("D,dtype", [(32, "bf16"), (64, "bf16"), (32, "f32"), (64, "f32")])
def test_backward_head_widths(D, dtype):
    w = inp.Workload("bwd-width", 2, 600, 2 * D, 2, 40, dtype, "normal")
    _check(w, inp.make_inputs(w, 5, seed_scale=4.0), f"D{D}")


def test_backward_wide_channels_bf16():
    # C = 256 (eight heads of 32), the mesh workload's width, at a small N
    w = inp.Workload("bwd-c256", 1, 2000, 256, 8, 96, "bf16", "fourier")
    _check(w, inp.make_inputs(w, 6), "C256")


def test_backward_plain_entry_matches_debug():
    w = inp.Workload("bwd-plain", 1, 700, 64, 4, 32, "bf16", "normal")
    d = inp.make_inputs(w, 7, seed_scale=4.0)
    dO = inp.make_tensor((w.B, w.N, w.C), 8, w.dtype)
    a = _run(w, d, dO, debug=True)
    b = _run(w, d, dO, debug=False)
    for k in GRADS:
        assert np.array_equal(a[k], b[k]), k


def test_backward_deterministic_bitwise():
    w = inp.Workload("bwd-det", 2, 3000, 128, 8, 64, "bf16", "normal")
    d = inp.make_inputs(w, 9)
    dO = inp.make_tensor((w.B, w.N, w.C), 10, w.dtype)
    a = _run(w, d, dO)
    b = _run(w, d, dO)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_many_routes_in_windows(dtype):
    # M = 300 at D = 64: the route gradients of a head do not fit in LDS at
    # once, so the SDPA backward walks the routes in windows (the last one
    # partial) and the later windows add to the long-side gradients
    w = inp.Workload("bwd-windows", 1, 700, 128, 2, 300, dtype, "normal")
    _check(w, inp.make_inputs(w, 12, seed_scale=4.0), "M300")


def _golden_backward():
    """The stored float64-oracle gradients at 2^18 tokens and the script that
    wrote them (its workload and seeds)."""
    import importlib.util
    import os
    here = os.path.join(os.path.dirname(__file__), "golden")
    spec = importlib.util.spec_from_file_location("make_backward_expected",
                                                  os.path.join(here, "make_backward_expected.py"))
    mk = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mk)
    return mk, np.load(mk.OUT, allow_pickle=False)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_backward_quarter_million_tokens_against_stored_oracle(dtype):
    # N = 2^18 tokens, C = 128, H = 8, M = 128: the seed gradient, the five
    # weight gradients, dZ, dQ and dX at one token of every 512-token block
    # against float64 oracle values stored by
    # tests/golden/make_backward_expected.py (the oracle takes a few minutes
    # here).  Both storage types read the same bf16-rounded inputs.
    mk, ref = _golden_backward()
    wb = mk.workload()
    w = wb.replace(dtype=dtype)
    print(f"[case] backward stored-oracle {inp.describe(w)}", flush=True)
    d = inp.make_inputs(wb, mk.INPUT_SEED)
    dO = inp.make_tensor((wb.B, wb.N, wb.C), mk.DO_SEED, wb.dtype)
    got = _run(w, d, dO)
    tol = TOL[dtype]
    tok = ref["tokens"]
    assert len(tok) >= w.N // mk.BLOCK
    for k in ("dseeds", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dZ", "dQ"):
        assert_close(k, got[k], ref[k], tol, "quartermega")
    assert_close("dX[tokens]", got["dX"][:, tok], ref["dX"], tol, "quartermega")


def test_value_gradients_keep_their_token_part_at_half_a_million_tokens(monkeypatch):
    # N = 2^19, M = 512: the encoders' softmaxes over the tokens are near
    # uniform, so a value gradient P^T dOut is a large common part plus a
    # small token-dependent part, which bf16 alone rounds away; dW_V = X^T dV
    # is made of that part.  The bf16 path keeps dV, dV~ as hi + lo pairs;
    # checked against the fp32 path (itself held to the oracle above), and
    # the same shape with hi alone must miss the gate (the case has power).
    w = inp.Workload("bwd-halfmega", 1, 1 << 19, 128, 8, 512, "bf16", "normal")
    print(f"[case] backward value-gradient precision {inp.describe(w)}", flush=True)
    d = inp.make_inputs(w, 20)
    dO = inp.make_tensor((w.B, w.N, w.C), 21, "bf16")  # exact in both types
    ref = _run(w.replace(dtype="f32"), d, dO, debug=False)
    got = _run(w, d, dO, debug=False)
    for k in GRADS:
        assert_close(k, got[k], ref[k], 1e-2, "halfmega")
    monkeypatch.setenv("FLAREPP_BWD_NO_LO", "1")
    hi = _run(w, d, dO, debug=False)
    e = rel_err(hi["dWv"], ref["dWv"])
    print(f"  hi alone: dWv {e:.3e}", flush=True)
    assert e > TOL["bf16"], "with hi alone dW_V should miss the bf16 gate at this size"


@pytest.mark.parametrize("name", ["tiny", "grid2d"])
def test_shared_projection_backward(name):
    # K~ = K, V~ = V: the tied weights' gradients sum their two uses
    w = inp.workload(name)
    d = inp.make_inputs(w, 22, seed_scale=4.0)
    print(f"[case] backward shared {inp.describe(w)}", flush=True)
    dO = inp.make_tensor((w.B, w.N, w.C), 23, w.dtype)
    t = upload(d, w)
    dOt = torch.from_numpy(dO).to("cuda", t["X"].dtype)
    g = fp.flarepp_mixer_backward_shared(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], dOt, H=w.H)
    torch.cuda.synchronize()
    ref = orc.mixer_backward_shared(d["X"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], w.H, dO)
    for k in ("dX", "dWk", "dWv", "dWo", "dseeds"):
        assert_close(k, g[k].cpu().numpy(), ref[k], TOL[w.dtype], f"shared-{name}")


@pytest.mark.parametrize("name", ["tiny", "grid2d"])
def test_training_forward_then_backward_from_saved(name):
    # the training forward's O against the oracle; the backward from its
    # saved state bitwise equal to the backward that runs the forward again,
    # for two output gradients from one forward
    w = inp.workload(name)
    d = inp.make_inputs(w, 24, seed_scale=4.0)
    print(f"[case] training pair {inp.describe(w)}", flush=True)
    t = upload(d, w)
    args = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])
    dt = fp.F32 if w.dtype == "f32" else fp.BF16
    ws = torch.empty(fp.flarepp_mixer_backward_workspace_bytes(dt, w.B, w.N, w.C, w.H, w.M), dtype=torch.uint8,
                     device="cuda")
    O = fp.flarepp_mixer_forward_train(*args, H=w.H, ws=ws)
    torch.cuda.synchronize()
    ref = orc.mixer_forward(d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H)
    assert_close("O", O.float().cpu().numpy(), ref["O"], TOL[w.dtype], f"train-{name}")
    for seed in (25, 26):
        dO = torch.from_numpy(inp.make_tensor((w.B, w.N, w.C), seed, w.dtype)).to("cuda", t["X"].dtype)
        a = fp.flarepp_mixer_backward_from_saved(*args, dO, H=w.H, ws=ws)
        b = fp.flarepp_mixer_backward(*args, dO, H=w.H)
        torch.cuda.synchronize()
        for k in GRADS:
            assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("B,N,C,H,M,dtype", [(1, 2000, 256, 8, 96, "bf16"), (2, 33, 64, 4, 300, "f32"),
                                             (1, 700, 128, 2, 300, "bf16")])
def test_shared_and_training_pair_on_other_shapes(B, N, C, H, M, dtype):
    # C = 256 (eight heads of 32), a token tail with M > N, and M = 300 at
    # D = 64 (route windows): the shared backward against the oracle, the
    # training pair bitwise against the full backward
    w = inp.Workload("bwd-shapes", B, N, C, H, M, dtype, "normal")
    d = inp.make_inputs(w, 31, seed_scale=4.0)
    print(f"[case] shared + training pair {inp.describe(w)}", flush=True)
    dO = inp.make_tensor((w.B, w.N, w.C), 32, w.dtype)
    t = upload(d, w)
    dOt = torch.from_numpy(dO).to("cuda", t["X"].dtype)
    g = fp.flarepp_mixer_backward_shared(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], dOt, H=w.H)
    torch.cuda.synchronize()
    ref = orc.mixer_backward_shared(d["X"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], w.H, dO)
    for k in ("dX", "dWk", "dWv", "dWo", "dseeds"):
        assert_close(k, g[k].cpu().numpy(), ref[k], TOL[w.dtype], "shared-shapes")
    args = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])
    dt = fp.F32 if w.dtype == "f32" else fp.BF16
    ws = torch.empty(fp.flarepp_mixer_backward_workspace_bytes(dt, w.B, w.N, w.C, w.H, w.M), dtype=torch.uint8,
                     device="cuda")
    fp.flarepp_mixer_forward_train(*args, H=w.H, ws=ws)
    a = fp.flarepp_mixer_backward_from_saved(*args, dOt, H=w.H, ws=ws)
    b = fp.flarepp_mixer_backward(*args, dOt, H=w.H)
    torch.cuda.synchronize()
    for k in GRADS:
        assert torch.equal(a[k], b[k]), k

"""GPU parity of the fixed-query FLARE mixer (Sec. 3.1, Eqs. (4)-(5)) against
the float64 oracle, through the C ABI.

FLARE is FLARE++ without the query synthesis: the learned queries (here the
seeded `seeds` tensor, [H, M, D]) are the routes of both calls.  Gates as for
the FLARE++ mixer: fp32 1e-4, bf16 2e-2 of the reference's max |.|, on O and
on the stage results Z and Y; the fp32 cases also get the centred gate.
"""

import numpy as np
import pytest
import torch

from oracle import flarepp_oracle as orc
from paper_2608_11519_amd import flarepp as fp
from paper_2608_11519_amd import inputs as inp

from gpu_util import CENTRED_TOL, TOL, assert_close, centred, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp.load()
    yield


def _check_flare(w, d, label, centred_gate=False):
    print(f"[case] flare {label} {inp.describe(w)}", flush=True)
    t = upload(d, w)
    O, Z, Y = fp.flarepp_flare_forward_debug(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H)
    O2 = fp.flarepp_flare_forward(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H)
    torch.cuda.synchronize()
    assert torch.equal(O, O2), "the debug entry point computes the same O"
    got = {"O": O.float().cpu().numpy(), "Z": Z.cpu().numpy(), "Y": Y.float().cpu().numpy()}
    ref = orc.flare_forward(d["X"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], w.H)
    tol = TOL[w.dtype]
    for k in ("O", "Z", "Y"):
        assert_close(k, got[k], ref[k], tol, label)
    if centred_gate:
        for k in ("Y", "O"):
            assert_close(k + "-centred", centred(got[k]), centred(ref[k]), CENTRED_TOL, label)
    return got, ref


def test_flare_tiny_fp32_centred():
    w = inp.workload("tiny")
    _check_flare(w, inp.make_inputs(w, 0, seed_scale=4.0), "tiny", centred_gate=True)


@pytest.mark.parametrize("name", ["grid2d", "lra"])
def test_flare_bf16_workloads_full_size(name):
    w = inp.workload(name)
    _check_flare(w, inp.make_inputs(w, 0), name)


def test_flare_mesh_workload_full_size():
    w = inp.workload("mesh")
    _check_flare(w, inp.make_inputs(w, 0), "mesh")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_flare_sharp_queries(dtype):
    # queries x8: the routing weights are far from uniform
    w = inp.Workload("sharp", 2, 3000, 64, 4, 64, dtype, "normal")
    _check_flare(w, inp.make_inputs(w, 2, seed_scale=8.0), "sharp", centred_gate=(dtype == "f32"))


@pytest.mark.parametrize("N,M", [(33, 100), (1000, 1), (777, 48)])
def test_flare_tails_and_route_counts(N, M):
    w = inp.Workload("flare-tail", 2, N, 64, 4, M, "f32", "normal")
    # (with one route Y is token-constant: the centred gate has nothing to measure)
    got, _ = _check_flare(w, inp.make_inputs(w, 3, seed_scale=4.0), f"N{N}-M{M}", centred_gate=M > 1)
    if M == 1:  # one route: every token receives Z
        for h in range(w.H):
            ys = got["Y"][:, :, h * w.D:(h + 1) * w.D]
            np.testing.assert_allclose(ys, np.broadcast_to(got["Z"][:, h, 0][:, None], ys.shape),
                                       rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("D", [32, 64])
def test_flare_head_widths(D):
    w = inp.Workload("flare-width", 2, 500, 2 * D, 2, 40, "bf16", "normal")
    _check_flare(w, inp.make_inputs(w, 5, seed_scale=4.0), f"D{D}")


# C = 256, H = 8 (D = 32), M = 256, Fourier-feature tokens and a token tail:
# the irregular-mesh workload's kernels away from near-uniform softmaxes
_C256 = inp.Workload("flare-c256", 1, 5000, 256, 8, 256, "bf16", "fourier")


@pytest.mark.parametrize("variant", ["sharp", "hot", "nofast"])
def test_flare_c256_stress_bf16(monkeypatch, variant):
    w = _C256
    assert fp.flarepp_mixer_path(fp.BF16, w.B, w.N, w.C, w.H, w.M) == fp.PATH_FUSED
    if variant == "sharp":
        d = inp.make_inputs(w, 41, seed_scale=8.0)
    elif variant == "hot":
        d = inp.make_inputs(w, 42, x_scale=3.0, seed_scale=2.0)
    else:
        monkeypatch.setenv("FLAREPP_NO_FAST_PATH", "1")
        d = inp.make_inputs(w, 43, seed_scale=4.0)
    _check_flare(w, d, f"c256-{variant}")


def test_flare_empty_chunks_with_very_negative_row_maxima(monkeypatch):
    """Tokens with a common offset, and every fourth query pointing away from
    the offset's key: those routes' scores are all far below zero (row maxima
    between about -100 and -180 in log2 units), so their encode runs on the
    online maximum.  With 40 forced chunks of 128 tokens over N = 1024 the
    chunks past the last token start on super-tile boundaries; their partials
    must be (-inf, 0, 0) (App. A.3), or the merge would scale those routes'
    sums by 2^(max - 0), which underflows to zero."""
    monkeypatch.setenv("FLAREPP_FORCE_CHUNKS", "40")
    w = inp.Workload("flare-offset", 1, 1024, 64, 4, 64, "f32", "normal")
    d = inp.make_inputs(w, 21, seed_scale=2.0)
    off = np.float32(8.0)
    d["X"] = (d["X"] + off).astype(np.float32)
    # the key of the common offset, per head, and queries of length 16 against it
    k0 = np.full(w.C, float(off)) @ d["Wk"].astype(np.float64)
    q = d["seeds"].astype(np.float64).copy()
    for h in range(w.H):
        kh = k0[h * w.D:(h + 1) * w.D]
        q[h, ::4] = -16.0 * kh / np.linalg.norm(kh)
    d["seeds"] = q.astype(np.float32)
    _check_flare(w, d, "offset-R40")


@pytest.mark.parametrize("M", [96, 512])
def test_flare_persistent_decode(monkeypatch, M):
    # the persistent decode on the fixed queries (natural at M = 512)
    monkeypatch.setenv("FLAREPP_DECODE_KIND", "3")
    w = inp.Workload("flare-persist", 2, 3000, 128, 8, M, "bf16", "normal")
    _check_flare(w, inp.make_inputs(w, 44, seed_scale=6.0), f"persist-M{M}")


def test_flare_online_max_path(monkeypatch):
    monkeypatch.setenv("FLAREPP_NO_FAST_PATH", "1")
    w = inp.Workload("flare-online", 2, 900, 64, 4, 40, "f32", "normal")
    _check_flare(w, inp.make_inputs(w, 6, seed_scale=4.0), "online", centred_gate=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_flare_unfused_path(monkeypatch, dtype):
    monkeypatch.setenv("FLAREPP_UNFUSED", "1")
    w = inp.Workload("flare-unfused", 2, 300, 64, 4, 40, dtype, "normal")
    _check_flare(w, inp.make_inputs(w, 7, seed_scale=4.0), "unfused", centred_gate=(dtype == "f32"))


def test_flare_equals_flarepp_given_its_synthesised_queries():
    # FLARE++ is FLARE run with Q(X) as the query set (Sec. 3.2): feed the
    # GPU mixer's own Q(X) (batch entry 0) to the GPU FLARE and compare O
    w = inp.Workload("flare-eq", 1, 2000, 64, 4, 32, "f32", "normal")
    d = inp.make_inputs(w, 8, seed_scale=4.0)
    t = upload(d, w)
    O, Q, Z, Y = fp.flarepp_mixer_forward_debug(t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"],
                                                t["seeds"], H=w.H)
    Of = fp.flarepp_flare_forward(t["X"], t["Wk"], t["Wv"], t["Wo"], Q[0].contiguous(), H=w.H)
    torch.cuda.synchronize()
    e = assert_close("O", Of.cpu().numpy(), O.cpu().numpy(), TOL["f32"], "flare-vs-flarepp")
    assert e <= TOL["f32"]


def test_flare_deterministic_bitwise():
    w = inp.Workload("flare-det", 2, 5000, 128, 8, 128, "bf16", "normal")
    t = upload(inp.make_inputs(w, 9), w)
    a = fp.flarepp_flare_forward(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H)
    b = fp.flarepp_flare_forward(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["tiny", "grid2d"])
def test_shared_projection_variant(name):
    # K~, V~ tied to K, V (the variant of App. C.2): the oracle's mixer with
    # W~_K = W_K and W~_V = W_V, and bitwise the mixer entry point given the
    # tied weights
    w = inp.workload(name)
    d = inp.make_inputs(w, 11, seed_scale=4.0)
    print(f"[case] shared {inp.describe(w)}", flush=True)
    t = upload(d, w)
    O = fp.flarepp_mixer_forward_shared(t["X"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H)
    O2 = fp.flarepp_mixer_forward(t["X"], t["Wk"], t["Wv"], t["Wk"], t["Wv"], t["Wo"], t["seeds"], H=w.H)
    torch.cuda.synchronize()
    assert torch.equal(O, O2)
    ref = orc.mixer_forward(d["X"], d["Wk"], d["Wv"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], w.H)
    assert_close("O", O.float().cpu().numpy(), ref["O"], TOL[w.dtype], "shared")

"""The allocation-free mixer forward (flarepp_mixer_forward_noalloc), through
the C ABI: its workspace is the library's own scratch array, so it must
reproduce flarepp_mixer_forward (same kernels, caller workspace) bit for bit,
call after call, including a second, smaller call that runs over what the
first one left in the array."""

import numpy as np
import pytest
import torch

from oracle import flarepp_oracle as orc
from paper_2608_11519_amd import flarepp as fp
from paper_2608_11519_amd import inputs as inp

from gpu_util import TOL, assert_close, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp.load()
    yield


def _both(w, seed, seed_scale):
    d = inp.make_inputs(w, seed, seed_scale=seed_scale)
    t = upload(d, w)
    args = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])
    ref = fp.flarepp_mixer_forward(*args, H=w.H)
    got = fp.flarepp_mixer_forward_noalloc(*args, H=w.H)
    torch.cuda.synchronize()
    return d, got, ref


def test_noalloc_equals_the_workspace_entry_point_on_two_calls_in_a_row():
    cases = [(inp.workload("grid2d"), 50, 1.0), (inp.Workload("noalloc-small", 1, 777, 64, 4, 40, "bf16", "normal"), 51, 4.0)]
    assert cases[1][0].B * cases[1][0].N < cases[0][0].B * cases[0][0].N
    for w, seed, sc in cases:
        print(f"[case] noalloc {inp.describe(w, seed)}", flush=True)
        assert fp.flarepp_mixer_workspace_bytes(fp.BF16, w.B, w.N, w.C, w.H, w.M) <= fp.flarepp_mixer_noalloc_max_bytes()
        d, got, ref = _both(w, seed, sc)
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), "bitwise equal to flarepp_mixer_forward"
        if w.B * w.N <= 4096:  # and within the bf16 gate of the oracle
            r = orc.mixer_forward(d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H)
            assert_close("O", got.float().cpu().numpy(), r["O"], TOL[w.dtype], "noalloc")


def test_noalloc_fp32_and_the_larger_shape_again():
    # the fp32 path, then the first shape once more over what the small call left
    w = inp.workload("tiny")
    _, got, ref = _both(w, 52, 4.0)
    assert torch.equal(got, ref)
    w = inp.Workload("noalloc-again", 2, 5000, 128, 8, 128, "bf16", "normal")
    _, got, ref = _both(w, 53, 4.0)
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))

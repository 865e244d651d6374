"""The mixer captured into a HIP graph (as the benchmark replays it): every
replay, with eager work and synchronisations in between, must reproduce the
eager result bit for bit (the library records no memset nodes)."""

import pytest
import torch

from paper_2608_11519_amd import flarepp as fp
from paper_2608_11519_amd import inputs as inp

from gpu_util import upload

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_graph_replays_match_eager(dtype):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = inp.Workload("graph", 2, 3000, 128, 8, 96, dtype, "normal")
    t = upload(inp.make_inputs(w, 21, seed_scale=4.0), w)
    other = upload(inp.make_inputs(w, 22), w)
    args = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])
    dcode = fp.BF16 if dtype == "bf16" else fp.F32
    ws = torch.empty(fp.flarepp_mixer_workspace_bytes(dcode, w.B, w.N, w.C, w.H, w.M),
                     dtype=torch.uint8, device="cuda")
    eager = fp.flarepp_mixer_forward(*args, H=w.H, ws=ws).clone()
    torch.cuda.synchronize()
    O = torch.empty_like(eager)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fp.flarepp_mixer_forward(*args, H=w.H, out=O, ws=ws)
    for i in range(4):
        O.zero_()
        # eager work between replays that reuses the same workspace
        fp.flarepp_mixer_forward(other["X"], other["Wk"], other["Wv"], other["Wkt"], other["Wvt"],
                                 other["Wo"], other["seeds"], H=w.H, ws=ws)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(O.view(torch.int16 if dtype == "bf16" else torch.int32),
                           eager.view(torch.int16 if dtype == "bf16" else torch.int32)), f"replay {i}"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_single_stage_reruns_reproduce_the_forward(dtype):
    """flarepp_mixer_stage re-runs one stage on the workspace of a complete
    forward: every stage run alone (in order, then in reverse) leaves O
    bit-identical to the forward's."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = inp.Workload("stages", 2, 1500, 128, 8, 64, dtype, "normal")
    t = upload(inp.make_inputs(w, 23, seed_scale=4.0), w)
    args = (t["X"], t["Wk"], t["Wv"], t["Wkt"], t["Wvt"], t["Wo"], t["seeds"])
    dcode = fp.BF16 if dtype == "bf16" else fp.F32
    ws = torch.empty(fp.flarepp_mixer_workspace_bytes(dcode, w.B, w.N, w.C, w.H, w.M),
                     dtype=torch.uint8, device="cuda")
    O = fp.flarepp_mixer_forward(*args, H=w.H, ws=ws)
    ref = O.clone()
    view = torch.int16 if dtype == "bf16" else torch.int32
    order = list(range(1, fp.PROFILE_EVENTS)) + list(range(fp.PROFILE_EVENTS - 1, 0, -1))
    for k in order:
        fp.flarepp_mixer_stage(k, *args, H=w.H, out=O, ws=ws)
        torch.cuda.synchronize()
        assert torch.equal(O.view(view), ref.view(view)), f"stage {k}"
    with pytest.raises(fp.FlareppError):
        fp.flarepp_mixer_stage(0, *args, H=w.H, out=O, ws=ws)
    with pytest.raises(fp.FlareppError):
        fp.flarepp_mixer_stage(fp.PROFILE_EVENTS, *args, H=w.H, out=O, ws=ws)

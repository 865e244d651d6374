"""CPU tests of the Python binding's argument checks.

The kernels trust the sizes they are given, so the binding checks every
tensor against X before any call reaches the library: dtypes, shapes and
devices.  Each case here must raise TypeError or ValueError on the host; a
consistent set of (CPU) tensors passes the checks and is then refused only
because it does not live on the GPU, so nothing is ever launched.
"""

import pytest
import torch

from paper_2608_11519_amd import flarepp as fp

B, N, C, H, M = 2, 40, 64, 4, 8
D = C // H


def _args(dtype=torch.bfloat16):
    X = torch.zeros(B, N, C, dtype=dtype)
    W = {k: torch.zeros(C, C, dtype=dtype) for k in ("Wk", "Wv", "Wkt", "Wvt", "Wo")}
    seeds = torch.zeros(H, M, D, dtype=dtype)
    return X, W, seeds


def _mixer(X, W, seeds, **kw):
    return fp.flarepp_mixer_forward(X, W["Wk"], W["Wv"], W["Wkt"], W["Wvt"], W["Wo"], seeds, **kw)


@pytest.fixture(autouse=True)
def _lib():
    fp.load()  # the library loads without a GPU; no entry point below reaches it


def test_consistent_arguments_pass_the_checks_and_stop_at_the_device():
    X, W, seeds = _args()
    with pytest.raises(ValueError, match="GPU"):
        _mixer(X, W, seeds, H=H)


def test_rejects_unsupported_x():
    X, W, seeds = _args()
    with pytest.raises(TypeError):
        _mixer(X.half(), W, seeds, H=H)
    with pytest.raises(ValueError):
        _mixer(X[0], W, seeds, H=H)
    with pytest.raises(TypeError):
        _mixer(X.numpy() if X.dtype == torch.float32 else X.float().numpy(), W, seeds, H=H)


@pytest.mark.parametrize("h", [3, 0, -4])
def test_rejects_head_counts_that_do_not_divide_c(h):
    X, W, seeds = _args()
    with pytest.raises(ValueError):
        _mixer(X, W, seeds, H=h)


def test_rejects_a_non_integer_head_count():
    X, W, seeds = _args()
    with pytest.raises(TypeError):
        _mixer(X, W, seeds, H=4.0)


@pytest.mark.parametrize("name", ["Wk", "Wv", "Wkt", "Wvt", "Wo"])
def test_rejects_weights_of_the_wrong_shape_or_dtype(name):
    X, W, seeds = _args()
    bad = dict(W)
    bad[name] = torch.zeros(C, C + 1, dtype=X.dtype)
    with pytest.raises(ValueError):
        _mixer(X, bad, seeds, H=H)
    bad[name] = torch.zeros(C, C, dtype=torch.float32)  # twice the bytes the kernels read
    with pytest.raises(TypeError):
        _mixer(X, bad, seeds, H=H)


def test_rejects_seeds_of_the_wrong_shape_or_dtype():
    X, W, seeds = _args()
    with pytest.raises(ValueError):
        _mixer(X, W, torch.zeros(H, M, D + 1, dtype=X.dtype), H=H)
    with pytest.raises(ValueError):
        _mixer(X, W, torch.zeros(H + 1, M, D, dtype=X.dtype), H=H)
    with pytest.raises(ValueError):
        _mixer(X, W, torch.zeros(M, D, dtype=X.dtype), H=H)
    with pytest.raises(TypeError):
        _mixer(X, W, seeds.float(), H=H)


def test_rejects_outputs_and_workspaces_that_do_not_fit():
    X, W, seeds = _args()
    with pytest.raises(ValueError):
        _mixer(X, W, seeds, H=H, out=torch.zeros(B, N - 1, C, dtype=X.dtype))
    with pytest.raises(TypeError):
        _mixer(X, W, seeds, H=H, out=torch.zeros(B, N, C, dtype=torch.float32))
    with pytest.raises(TypeError):
        _mixer(X, W, seeds, H=H, ws=torch.zeros(1024, dtype=torch.float32))


def test_rejects_tensors_on_another_device():
    X, W, seeds = _args()
    bad = dict(W, Wo=torch.empty(C, C, dtype=X.dtype, device="meta"))
    with pytest.raises(ValueError, match="device"):
        _mixer(X, bad, seeds, H=H)


def test_flare_and_shared_variants_check_their_arguments():
    X, W, seeds = _args()
    with pytest.raises(ValueError):
        fp.flarepp_flare_forward(X, W["Wk"], W["Wv"], W["Wo"], torch.zeros(H, M, D - 1, dtype=X.dtype), H=H)
    with pytest.raises(TypeError):
        fp.flarepp_flare_forward(X, W["Wk"], W["Wv"].float(), W["Wo"], seeds, H=H)
    with pytest.raises(ValueError):
        fp.flarepp_mixer_forward_shared(X, W["Wk"], W["Wv"], torch.zeros(C, 2 * C, dtype=X.dtype), seeds, H=H)


def test_backward_checks_the_output_gradient_and_its_outputs():
    X, W, seeds = _args()
    args = (X, W["Wk"], W["Wv"], W["Wkt"], W["Wvt"], W["Wo"], seeds)
    with pytest.raises(ValueError):
        fp.flarepp_mixer_backward(*args, torch.zeros(B, N, C + 1, dtype=X.dtype), H=H)
    with pytest.raises(TypeError):
        fp.flarepp_mixer_backward(*args, torch.zeros(B, N, C, dtype=torch.float32), H=H)
    dO = torch.zeros(B, N, C, dtype=X.dtype)
    out = {"dX": torch.zeros(B, N, C), "dseeds": torch.zeros(H, M, D)}
    for k in ("dWk", "dWv", "dWkt", "dWvt", "dWo"):
        out[k] = torch.zeros(C, C)
    with pytest.raises(ValueError, match="GPU"):  # consistent: stops at the device
        fp.flarepp_mixer_backward(*args, dO, H=H, out=out)
    bad = dict(out, dWo=torch.zeros(C, C, dtype=torch.bfloat16))  # outputs are fp32
    with pytest.raises(TypeError):
        fp.flarepp_mixer_backward(*args, dO, H=H, out=bad)
    bad = dict(out, dseeds=torch.zeros(H, M + 1, D))
    with pytest.raises(ValueError):
        fp.flarepp_mixer_backward(*args, dO, H=H, out=bad)


def test_block_checks_its_norm_parameters():
    X, W, seeds = _args()
    g = torch.ones(C, dtype=X.dtype)
    with pytest.raises(ValueError):
        fp.flarepp_block_forward(X, torch.ones(C + 1, dtype=X.dtype), g, W["Wk"], W["Wv"], W["Wkt"], W["Wvt"],
                                 W["Wo"], seeds, H=H)
    with pytest.raises(TypeError):
        fp.flarepp_block_forward(X, g, g.float(), W["Wk"], W["Wv"], W["Wkt"], W["Wvt"], W["Wo"], seeds, H=H)


def test_route_checks_both_sides():
    tok = torch.zeros(B, H, N, D, dtype=torch.bfloat16)
    rt = torch.zeros(B, H, M, D)
    with pytest.raises(TypeError):  # route-side tensors are fp32
        fp.flarepp_route(fp.ENCODE, rt.bfloat16(), tok, tok)
    with pytest.raises(ValueError):
        fp.flarepp_route(fp.ENCODE, rt, tok, torch.zeros(B, H, N + 1, D, dtype=torch.bfloat16))
    with pytest.raises(ValueError):  # shared routes are one [1, H, M, D] set
        fp.flarepp_route(fp.ENCODE, rt, tok, tok, shared_routes=True)
    with pytest.raises(ValueError):
        fp.flarepp_route(fp.DECODE, tok, rt, torch.zeros(B, H, M + 1, D))
    with pytest.raises(ValueError):
        fp.flarepp_route(7, rt, tok, tok)
    with pytest.raises(ValueError, match="GPU"):
        fp.flarepp_route(fp.DECODE, tok, rt, rt)

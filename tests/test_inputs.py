"""Input generator: determinism, shapes, distributions and bf16 rounding."""

import numpy as np
import pytest

from paper_2608_11519_amd import inputs as inp


def test_same_seed_same_bytes():
    w = inp.workload("tiny")
    a = inp.make_inputs(w, 0)
    b = inp.make_inputs(w, 0)
    for k in a:
        assert a[k].tobytes() == b[k].tobytes()
    c = inp.make_inputs(w, 1)
    assert a["X"].tobytes() != c["X"].tobytes()


@pytest.mark.parametrize("name", ["tiny", "lra"])
def test_shapes_and_ranges(name):
    w = inp.workload(name, N=256) if name == "lra" else inp.workload(name)
    d = inp.make_inputs(w, 0)
    assert d["X"].shape == (w.B, w.N, w.C)
    assert d["seeds"].shape == (w.H, w.M, w.D)
    a = np.sqrt(3.0 / w.C)
    for k in ("Wk", "Wv", "Wkt", "Wvt", "Wo"):
        assert d[k].shape == (w.C, w.C)
        assert np.abs(d[k]).max() <= a * (1 + 2 ** -8)
        assert abs(d[k].std() - a / np.sqrt(3)) < 0.05 * a
    assert abs(d["seeds"].std() - 1 / np.sqrt(w.D)) < 0.1 / np.sqrt(w.D)


def test_embedding_workload_has_at_most_vocab_distinct_rows():
    w = inp.workload("lra", B=2, N=2048)
    X = inp.make_inputs(w, 0)["X"]
    rows = np.unique(X.reshape(-1, w.C), axis=0)
    assert len(rows) <= inp.EMBED_VOCAB


def test_fourier_workload_statistics():
    w = inp.workload("mesh", B=1, N=4000)
    X = inp.make_inputs(w, 0)["X"].astype(np.float64)
    # cos/sin features have mean ~0 and variance 1/2; noise adds 0.1
    assert abs(X.var() - 0.6) < 0.05


def test_bf16_rounding_ties_to_even_and_exactness():
    # values exactly representable in bf16 are unchanged
    v = np.array([1.0, -2.5, 3.0e-3, 65280.0, 0.0], dtype=np.float32)
    bf = inp.round_to_bf16(v)
    np.testing.assert_array_equal(inp.round_to_bf16(bf), bf)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even -> 1
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20], dtype=np.float32)
    np.testing.assert_array_equal(inp.round_to_bf16(x), [1.0, 1 + 2 ** -6, 1 + 2 ** -7])
    # bits round-trip
    bits = inp.bf16_bits(bf)
    np.testing.assert_array_equal(inp.bits_to_f32(bits), bf)


def test_bf16_storage_matches_torch_rounding():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    v = (rng.standard_normal(100000) * 10).astype(np.float32)
    mine = inp.round_to_bf16(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(mine, ref)

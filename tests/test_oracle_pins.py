"""Pins for the float64 oracle, checked on the CPU.

Each test checks the oracle against something other than itself: a
hand-derived worked example with exact rational answers, brute-force loops
with ``math.fsum``, PyTorch's own scaled_dot_product_attention (the paper
states that the whole mixer is three standard SDPA calls, Sec. 3.2 and
Fig. 1), closed forms, and the structural facts the paper states (rank <= M,
row-stochastic routing factors, token-order independence, the exact
split-key merge of App. A.2-A.3).
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import flarepp_oracle as orc
from paper_2608_11519_amd import inputs as inp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ---------------------------------------------------------------------------
# worked example with exact answers
# ---------------------------------------------------------------------------

def _worked_example():
    g = json.load(open(os.path.join(GOLDEN, "worked_example_rational.json")))
    B, N, C, H, M = g["B"], g["N"], g["C"], g["H"], g["M"]
    w, v, u, alpha = g["w"], g["v"], g["u"], g["alpha"]
    D = C // H
    trip = [(math.sqrt(3.0) * math.log(w[n]), v[n], u[n]) for n in range(N)]
    X = np.zeros((B, N, C))
    for n in range(N):
        X[0, n, 0:3] = trip[n]
        X[0, n, 3:6] = trip[(n + 1) % N]
    X[1] = X[0, ::-1]
    Wk = np.zeros((C, C)); Wv = np.zeros((C, C))
    Wkt = np.zeros((C, C)); Wvt = np.zeros((C, C))
    for o in (0, 3):
        Wkt[o + 0, o + 0] = 1
        Wk[o + 0, o + 0] = 1
        Wvt[o + 1, o + 0] = 1
        Wv[o + 2, o + 0] = 1
        Wv[o + 1, o + 2] = 1
    Wo = np.array(g["Wo"], dtype=np.float64)
    seeds = np.zeros((H, M, D))
    seeds[:, :, 0] = alpha
    return g, X, Wk, Wv, Wkt, Wvt, Wo, seeds


def test_worked_example_exact_values():
    g, X, Wk, Wv, Wkt, Wvt, Wo, seeds = _worked_example()
    r = orc.mixer_forward(X, Wk, Wv, Wkt, Wvt, Wo, seeds, g["H"])
    B, N, H, M = g["B"], g["N"], g["H"], g["M"]
    q1 = [float(Fraction(s)) for s in g["Q_first_coord"]]
    zr = [[float(Fraction(s)) for s in row] for row in g["Z_route"]]
    lse = [math.log(6.0), math.log(14.0)]
    for b in range(B):
        for h in range(H):
            np.testing.assert_allclose(r["Q"][b, h, :, 0], q1, rtol=0, atol=1e-12)
            np.testing.assert_allclose(r["Q"][b, h, :, 1:], 0.0, atol=1e-12)
            np.testing.assert_allclose(r["Z"][b, h], zr, rtol=0, atol=1e-12)
            np.testing.assert_allclose(r["L1"][b, h], lse, atol=1e-12)
            np.testing.assert_allclose(r["L2"][b, h], lse, atol=1e-12)
    # Y per token from its w value; head 1 sees the rotated token, batch 1
    # the reversed order
    w = g["w"]
    Yexp = np.zeros((B, N, 6), dtype=object)
    for n in range(N):
        y0 = [Fraction(s) for s in g["Y_by_w"][str(w[n])]]
        y1 = [Fraction(s) for s in g["Y_by_w"][str(w[(n + 1) % N])]]
        Yexp[0, n, 0:3] = y0
        Yexp[0, n, 3:6] = y1
    Yexp[1] = Yexp[0, ::-1]
    np.testing.assert_allclose(r["Y"], Yexp.astype(np.float64), atol=1e-12)
    # O = Y @ Wo in exact arithmetic
    Wo_f = [[Fraction(int(c)) for c in row] for row in g["Wo"]]
    for b in range(B):
        for n in range(N):
            for j in range(6):
                ex = sum(Yexp[b, n, i] * Wo_f[i][j] for i in range(6))
                assert abs(r["O"][b, n, j] - float(ex)) < 1e-11


# ---------------------------------------------------------------------------
# project
# ---------------------------------------------------------------------------

def test_project_explicit_loops():
    rng = _rng(1)
    B, N, C, H = 2, 3, 6, 3
    D = C // H
    X = rng.standard_normal((B, N, C))
    W = rng.standard_normal((C, C))  # not symmetric: a transposed W fails
    K = orc.project(X, W, H)
    assert K.shape == (B, H, N, D)
    for b in range(B):
        for h in range(H):
            for n in range(N):
                for d in range(D):
                    ref = math.fsum(X[b, n, c] * W[c, h * D + d] for c in range(C))
                    assert abs(K[b, h, n, d] - ref) < 1e-13


def test_merge_heads_layout():
    rng = _rng(2)
    Yh = rng.standard_normal((2, 3, 4, 5))
    Y = orc.merge_heads(Yh)
    for b in range(2):
        for h in range(3):
            for n in range(4):
                for d in range(5):
                    assert Y[b, n, h * 5 + d] == Yh[b, h, n, d]


# ---------------------------------------------------------------------------
# SDPA
# ---------------------------------------------------------------------------

def _brute_sdpa(Q, K, V):
    Nq, D = Q.shape
    Nk = K.shape[0]
    s = 1.0 / math.sqrt(D)
    out = np.zeros((Nq, V.shape[1]))
    L = np.zeros(Nq)
    for i in range(Nq):
        sc = [s * math.fsum(Q[i, d] * K[j, d] for d in range(D)) for j in range(Nk)]
        m = max(sc)
        e = [math.exp(x - m) for x in sc]
        den = math.fsum(e)
        for c in range(V.shape[1]):
            out[i, c] = math.fsum(e[j] * V[j, c] for j in range(Nk)) / den
        L[i] = m + math.log(den)
    return out, L


@pytest.mark.parametrize("Nq,Nk,D", [(3, 5, 4), (4, 2, 16), (1, 7, 3), (6, 1, 2)])
def test_sdpa_bruteforce(Nq, Nk, D):
    rng = _rng(Nq * 100 + Nk)
    Q = rng.standard_normal((Nq, D)) * 2
    K = rng.standard_normal((Nk, D))
    V = rng.standard_normal((Nk, D + 1))
    out, L = orc.sdpa(Q, K, V)
    ref, Lref = _brute_sdpa(Q, K, V)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)
    np.testing.assert_allclose(L, Lref, rtol=0, atol=1e-13)


def _torch_sdpa(Q, K, V):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))
    return torch.nn.functional.scaled_dot_product_attention(t(Q), t(K), t(V)).numpy()


@pytest.mark.parametrize("shape", [((2, 3, 8, 16), (2, 3, 50, 16)),
                                   ((1, 2, 40, 32), (1, 2, 9, 32)),
                                   ((4, 1, 5, 64), (4, 1, 300, 64))])
def test_sdpa_matches_library(shape):
    qs, ks = shape
    rng = _rng(7)
    Q = rng.standard_normal(qs)
    K = rng.standard_normal(ks)
    V = rng.standard_normal(ks)
    out, _ = orc.sdpa(Q, K, V)
    np.testing.assert_allclose(out, _torch_sdpa(Q, K, V), rtol=0, atol=1e-12)


def test_sdpa_long_key_axis_matches_library():
    # more keys than one oracle chunk: exercises the two-pass chunked path
    rng = _rng(8)
    Q = rng.standard_normal((1, 2, 6, 16)) * 3
    K = rng.standard_normal((1, 2, 20011, 16))
    V = rng.standard_normal((1, 2, 20011, 16))
    out, L = orc.sdpa(Q, K, V)
    np.testing.assert_allclose(out, _torch_sdpa(Q, K, V), rtol=0, atol=1e-12)
    S = (Q @ np.swapaxes(K, -1, -2)) / 4.0
    Lref = np.log(np.exp(S - S.max(-1, keepdims=True)).sum(-1)) + S.max(-1)
    np.testing.assert_allclose(L, Lref, atol=1e-11)


def test_sdpa_many_queries_matches_library():
    # more queries than one oracle chunk (decode-shaped call)
    rng = _rng(9)
    Kt = rng.standard_normal((1, 1, 40000, 16))
    Q = rng.standard_normal((1, 1, 12, 16))
    Z = rng.standard_normal((1, 1, 12, 16))
    out, _ = orc.sdpa(Kt, Q, Z)
    np.testing.assert_allclose(out, _torch_sdpa(Kt, Q, Z), rtol=0, atol=1e-12)


def test_sdpa_shift_invariance_encode_and_decode():
    rng = _rng(10)
    D = 16
    Qr = rng.standard_normal((8, D))
    K = rng.standard_normal((100, D))
    V = rng.standard_normal((100, D))
    u = rng.standard_normal(D) * 40.0  # large shift -> large logits
    a, _ = orc.sdpa(Qr, K, V)
    b, _ = orc.sdpa(Qr, K + u[None], V)  # constant along keys for each query
    np.testing.assert_allclose(a, b, atol=1e-11)
    Z = rng.standard_normal((8, D))
    c, _ = orc.sdpa(K, Qr, Z)
    d, _ = orc.sdpa(K, Qr + u[None], Z)  # constant along routes per token
    np.testing.assert_allclose(c, d, atol=1e-11)


def test_sdpa_constant_values_and_one_hot_limit():
    rng = _rng(11)
    D = 16
    Q = rng.standard_normal((5, D))
    K = rng.standard_normal((30, D))
    V = np.full((30, D), 3.25)
    out, _ = orc.sdpa(Q, K, V)
    np.testing.assert_allclose(out, 3.25, atol=1e-13)
    # one-hot limit: unit-norm keys, query lambda * k_j picks v_j
    Ku = K / np.linalg.norm(K, axis=1, keepdims=True)
    V = rng.standard_normal((30, D))
    for j in (0, 13, 29):
        q = (2000.0 * Ku[j])[None]
        o, _ = orc.sdpa(q, Ku, V)
        np.testing.assert_allclose(o[0], V[j], atol=1e-9)


def test_sdpa_empty_keys():
    out, L = orc.sdpa(np.ones((3, 4)), np.zeros((0, 4)), np.zeros((0, 4)))
    assert np.all(out == 0) and np.all(np.isneginf(L))


# ---------------------------------------------------------------------------
# split-key merge
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("bounds", [[0, 17, 40, 100], [0, 0, 50, 50, 100],
                                    [0, 100], [0, 1, 2, 3, 99, 100, 100]])
def test_split_merge_identity(bounds):
    rng = _rng(12)
    Qr = rng.standard_normal((2, 6, 16)) * 4
    K = rng.standard_normal((2, 100, 16))
    V = rng.standard_normal((2, 100, 16))
    full, Lf = orc.sdpa(Qr, K, V)
    parts = orc.partial_encode(Qr, K, V, bounds)
    for (O, L), a, b in zip(parts, bounds[:-1], bounds[1:]):
        if a == b:
            assert np.all(O == 0) and np.all(np.isneginf(L))
            assert not np.any(np.isnan(O))
    Z, L = orc.split_merge(parts)
    np.testing.assert_allclose(Z, full, atol=1e-12)
    np.testing.assert_allclose(L, Lf, atol=1e-12)


def test_split_merge_rejects_all_empty():
    z = np.zeros((2, 3))
    with pytest.raises(ValueError):
        orc.split_merge([(z, np.full(2, -np.inf)), (z, np.full(2, -np.inf))])


# ---------------------------------------------------------------------------
# whole mixer
# ---------------------------------------------------------------------------

def _small(seed=0, B=2, N=40, C=32, H=2, M=6, seed_scale=1.0):
    w = inp.Workload("t", B, N, C, H, M, "f32", "normal")
    d = inp.make_inputs(w, seed, seed_scale=seed_scale)
    return w, d


def _args(d):
    return (d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"])


def test_mixer_is_three_library_sdpa_calls():
    w, d = _small(seed=3, seed_scale=8.0)
    r = orc.mixer_forward(*_args(d), w.H)
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    X = t(d["X"])
    B, N, C, H, D = w.B, w.N, w.C, w.H, w.D

    def heads(W):  # [B,N,C] -> [B,H,N,D] with contiguous head channels
        return (X @ t(W)).view(B, N, H, D).permute(0, 2, 1, 3).contiguous()

    K, V, Kt, Vt = heads(d["Wk"]), heads(d["Wv"]), heads(d["Wkt"]), heads(d["Wvt"])
    sd = torch.nn.functional.scaled_dot_product_attention
    seeds = t(d["seeds"]).unsqueeze(0).expand(B, -1, -1, -1).contiguous()
    Q = sd(seeds, Kt, Vt)
    Z = sd(Q, K, V)
    Y = sd(K, Q, Z).permute(0, 2, 1, 3).reshape(B, N, C)
    O = Y @ t(d["Wo"])
    np.testing.assert_allclose(r["Q"], Q.numpy(), atol=1e-12)
    np.testing.assert_allclose(r["Z"], Z.numpy(), atol=1e-12)
    np.testing.assert_allclose(r["Y"], Y.numpy(), atol=1e-12)
    np.testing.assert_allclose(r["O"], O.numpy(), atol=1e-12)


def test_materialised_operator_rank_and_rows():
    w, d = _small(seed=4, B=1, N=48, C=32, H=2, M=5, seed_scale=8.0)
    r = orc.mixer_forward(*_args(d), w.H)
    mo = orc.materialised_operator(d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["seeds"], w.H)
    Yh = mo["W_eff"] @ mo["V"]  # [B,H,N,D]
    np.testing.assert_allclose(orc.merge_heads(Yh), r["Y"], atol=1e-12)
    np.testing.assert_allclose(mo["Q"], r["Q"], atol=1e-12)
    # routing factors are row-stochastic: W_enc over tokens, W_dec over routes
    np.testing.assert_allclose(mo["W_enc"].sum(-1), 1.0, atol=1e-14)
    np.testing.assert_allclose(mo["W_dec"].sum(-1), 1.0, atol=1e-14)
    np.testing.assert_allclose(mo["W_eff"].sum(-1), 1.0, atol=1e-13)
    assert mo["W_enc"].shape[-2:] == (w.M, w.N)
    assert mo["W_dec"].shape[-2:] == (w.N, w.M)
    # rank <= M (Sec. 3.2, Eq. (12))
    for h in range(w.H):
        sv = np.linalg.svd(mo["W_eff"][0, h], compute_uv=False)
        assert sv[w.M] / sv[0] < 1e-10
        assert sv[w.M - 1] / sv[0] > 1e-8  # and generically exactly M


def test_permutation_equivariance():
    w, d = _small(seed=5, seed_scale=8.0)
    r = orc.mixer_forward(*_args(d), w.H)
    perm = _rng(55).permutation(w.N)
    d2 = dict(d)
    d2["X"] = d["X"][:, perm]
    r2 = orc.mixer_forward(*_args(d2), w.H)
    np.testing.assert_allclose(r2["O"], r["O"][:, perm], atol=1e-12)
    np.testing.assert_allclose(r2["Q"], r["Q"], atol=1e-12)
    np.testing.assert_allclose(r2["Z"], r["Z"], atol=1e-12)


def test_single_route_broadcasts_latent():
    w, d = _small(seed=6, M=1)
    r = orc.mixer_forward(*_args(d), w.H)
    D = w.D
    for h in range(w.H):
        np.testing.assert_allclose(
            r["Y"][:, :, h * D:(h + 1) * D],
            np.broadcast_to(r["Z"][:, h, 0][:, None, :], (w.B, w.N, D)), atol=1e-13)


def test_single_token_reduces_to_value_path():
    w, d = _small(seed=7, N=1)
    r = orc.mixer_forward(*_args(d), w.H)
    X = d["X"].astype(np.float64)
    ref = X @ d["Wv"].astype(np.float64) @ d["Wo"].astype(np.float64)
    np.testing.assert_allclose(r["O"], ref, atol=1e-13)


def test_zero_seeds_give_mean_queries_and_constant_output():
    w = inp.Workload("t", 2, 30, 32, 2, 4, "f32", "normal")
    d = inp.make_inputs(w, 8, zero_seeds=True)
    r = orc.mixer_forward(*_args(d), w.H)
    Vt = orc.project(d["X"], d["Wvt"], w.H)
    mean = Vt.mean(axis=2)  # [B,H,D]
    np.testing.assert_allclose(r["Q"], np.broadcast_to(mean[:, :, None], r["Q"].shape), atol=1e-13)
    np.testing.assert_allclose(r["Y"], np.broadcast_to(r["Y"][:, :1], r["Y"].shape), atol=1e-13)


def test_batch_independence_and_head_locality():
    w, d = _small(seed=9, B=3, seed_scale=4.0)
    r = orc.mixer_forward(*_args(d), w.H)
    # batch independence
    d2 = dict(d)
    X2 = d["X"].copy()
    X2[1] += 1.0
    d2["X"] = X2
    r2 = orc.mixer_forward(*_args(d2), w.H)
    np.testing.assert_array_equal(r2["O"][0], r["O"][0])
    np.testing.assert_array_equal(r2["O"][2], r["O"][2])
    assert np.abs(r2["O"][1] - r["O"][1]).max() > 1e-3
    # head locality: changing head 1's key weights leaves head 0's Y alone
    D = w.D
    d3 = dict(d)
    Wk3 = d["Wk"].copy()
    Wk3[:, D:2 * D] *= -1.5
    d3["Wk"] = Wk3
    r3 = orc.mixer_forward(*_args(d3), w.H)
    np.testing.assert_array_equal(r3["Y"][:, :, :D], r["Y"][:, :, :D])
    assert np.abs(r3["Y"][:, :, D:] - r["Y"][:, :, D:]).max() > 1e-4


def test_flare_special_case_matches_flarepp_with_synthesised_queries():
    # FLARE++ equals FLARE run with Q(X) as its learned query set (Sec. 3.2)
    w, d = _small(seed=10, B=1, seed_scale=6.0)
    r = orc.mixer_forward(*_args(d), w.H)
    f = orc.flare_forward(d["X"], d["Wk"], d["Wv"], d["Wo"], r["Q"][0], w.H)
    np.testing.assert_allclose(f["O"], r["O"], atol=1e-12)
    np.testing.assert_allclose(f["Z"], r["Z"], atol=1e-12)


def test_flare_matches_two_library_sdpa_calls():
    # FLARE (Sec. 3.1, Eq. (5)): Z = SDPA(Q, K, V), Y = SDPA(K, Q, Z), merge with W_O;
    # checked against torch's own SDPA in float64
    w, d = _small(seed=12, B=2, seed_scale=4.0)
    H = w.H
    Qlat = d["seeds"].astype(np.float64)
    f = orc.flare_forward(d["X"], d["Wk"], d["Wv"], d["Wo"], Qlat, H)
    X = torch.from_numpy(d["X"].astype(np.float64))
    B, N, C = X.shape
    D = C // H
    K = (X @ torch.from_numpy(d["Wk"].astype(np.float64))).reshape(B, N, H, D).transpose(1, 2)
    V = (X @ torch.from_numpy(d["Wv"].astype(np.float64))).reshape(B, N, H, D).transpose(1, 2)
    Q = torch.from_numpy(Qlat)[None].expand(B, -1, -1, -1)
    Z = torch.nn.functional.scaled_dot_product_attention(Q, K, V)
    Y = torch.nn.functional.scaled_dot_product_attention(K, Q, Z)
    Ym = Y.transpose(1, 2).reshape(B, N, C)
    O = Ym @ torch.from_numpy(d["Wo"].astype(np.float64))
    np.testing.assert_allclose(f["Z"], Z.numpy(), atol=1e-12)
    np.testing.assert_allclose(f["Y"], Ym.numpy(), atol=1e-12)
    np.testing.assert_allclose(f["O"], O.numpy(), atol=1e-12)


def test_flare_operator_has_rank_at_most_m_and_stochastic_rows():
    # W_eff = W_dec W_enc (Sec. 3.1, Eq. (6)) with fixed queries: Y_h = W_eff V_h,
    # rank <= M, rows sum to one
    w, d = _small(seed=13, B=1, N=24, C=16, H=2, M=3, seed_scale=3.0)
    H, D, M = w.H, w.D, w.M
    f = orc.flare_forward(d["X"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], H)
    K = orc.project(d["X"], d["Wk"], H)[0]
    V = orc.project(d["X"], d["Wv"], H)[0]
    for h in range(H):
        S = d["seeds"][h].astype(np.float64) @ K[h].T / math.sqrt(D)  # M x N
        enc = np.exp(S - S.max(axis=1, keepdims=True))
        enc /= enc.sum(axis=1, keepdims=True)
        dec = np.exp(S.T - S.T.max(axis=1, keepdims=True))
        dec /= dec.sum(axis=1, keepdims=True)
        Weff = dec @ enc
        np.testing.assert_allclose(Weff.sum(axis=1), 1.0, atol=1e-13)
        sv = np.linalg.svd(Weff, compute_uv=False)
        assert sv[M] / sv[0] < 1e-10
        np.testing.assert_allclose(f["Y"][0, :, h * D:(h + 1) * D], Weff @ V[h], atol=1e-12)


def test_flare_single_route_broadcasts_the_latent():
    # with M = 1 the decode softmax has one entry: every token receives Z
    w, d = _small(seed=14, B=2, M=1, seed_scale=2.0)
    f = orc.flare_forward(d["X"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], w.H)
    D = w.D
    for h in range(w.H):
        np.testing.assert_allclose(f["Y"][:, :, h * D:(h + 1) * D], np.broadcast_to(
            f["Z"][:, h, 0][:, None, :], f["Y"][:, :, h * D:(h + 1) * D].shape), atol=1e-13)


def test_lse_outputs_match_bruteforce():
    w, d = _small(seed=11, B=1, N=9, C=8, H=2, M=3, seed_scale=5.0)
    r = orc.mixer_forward(*_args(d), w.H)
    Kt = orc.project(d["X"], d["Wkt"], w.H)
    for h in range(w.H):
        _, L = _brute_sdpa(d["seeds"][h].astype(np.float64), Kt[0, h], Kt[0, h])
        np.testing.assert_allclose(r["L1"][0, h], L, atol=1e-13)


# ---------------------------------------------------------------------------
# backward (App. A.5)
# ---------------------------------------------------------------------------

def _library_mixer_grads(d, w, dO):
    """Gradients of <O, dO> through three library SDPA calls, by autograd in
    float64 (independent of the oracle's explicit backward)."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64)).clone().requires_grad_(True)
    X, Wk, Wv, Wkt, Wvt, Wo, seeds = (t(d[k]) for k in ("X", "Wk", "Wv", "Wkt", "Wvt", "Wo", "seeds"))
    B, N, C, H, D = w.B, w.N, w.C, w.H, w.D

    def heads(W):
        return (X @ W).view(B, N, H, D).permute(0, 2, 1, 3)

    sd = torch.nn.functional.scaled_dot_product_attention
    K, V, Kt, Vt = heads(Wk), heads(Wv), heads(Wkt), heads(Wvt)
    Q = sd(seeds.unsqueeze(0).expand(B, -1, -1, -1), Kt, Vt)
    Z = sd(Q, K, V)
    Y = sd(K, Q, Z).permute(0, 2, 1, 3).reshape(B, N, C)
    O = Y @ Wo
    (O * torch.from_numpy(dO)).sum().backward()
    return {"dX": X.grad, "dWk": Wk.grad, "dWv": Wv.grad, "dWkt": Wkt.grad, "dWvt": Wvt.grad,
            "dWo": Wo.grad, "dseeds": seeds.grad}


@pytest.mark.parametrize("seed,seed_scale", [(11, 1.0), (12, 8.0)])
def test_backward_matches_library_autograd(seed, seed_scale):
    w, d = _small(seed=seed, seed_scale=seed_scale)
    dO = _rng(seed + 100).standard_normal((w.B, w.N, w.C))
    r = orc.mixer_backward(*_args(d), w.H, dO)
    ref = _library_mixer_grads(d, w, dO)
    for k, v in ref.items():
        v = v.numpy()
        assert np.abs(r[k] - v).max() <= 1e-10 * max(1.0, np.abs(v).max()), k


def test_backward_directional_finite_difference():
    # <grad, u> against the central difference of <O(theta + e u), dO>
    w, d = _small(seed=13, seed_scale=4.0)
    rng = _rng(14)
    dO = rng.standard_normal((w.B, w.N, w.C))
    r = orc.mixer_backward(*_args(d), w.H, dO)
    keys = ("X", "Wk", "Wv", "Wkt", "Wvt", "Wo", "seeds")
    u = {k: rng.standard_normal(np.shape(d[k])) for k in keys}
    eps = 1e-5

    def f(sign):
        a = {k: np.asarray(d[k], dtype=np.float64) + sign * eps * u[k] for k in keys}
        return float((orc.mixer_forward(*(a[k] for k in keys), w.H)["O"] * dO).sum())

    fd = (f(1.0) - f(-1.0)) / (2 * eps)
    an = sum(float((r["d" + k] * u[k]).sum()) for k in keys)
    assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (fd, an)


def test_backward_single_token_closed_form():
    # N = 1: every softmax over tokens has one key, Q and Z are that token's
    # V~ and V, and O = X W_V W_O whatever the keys: the key, tilde and seed
    # gradients vanish and the rest is the two-GEMM chain rule
    w, d = _small(seed=15, N=1)
    dO = _rng(16).standard_normal((w.B, 1, w.C))
    r = orc.mixer_backward(*_args(d), w.H, dO)
    X, Wv, Wo = (np.asarray(d[k], dtype=np.float64) for k in ("X", "Wv", "Wo"))
    G = dO @ Wo.T
    np.testing.assert_allclose(r["dX"], G @ Wv.T, atol=1e-12)
    np.testing.assert_allclose(r["dWv"], np.einsum("bni,bno->io", X, G), atol=1e-12)
    np.testing.assert_allclose(r["dWo"], np.einsum("bni,bno->io", X @ Wv, dO), atol=1e-12)
    for k in ("dWk", "dWkt", "dWvt", "dseeds"):
        assert np.abs(r[k]).max() <= 1e-12, k


def _sdpa_case(seed, lead=(2, 3), Nq=5, Nk=7, D=4, Dv=3, scale=2.0):
    g = _rng(seed)
    Q = g.standard_normal(lead + (Nq, D)) * scale
    K = g.standard_normal(lead + (Nk, D))
    V = g.standard_normal(lead + (Nk, Dv))
    dO = g.standard_normal(lead + (Nq, Dv))
    O, L = orc.sdpa(Q, K, V)
    return Q, K, V, O, L, dO


def test_sdpa_backward_bruteforce_loops():
    # every gradient element from its scalar definition, summed with fsum
    Q, K, V, O, L, dO = _sdpa_case(21, lead=(), Nq=3, Nk=4, D=2, Dv=2)
    dQ, dK, dV = orc.sdpa_backward(Q, K, V, O, L, dO)
    s = 1.0 / math.sqrt(2)
    Nq, Nk = 3, 4
    P = [[math.exp(s * math.fsum(Q[i, t] * K[j, t] for t in range(2)) - L[i]) for j in range(Nk)] for i in range(Nq)]
    dP = [[math.fsum(dO[i, t] * V[j, t] for t in range(2)) for j in range(Nk)] for i in range(Nq)]
    c = [math.fsum(P[i][j] * dP[i][j] for j in range(Nk)) for i in range(Nq)]
    dS = [[P[i][j] * (dP[i][j] - c[i]) for j in range(Nk)] for i in range(Nq)]
    for j in range(Nk):
        for t in range(2):
            assert abs(dV[j, t] - math.fsum(P[i][j] * dO[i, t] for i in range(Nq))) < 1e-13
            assert abs(dK[j, t] - s * math.fsum(dS[i][j] * Q[i, t] for i in range(Nq))) < 1e-13
    for i in range(Nq):
        for t in range(2):
            assert abs(dQ[i, t] - s * math.fsum(dS[i][j] * K[j, t] for j in range(Nk))) < 1e-13


def test_sdpa_backward_invariants():
    Q, K, V, O, L, dO = _sdpa_case(22)
    dQ, dK, dV = orc.sdpa_backward(Q, K, V, O, L, dO)
    # adding one vector to every key shifts each query's scores by a
    # constant: the key gradients sum to zero
    assert np.abs(dK.sum(axis=-2)).max() < 1e-12
    # the softmax weights of a query sum to one: the value gradients sum to
    # the output gradients
    np.testing.assert_allclose(dV.sum(axis=-2), dO.sum(axis=-2), atol=1e-12)
    # constant values make the output independent of the scores
    Vc = np.ones_like(V) * 0.7
    Oc, Lc = orc.sdpa(Q, K, Vc)
    dQc, dKc, _ = orc.sdpa_backward(Q, K, Vc, Oc, Lc, dO)
    assert np.abs(dQc).max() < 1e-12 and np.abs(dKc).max() < 1e-12


def test_sdpa_backward_chunked_key_axis(monkeypatch):
    Q, K, V, O, L, dO = _sdpa_case(23, Nk=50)
    a = orc.sdpa_backward(Q, K, V, O, L, dO)
    monkeypatch.setattr(orc, "_KEY_CHUNK", 7)
    b = orc.sdpa_backward(Q, K, V, O, L, dO)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, atol=1e-13)


# ---------------------------------------------------------------------------
# the pre-norm residual block around the mixer
# ---------------------------------------------------------------------------

def test_layer_norm_matches_library():
    g = _rng(31)
    X = g.standard_normal((2, 7, 32)) * 3 + 1
    gamma, beta = g.standard_normal(32), g.standard_normal(32)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(X), (32,), torch.from_numpy(gamma),
                                         torch.from_numpy(beta), eps=1e-5).numpy()
    np.testing.assert_allclose(orc.layer_norm(X, gamma, beta, 1e-5), ref, atol=1e-12)


def test_block_is_residual_plus_mixer_of_library_layer_norm():
    w, d = _small(seed=32, seed_scale=4.0)
    g = _rng(33)
    gamma, beta = 1 + 0.1 * g.standard_normal(w.C), 0.1 * g.standard_normal(w.C)
    out = orc.block_forward(d["X"], gamma, beta, 1e-5, *_args(d)[1:], w.H)
    Xn = torch.nn.functional.layer_norm(torch.from_numpy(np.asarray(d["X"], dtype=np.float64)), (w.C,),
                                        torch.from_numpy(gamma), torch.from_numpy(beta), eps=1e-5).numpy()
    mix = orc.mixer_forward(Xn, *_args(d)[1:], w.H)["O"]
    np.testing.assert_allclose(out, np.asarray(d["X"], dtype=np.float64) + mix, atol=1e-12)
    # zero gamma and beta: the mixer sees zeros, every softmax is uniform and
    # its values are zero, so the block is the identity
    np.testing.assert_allclose(orc.block_forward(d["X"], 0 * gamma, 0 * beta, 1e-5, *_args(d)[1:], w.H),
                               np.asarray(d["X"], dtype=np.float64), atol=1e-12)


def test_shared_backward_matches_library_autograd_with_tied_weights():
    # K~ = K, V~ = V: autograd through one tensor used twice sums its two
    # gradients by itself
    w, d = _small(seed=34, seed_scale=4.0)
    dO = _rng(35).standard_normal((w.B, w.N, w.C))
    tied = dict(d, Wkt=d["Wk"], Wvt=d["Wv"])
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64)).clone().requires_grad_(True)
    X, Wk, Wv, Wo, seeds = (t(d[k]) for k in ("X", "Wk", "Wv", "Wo", "seeds"))
    B, N, C, H, D = w.B, w.N, w.C, w.H, w.D
    heads = lambda W: (X @ W).view(B, N, H, D).permute(0, 2, 1, 3)
    sd = torch.nn.functional.scaled_dot_product_attention
    K, V = heads(Wk), heads(Wv)
    Q = sd(seeds.unsqueeze(0).expand(B, -1, -1, -1), K, V)
    Z = sd(Q, K, V)
    O = sd(K, Q, Z).permute(0, 2, 1, 3).reshape(B, N, C) @ Wo
    (O * torch.from_numpy(dO)).sum().backward()
    r = orc.mixer_backward_shared(d["X"], d["Wk"], d["Wv"], d["Wo"], d["seeds"], w.H, dO)
    for k, g in (("dX", X.grad), ("dWk", Wk.grad), ("dWv", Wv.grad), ("dWo", Wo.grad), ("dseeds", seeds.grad)):
        g = g.numpy()
        assert np.abs(r[k] - g).max() <= 1e-10 * max(1.0, np.abs(g).max()), k
    # and it is not the untied gradient: the tilde uses contribute
    u = orc.mixer_backward(*_args(tied), w.H, dO)
    assert np.abs(r["dWk"] - u["dWk"]).max() > 1e-6 * np.abs(r["dWk"]).max()


def test_block_backward_matches_library_autograd():
    w, d = _small(seed=36, seed_scale=4.0)
    g0 = _rng(37)
    gamma, beta = 1 + 0.2 * g0.standard_normal(w.C), 0.2 * g0.standard_normal(w.C)
    dO = g0.standard_normal((w.B, w.N, w.C))
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64)).clone().requires_grad_(True)
    X, ga, be, Wk, Wv, Wkt, Wvt, Wo, seeds = (t(v) for v in (d["X"], gamma, beta, d["Wk"], d["Wv"], d["Wkt"],
                                                             d["Wvt"], d["Wo"], d["seeds"]))
    B, N, C, H, D = w.B, w.N, w.C, w.H, w.D
    Xn = torch.nn.functional.layer_norm(X, (C,), ga, be, eps=1e-5)
    heads = lambda W: (Xn @ W).view(B, N, H, D).permute(0, 2, 1, 3)
    sd = torch.nn.functional.scaled_dot_product_attention
    Q = sd(seeds.unsqueeze(0).expand(B, -1, -1, -1), heads(Wkt), heads(Wvt))
    K = heads(Wk)
    Z = sd(Q, K, heads(Wv))
    O = X + sd(K, Q, Z).permute(0, 2, 1, 3).reshape(B, N, C) @ Wo
    (O * torch.from_numpy(dO)).sum().backward()
    r = orc.block_backward(d["X"], gamma, beta, 1e-5, *_args(d)[1:], w.H, dO)
    for k, v in (("dX", X), ("dgamma", ga), ("dbeta", be), ("dWk", Wk), ("dWv", Wv), ("dWkt", Wkt),
                 ("dWvt", Wvt), ("dWo", Wo), ("dseeds", seeds)):
        ref = v.grad.numpy()
        assert np.abs(r[k] - ref).max() <= 1e-10 * max(1.0, np.abs(ref).max()), k

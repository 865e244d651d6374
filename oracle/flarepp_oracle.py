"""Float64 CPU oracle for the FLARE++ mixer forward and backward.

TEST INFRASTRUCTURE ONLY.  This module is the correctness reference that the
HIP path is compared against.  Only the tests, the package's ``smoke()`` and
the CPU-baseline leg of the benchmark may import it; the product path never
calls it and shares no code with it.

It computes the plain definitions, in float64, in the paper's order:

* ``project``     K = X W per weight, heads are contiguous D-wide column
                  blocks (Sec. 3.1, Eq. (4); Sec. 3.2, Eqs. (7), (9)).
* ``sdpa``        rectangular scaled dot-product attention, softmax over the
                  keys, scale 1/sqrt(D) (Sec. 3.1, Eq. (3)).  Also returns the
                  row log-normaliser L = logsumexp of the scaled scores
                  (App. A.2, Eq. (20)).
* ``mixer_forward`` project; Q = SDPA(Q~, K~, V~) (Eq. (8));
                  Z = SDPA(Q, K, V) (Eq. (10)); Y = SDPA(K, Q, Z) (Eq. (11));
                  heads merged and multiplied by W_O (Sec. 3.1 after Eq. (2);
                  Fig. 1).
* ``split_merge`` the exact split-key merge of partial results
                  (App. A.2, Eqs. (22)-(23); stable form App. A.3,
                  Eqs. (24)-(28), including the empty-row convention).
* ``materialised_operator`` W_eff = W_dec W_enc per head (Sec. 3.1, Eq. (6);
                  Sec. 3.2, Eq. (12)), for small N only.
* ``sdpa_backward`` the gradient of one SDPA call from its global output and
                  log-normaliser (App. A.5): P = exp(s S - L), c = <dO, O>
                  per row, dV = P^T dO, dS = P (dO V^T - c), dK = s dS^T Q,
                  dQ = s dS K.
* ``block_forward`` the pre-norm residual block around the mixer,
                  X + mixer(LN(X)) (the residual stream the paper leaves
                  unchanged, Sec. 3.2); ``layer_norm`` normalises each token
                  over its channels with the biased variance.
* ``block_backward`` the block's gradients: the mixer's backward on the
                  normalised tokens, the layer norm's backward, the residual.
* ``mixer_backward`` the reverse pass of the whole mixer (App. A.5): W_O and
                  the merge, the decode (call 3), the physical-value encode
                  (call 2), the summed query gradient through the query
                  synthesis (call 1), the seeds (summed over the batch) and
                  the four projections.  ``mixer_backward_shared`` the same
                  with K~ = K, V~ = V (App. C.2): a tied weight's gradient
                  sums its two uses.

Readings of points the paper leaves open (all fixed here, in the same way as
in the input generator):

* head h owns channels [h D, (h+1) D) of every projection;
* weights are [C_in][C_out] and applied as X @ W; there are no biases;
* the scale is 1/sqrt(D) in all three calls, including the decode whose keys
  are the M routes;
* seeds are shared across the batch; Q(X) is per batch element;
* an empty key set gives L = -inf and a zero output (App. A.3).

The softmax over a long key axis is evaluated in key chunks as a plain
two-pass computation (pass 1: the exact row maximum; pass 2: exponentials,
their sum and the weighted sum of values).  Chunking only bounds memory; the
arithmetic is the textbook max-shifted softmax.

Every function here is pinned by CPU tests against facts independent of this
code (closed forms, brute force, a library SDPA, the structural invariants the
paper states); no function is "parity unpinned".
"""

from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

__all__ = [
    "project",
    "sdpa",
    "mixer_forward",
    "flare_forward",
    "split_merge",
    "partial_encode",
    "materialised_operator",
    "merge_heads",
    "split_heads",
    "sdpa_backward",
    "mixer_backward",
    "layer_norm",
    "block_forward",
    "mixer_backward_shared",
    "block_backward",
]

# Key chunk for the two-pass softmax and query chunk for independent rows;
# only bounds memory.
_KEY_CHUNK = 8192
_QUERY_CHUNK = 16384


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def project(X: np.ndarray, W: np.ndarray, H: int) -> np.ndarray:
    """Head-split projection ``X W`` (Sec. 3.1, Eq. (4); Sec. 3.2, Eq. (7)).

    X: [B, N, C]; W: [C, C] (out = X @ W).  Returns [B, H, N, D] where head h
    holds output channels [h D, (h+1) D).
    """
    X = _f64(X)
    W = _f64(W)
    B, N, C = X.shape
    if C % H:
        raise ValueError("C must be divisible by H")
    D = C // H
    Y = X @ W  # [B, N, C]
    return Y.reshape(B, N, H, D).transpose(0, 2, 1, 3).copy()


def merge_heads(Yh: np.ndarray) -> np.ndarray:
    """Concatenate heads: [B, H, N, D] -> [B, N, H*D] (Sec. 3.1, after Eq. (2))."""
    B, H, N, D = Yh.shape
    return Yh.transpose(0, 2, 1, 3).reshape(B, N, H * D).copy()


def split_heads(Y: np.ndarray, H: int) -> np.ndarray:
    """Inverse of ``merge_heads``: [B, N, H*D] -> [B, H, N, D]."""
    B, N, C = Y.shape
    return _f64(Y).reshape(B, N, H, C // H).transpose(0, 2, 1, 3).copy()


def sdpa(Q: np.ndarray, K: np.ndarray, V: np.ndarray,
         scale: float | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """Rectangular SDPA, softmax over the keys (Sec. 3.1, Eq. (3)).

    Q: [..., Nq, D]; K: [..., Nk, D]; V: [..., Nk, Dv]; leading dimensions
    broadcast.  Returns ``(out [..., Nq, Dv], L [..., Nq])`` where
    ``L = log sum_j exp(scale * q . k_j)`` (App. A.2, Eq. (20)).
    With no keys (Nk = 0) the output is zero and L = -inf (App. A.3).
    """
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    D = Q.shape[-1]
    s = 1.0 / math.sqrt(D) if scale is None else float(scale)
    Nq, Nk, Dv = Q.shape[-2], K.shape[-2], V.shape[-1]
    lead = np.broadcast_shapes(Q.shape[:-2], K.shape[:-2], V.shape[:-2])
    out = np.zeros(lead + (Nq, Dv))
    L = np.full(lead + (Nq,), -np.inf)
    if Nk == 0 or Nq == 0:
        return out, L
    for q0 in range(0, Nq, _QUERY_CHUNK):
        q = Q[..., q0:q0 + _QUERY_CHUNK, :]
        # pass 1: exact row maximum of the scaled scores
        mx = None
        for k0 in range(0, Nk, _KEY_CHUNK):
            S = s * (q @ np.swapaxes(K[..., k0:k0 + _KEY_CHUNK, :], -1, -2))
            cm = S.max(axis=-1)
            mx = cm if mx is None else np.maximum(mx, cm)
        # pass 2: exponentials, normaliser and weighted values
        den = 0.0
        num = 0.0
        for k0 in range(0, Nk, _KEY_CHUNK):
            S = s * (q @ np.swapaxes(K[..., k0:k0 + _KEY_CHUNK, :], -1, -2))
            E = np.exp(S - mx[..., None])
            den = den + E.sum(axis=-1)
            num = num + E @ V[..., k0:k0 + _KEY_CHUNK, :]
        out[..., q0:q0 + _QUERY_CHUNK, :] = num / den[..., None]
        L[..., q0:q0 + _QUERY_CHUNK] = mx + np.log(den)
    return out, L


def mixer_forward(X, Wk, Wv, Wkt, Wvt, Wo, seeds, H: int) -> Dict[str, np.ndarray]:
    """The FLARE++ mixer forward (Fig. 1; Sec. 3.2, Eqs. (7)-(11)).

    X: [B, N, C]; W*: [C, C]; seeds: [H, M, D].  Returns a dict with
    ``O [B,N,C]`` and the intermediates ``Q, Z [B,H,M,D]``, ``Y [B,N,C]``
    (heads merged, before W_O), ``L1, L2 [B,H,M]`` (log-normalisers of the
    two encode calls) and ``K, V, Kt, Vt [B,H,N,D]``.
    """
    X = _f64(X)
    seeds = _f64(seeds)
    B, N, C = X.shape
    if seeds.shape[0] != H or seeds.shape[2] * H != C:
        raise ValueError("seeds must be [H, M, C/H]")
    # project step (Fig. 1; Eqs. (7), (9))
    K = project(X, Wk, H)
    V = project(X, Wv, H)
    Kt = project(X, Wkt, H)
    Vt = project(X, Wvt, H)
    # call 1: query synthesis, softmax over the N tokens (Eq. (8));
    # the seeds are shared across the batch
    Q, L1 = sdpa(seeds[None], Kt, Vt)
    # call 2: encode, softmax over the N tokens (Eq. (10))
    Z, L2 = sdpa(Q, K, V)
    # call 3: decode, the tokens' keys query the M routes; softmax over M
    # (Eq. (11))
    Yh, _ = sdpa(K, Q, Z)
    Y = merge_heads(Yh)
    # merge: concatenated heads times W_O
    O = Y @ _f64(Wo)
    return {"O": O, "Q": Q, "Z": Z, "Y": Y, "L1": L1, "L2": L2,
            "K": K, "V": V, "Kt": Kt, "Vt": Vt}


def flare_forward(X, Wk, Wv, Wo, Qlat, H: int) -> Dict[str, np.ndarray]:
    """Fixed-query FLARE mixer (Sec. 3.1, Eqs. (4)-(5)): Z = SDPA(Q, K, V),
    Y = SDPA(K, Q, Z) with learned per-head queries Q [H, M, D]."""
    X = _f64(X)
    K = project(X, Wk, H)
    V = project(X, Wv, H)
    Qb = _f64(Qlat)[None]
    Z, L = sdpa(Qb, K, V)
    Yh, _ = sdpa(K, Qb, Z)
    Y = merge_heads(Yh)
    return {"O": Y @ _f64(Wo), "Z": Z, "Y": Y, "L": L}


def partial_encode(Qr, K, V, bounds: Sequence[int]) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Per-part encode on a split of the key axis (App. A.2, Eqs. (19)-(21)).

    ``bounds`` are the cut points [0 = b_0 <= b_1 <= ... <= b_R = N]; part r
    holds keys [b_r, b_{r+1}).  Returns ``[(O_r, L_r)]``; an empty part gives
    ``O_r = 0`` and ``L_r = -inf`` (App. A.3).
    """
    parts = []
    for a, b in zip(bounds[:-1], bounds[1:]):
        parts.append(sdpa(Qr, K[..., a:b, :], V[..., a:b, :]))
    return parts


def split_merge(parts: Sequence[Tuple[np.ndarray, np.ndarray]]) -> Tuple[np.ndarray, np.ndarray]:
    """Exact merge of per-part SDPA results (App. A.3, Eqs. (24)-(28)).

    ``parts`` is a sequence of ``(O_r [..., M, D], L_r [..., M])``.  Uses the
    stable form: L_max = max_r L_r; a_r = exp(L_r - L_max); a = sum_r a_r;
    U = sum_r a_r O_r; L = L_max + log a; Z = U / a.  Parts with L_r = -inf
    contribute nothing; at least one part must be non-empty for every row.
    """
    Ls = np.stack([_f64(L) for _, L in parts])  # [R, ..., M]
    Os = np.stack([_f64(O) for O, _ in parts])  # [R, ..., M, D]
    Lmax = Ls.max(axis=0)
    if not np.all(np.isfinite(Lmax)):
        raise ValueError("every row needs at least one non-empty part")
    a_r = np.exp(Ls - Lmax[None])
    a = a_r.sum(axis=0)
    U = (a_r[..., None] * Os).sum(axis=0)
    return U / a[..., None], Lmax + np.log(a)


def materialised_operator(X, Wk, Wv, Wkt, Wvt, seeds, H: int) -> Dict[str, np.ndarray]:
    """Materialise the per-head rank-<=M token operator for small N.

    W_enc = softmax over N of S = s Q K^T (rows are routes), W_dec = softmax
    over M of S^T (rows are tokens), W_eff = W_dec W_enc in R^{N x N}
    (Sec. 3.1, Eq. (6); Sec. 3.2, Eq. (12)).  Q is the synthesised query set
    Q(X) (Eq. (8)).  Returns ``W_enc [B,H,M,N]``, ``W_dec [B,H,N,M]``,
    ``W_eff [B,H,N,N]`` and ``V [B,H,N,D]``; the mixer's per-head output
    before merging is ``W_eff @ V``.
    """
    X = _f64(X)
    K = project(X, Wk, H)
    V = project(X, Wv, H)
    Kt = project(X, Wkt, H)
    Vt = project(X, Wvt, H)
    D = K.shape[-1]
    s = 1.0 / math.sqrt(D)

    def softmax_last(S):
        E = np.exp(S - S.max(axis=-1, keepdims=True))
        return E / E.sum(axis=-1, keepdims=True)

    Wq = softmax_last(s * (_f64(seeds)[None] @ np.swapaxes(Kt, -1, -2)))  # [B,H,M,N]
    Q = Wq @ Vt
    S = s * (Q @ np.swapaxes(K, -1, -2))  # [B,H,M,N]
    W_enc = softmax_last(S)
    W_dec = softmax_last(np.swapaxes(S, -1, -2))  # [B,H,N,M]
    return {"W_enc": W_enc, "W_dec": W_dec, "W_eff": W_dec @ W_enc, "V": V, "Q": Q}


def sdpa_backward(Q, K, V, O, L, dO, scale: float | None = None) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Gradient of ``O = SDPA(Q, K, V)`` (softmax over the keys) from the
    global output O and log-normaliser L of the forward (App. A.5).

    Q: [..., Nq, D]; K: [..., Nk, D]; V: [..., Nk, Dv]; O, dO: [..., Nq, Dv];
    L: [..., Nq].  Leading dimensions broadcast; every gradient comes back
    with the broadcast leading shape (a caller whose operand was shared over
    a dimension sums over it).  With P = exp(s Q K^T - L) and c = <dO, O>
    over the value dimension:

        dV = P^T dO,   dS = P * (dO V^T - c),   dK = s dS^T Q,   dQ = s dS K.

    The key axis is walked in chunks; every chunk reads the global L and c,
    so a chunk's dK, dV are final and its dQ share is a plain sum.
    Returns ``(dQ, dK, dV)``.
    """
    Q, K, V, O, L, dO = (_f64(a) for a in (Q, K, V, O, L, dO))
    D = Q.shape[-1]
    s = 1.0 / math.sqrt(D) if scale is None else float(scale)
    lead = np.broadcast_shapes(Q.shape[:-2], K.shape[:-2], V.shape[:-2], O.shape[:-2], dO.shape[:-2])
    Nq, Nk = Q.shape[-2], K.shape[-2]
    Q = np.broadcast_to(Q, lead + Q.shape[-2:])
    K = np.broadcast_to(K, lead + K.shape[-2:])
    V = np.broadcast_to(V, lead + V.shape[-2:])
    c = (dO * O).sum(axis=-1)  # [..., Nq]
    dQ = np.zeros(lead + (Nq, D))
    dK = np.zeros(lead + (Nk, D))
    dV = np.zeros(lead + (Nk, V.shape[-1]))
    for k0 in range(0, Nk, _KEY_CHUNK):
        k1 = min(Nk, k0 + _KEY_CHUNK)
        Kc, Vc = K[..., k0:k1, :], V[..., k0:k1, :]
        P = np.exp(s * (Q @ np.swapaxes(Kc, -1, -2)) - L[..., None])  # [..., Nq, nk]
        dV[..., k0:k1, :] = np.swapaxes(P, -1, -2) @ dO
        dS = P * (dO @ np.swapaxes(Vc, -1, -2) - c[..., None])
        dK[..., k0:k1, :] = s * (np.swapaxes(dS, -1, -2) @ Q)
        dQ += s * (dS @ Kc)
    return dQ, dK, dV


def mixer_backward(X, Wk, Wv, Wkt, Wvt, Wo, seeds, H: int, dO) -> Dict[str, np.ndarray]:
    """Reverse pass of the FLARE++ mixer (App. A.5) for the output gradient
    dO [B, N, C].

    Runs the forward (``mixer_forward``) for the operands and the global
    log-normalisers, then, in reverse order of the forward:

    * merge: dW_O = Y^T dO (summed over batch and tokens), dY = dO W_O^T;
    * call 3 (decode; queries K, keys Q, values Z): ``sdpa_backward`` gives
      the token-key gradient and the decoder's share of dQ and dZ;
    * call 2 (encode; queries Q, keys K, values V) with the summed dZ gives
      the encoder's share of dQ and the local dK, dV;
    * call 1 (query synthesis; seeds shared over the batch, keys K~, values
      V~) with dQ = decoder share + encoder share gives d(seeds), summed over
      the batch, and the local dK~, dV~;
    * the projections: dX = sum_j dG_j W_j^T, dW_j = X^T dG_j over the four
      projected tensors (heads merged back to channels).

    Returns the parameter and input gradients ``dX, dWk, dWv, dWkt, dWvt,
    dWo, dseeds`` and the intermediates ``dY, dZ, dQ, dQ3, dK, dV, dKt, dVt``
    ([B, H, *, D] for the per-head ones; dY is [B, N, C]).
    """
    X = _f64(X)
    dO = _f64(dO)
    f = mixer_forward(X, Wk, Wv, Wkt, Wvt, Wo, seeds, H)
    Q, Z, K, V, Kt, Vt = f["Q"], f["Z"], f["K"], f["V"], f["Kt"], f["Vt"]
    B, N, C = X.shape
    # merge
    dWo = np.einsum("bni,bno->io", f["Y"], dO)
    dYh = split_heads(dO @ _f64(Wo).T, H)
    # call 3: the decode's own log-normaliser (per token)
    Yh, L3 = sdpa(K, Q, Z)
    dK3, dQ3, dZ = sdpa_backward(K, Q, Z, Yh, L3, dYh)
    # call 2
    dQ2, dK2, dV = sdpa_backward(Q, K, V, Z, f["L2"], dZ)
    dQ = dQ3 + dQ2
    dK = dK3 + dK2
    # call 1: the seeds are shared over the batch
    dS1, dKt, dVt = sdpa_backward(_f64(seeds)[None], Kt, Vt, Q, f["L1"], dQ)
    dseeds = dS1.sum(axis=0)
    # projections
    grads = {}
    dX = np.zeros_like(X)
    for name, W, G in (("dWk", Wk, dK), ("dWv", Wv, dV), ("dWkt", Wkt, dKt), ("dWvt", Wvt, dVt)):
        Gm = merge_heads(G)  # [B, N, C]
        dX += Gm @ _f64(W).T
        grads[name] = np.einsum("bni,bno->io", X, Gm)
    out = {"dX": dX, "dWo": dWo, "dseeds": dseeds, "dY": merge_heads(dYh), "dZ": dZ, "dQ": dQ,
           "dQ3": dQ3, "dK": dK, "dV": dV, "dKt": dKt, "dVt": dVt}
    out.update(grads)
    return out


def layer_norm(X, gamma, beta, eps: float) -> np.ndarray:
    """Normalise every token over its channels: (x - mean) / sqrt(var + eps)
    * gamma + beta, var the biased variance (mean of squared deviations)."""
    X = _f64(X)
    mean = X.mean(axis=-1, keepdims=True)
    var = ((X - mean) ** 2).mean(axis=-1, keepdims=True)
    return (X - mean) / np.sqrt(var + eps) * _f64(gamma) + _f64(beta)


def block_forward(X, gamma, beta, eps: float, Wk, Wv, Wkt, Wvt, Wo, seeds, H: int) -> np.ndarray:
    """The pre-norm residual block around the mixer: X + mixer(LN(X))."""
    return _f64(X) + mixer_forward(layer_norm(X, gamma, beta, eps), Wk, Wv, Wkt, Wvt, Wo, seeds, H)["O"]


def mixer_backward_shared(X, Wk, Wv, Wo, seeds, H: int, dO) -> dict:
    """Backward of the shared-projection mixer (K~ = K, V~ = V): the mixer's
    backward with W~_K = W_K and W~_V = W_V, a tied weight's gradient being
    the sum of the gradients of its two uses."""
    g = mixer_backward(X, Wk, Wv, Wk, Wv, Wo, seeds, H, dO)
    return {"dX": g["dX"], "dWk": g["dWk"] + g["dWkt"], "dWv": g["dWv"] + g["dWvt"], "dWo": g["dWo"],
            "dseeds": g["dseeds"]}


def block_backward(X, gamma, beta, eps: float, Wk, Wv, Wkt, Wvt, Wo, seeds, H: int, dO) -> dict:
    """Gradients of <O, dO> for O = X + mixer(LN(X)).  With xhat the
    normalised token, r = 1 / sqrt(var + eps) and g = dXn * gamma (dXn the
    mixer's input gradient): dX = dO + r (g - mean_c g - xhat mean_c(g xhat)),
    dgamma = sum_tokens dXn xhat, dbeta = sum_tokens dXn."""
    X = _f64(X)
    mean = X.mean(axis=-1, keepdims=True)
    var = ((X - mean) ** 2).mean(axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(var + eps)
    xhat = (X - mean) * r
    Xn = xhat * _f64(gamma) + _f64(beta)
    g = mixer_backward(Xn, Wk, Wv, Wkt, Wvt, Wo, seeds, H, dO)
    dXn = g["dX"]
    gg = dXn * _f64(gamma)
    dX = _f64(dO) + r * (gg - gg.mean(axis=-1, keepdims=True) - xhat * (gg * xhat).mean(axis=-1, keepdims=True))
    out = {k: g[k] for k in ("dWk", "dWv", "dWkt", "dWvt", "dWo", "dseeds")}
    out.update(dX=dX, dgamma=(dXn * xhat).reshape(-1, X.shape[-1]).sum(axis=0),
               dbeta=dXn.reshape(-1, X.shape[-1]).sum(axis=0))
    return out

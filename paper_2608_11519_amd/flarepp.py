"""Thin ctypes binding over libflarepp.so (the C ABI in include/flarepp.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of the library.  PyTorch provides device memory and the current
stream.  If the library is missing this module raises; there is no fallback.
"""

from __future__ import annotations

import ctypes
import operator
import os
from typing import Optional, Tuple

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflarepp.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_HIP = -4
F32 = 0
BF16 = 1
ENCODE = 0
DECODE = 1

EXPORTS = (
    "flarepp_last_error", "flarepp_version",
    "flarepp_project_workspace_bytes", "flarepp_project",
    "flarepp_route_workspace_bytes", "flarepp_route",
    "flarepp_mixer_workspace_bytes", "flarepp_mixer_forward", "flarepp_mixer_forward_debug",
    "flarepp_mixer_forward_profiled", "flarepp_mixer_path", "flarepp_mixer_stage",
    "flarepp_flare_workspace_bytes", "flarepp_flare_forward", "flarepp_flare_forward_debug",
    "flarepp_mixer_backward_workspace_bytes", "flarepp_mixer_backward", "flarepp_mixer_backward_debug",
    "flarepp_mixer_forward_shared", "flarepp_block_workspace_bytes", "flarepp_block_forward",
    "flarepp_mixer_backward_shared", "flarepp_mixer_forward_train", "flarepp_mixer_backward_from_saved",
    "flarepp_block_backward_workspace_bytes", "flarepp_block_backward",
    "flarepp_mixer_noalloc_max_bytes", "flarepp_mixer_forward_noalloc",
)
PATH_UNFUSED = 0
PATH_FUSED = 1
PROFILE_EVENTS = 9
PROFILE_STAGES = ("prep", "project", "call1_encode", "call1_combine", "call2_encode",
                  "call2_combine", "call3_decode", "merge")

_lib = None


class FlareppError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"flarepp error {code}: {msg}")
        self.code = code


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libflarepp.so once and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_11519_amd.build`")
    lib = ctypes.CDLL(path)
    i64, vp, sz, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    fp = ctypes.c_void_p
    lib.flarepp_last_error.restype = ctypes.c_char_p
    lib.flarepp_last_error.argtypes = []
    lib.flarepp_version.restype = ctypes.c_char_p
    lib.flarepp_version.argtypes = []
    lib.flarepp_project_workspace_bytes.restype = sz
    lib.flarepp_project_workspace_bytes.argtypes = [i32, i64]
    lib.flarepp_project.restype = i32
    lib.flarepp_project.argtypes = [i32, i64, i64, i64, i64] + [vp] * 9 + [vp, sz, vp]
    lib.flarepp_route_workspace_bytes.restype = sz
    lib.flarepp_route_workspace_bytes.argtypes = [i32, i32, i64, i64, i64, i64, i64]
    lib.flarepp_route.restype = i32
    lib.flarepp_route.argtypes = [i32, i32, i64, i64, i64, i64, i64, vp, i64, vp, vp, vp, fp,
                                  vp, sz, vp]
    lib.flarepp_mixer_workspace_bytes.restype = sz
    lib.flarepp_mixer_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64]
    lib.flarepp_mixer_forward.restype = i32
    lib.flarepp_mixer_forward.argtypes = [i32, i64, i64, i64, i64, i64] + [vp] * 8 + [vp, sz, vp]
    lib.flarepp_mixer_forward_debug.restype = i32
    lib.flarepp_mixer_forward_debug.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 8
                                                + [fp, fp, vp] + [vp, sz, vp])
    lib.flarepp_mixer_path.restype = i32
    lib.flarepp_mixer_path.argtypes = [i32, i64, i64, i64, i64, i64]
    lib.flarepp_mixer_forward_profiled.restype = i32
    lib.flarepp_mixer_forward_profiled.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 8
                                                   + [vp, sz, vp, ctypes.POINTER(vp), i32])
    lib.flarepp_mixer_stage.restype = i32
    lib.flarepp_mixer_stage.argtypes = [i32, i32, i64, i64, i64, i64, i64] + [vp] * 8 + [vp, sz, vp]
    lib.flarepp_flare_workspace_bytes.restype = sz
    lib.flarepp_flare_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64]
    lib.flarepp_flare_forward.restype = i32
    lib.flarepp_flare_forward.argtypes = [i32, i64, i64, i64, i64, i64] + [vp] * 6 + [vp, sz, vp]
    lib.flarepp_flare_forward_debug.restype = i32
    lib.flarepp_flare_forward_debug.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 6
                                                + [fp, vp] + [vp, sz, vp])
    lib.flarepp_mixer_forward_shared.restype = i32
    lib.flarepp_mixer_forward_shared.argtypes = [i32, i64, i64, i64, i64, i64] + [vp] * 6 + [vp, sz, vp]
    lib.flarepp_mixer_backward_workspace_bytes.restype = sz
    lib.flarepp_mixer_backward_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64]
    lib.flarepp_mixer_backward.restype = i32
    lib.flarepp_mixer_backward.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 8 + [fp] * 7
                                           + [vp, sz, vp])
    lib.flarepp_mixer_backward_debug.restype = i32
    lib.flarepp_mixer_backward_debug.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 8 + [fp] * 9
                                                 + [vp, sz, vp])
    lib.flarepp_mixer_forward_train.restype = i32
    lib.flarepp_mixer_forward_train.argtypes = [i32, i64, i64, i64, i64, i64] + [vp] * 8 + [vp, sz, vp]
    lib.flarepp_mixer_backward_from_saved.restype = i32
    lib.flarepp_mixer_backward_from_saved.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 8 + [fp] * 7
                                                      + [vp, sz, vp])
    lib.flarepp_mixer_backward_shared.restype = i32
    lib.flarepp_mixer_backward_shared.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 6 + [fp] * 5
                                                  + [vp, sz, vp])
    lib.flarepp_block_backward_workspace_bytes.restype = sz
    lib.flarepp_block_backward_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64]
    lib.flarepp_block_backward.restype = i32
    lib.flarepp_block_backward.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 3 + [ctypes.c_float]
                                           + [vp] * 7 + [fp] * 9 + [vp, sz, vp])
    lib.flarepp_block_workspace_bytes.restype = sz
    lib.flarepp_block_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64]
    lib.flarepp_block_forward.restype = i32
    lib.flarepp_block_forward.argtypes = ([i32, i64, i64, i64, i64, i64] + [vp] * 3 + [ctypes.c_float]
                                          + [vp] * 7 + [vp, sz, vp])
    lib.flarepp_mixer_noalloc_max_bytes.restype = sz
    lib.flarepp_mixer_noalloc_max_bytes.argtypes = []
    lib.flarepp_mixer_forward_noalloc.restype = i32
    lib.flarepp_mixer_forward_noalloc.argtypes = [i32, i64, i64, i64, i64, i64] + [vp] * 8 + [vp]
    _lib = lib
    return lib


def last_error() -> str:
    return load().flarepp_last_error().decode()


def version() -> str:
    return load().flarepp_version().decode()


def _check(rc: int) -> None:
    if rc != OK:
        raise FlareppError(rc, last_error())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _same(t: torch.Tensor, name: str, shape, dtype: torch.dtype, device: torch.device) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device} (the device of X)")


def _validate(X: torch.Tensor, H: int, *, mats=(), routes=None, tokens=(), vecs=(), ws=None,
              f32_tokens=(), f32_mats=(), f32_routes=()):
    """Check every tensor argument of a mixer-level entry point against X
    before anything reaches the library (whose kernels trust the sizes they
    are given): X is [B, N, C] in float32 or bfloat16; every other tensor is
    on X's device, in X's dtype unless it is one of the float32 outputs, with
    the shape its role implies: C x C weights, [H, M, C/H] seeds or queries,
    [B, N, C] token tensors (outputs, output gradients), [C] vectors; the
    workspace is uint8.  Raises TypeError or ValueError; returns
    (B, N, C, M, D)."""
    if not isinstance(X, torch.Tensor):
        raise TypeError(f"X must be a torch.Tensor, got {type(X).__name__}")
    _dtype_code(X)
    if X.dim() != 3:
        raise ValueError(f"X must be [B, N, C], got shape {tuple(X.shape)}")
    B, N, C = X.shape
    try:
        H = operator.index(H)
    except TypeError:
        raise TypeError(f"H must be an integer, got {type(H).__name__}") from None
    if isinstance(H, bool) or H < 1 or C % H:
        raise ValueError(f"H={H!r} must be a positive integer dividing C={C}")
    D = C // H
    dev, dt = X.device, X.dtype
    M = None
    if routes is not None:
        name, t = routes
        if not isinstance(t, torch.Tensor) or t.dim() != 3:
            raise ValueError(f"{name} must be a [H, M, D] tensor")
        M = t.shape[1]
        _same(t, name, (H, M, D), dt, dev)
    for name, t in mats:
        _same(t, name, (C, C), dt, dev)
    for name, t in tokens:
        if t is not None:
            _same(t, name, (B, N, C), dt, dev)
    for name, t in vecs:
        _same(t, name, (C,), dt, dev)
    for name, t in f32_tokens:
        _same(t, name, (B, N, C), torch.float32, dev)
    for name, t in f32_mats:
        _same(t, name, (C, C), torch.float32, dev)
    for name, t in f32_routes:
        _same(t, name, (H, M, D), torch.float32, dev)
    if ws is not None:
        if not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8:
            raise TypeError("ws must be a uint8 torch.Tensor")
        if ws.device != dev:
            raise ValueError(f"ws is on {ws.device}, expected {dev} (the device of X)")
    return B, N, C, M, D


def _stream(device: torch.device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(nbytes: int, device, ws: Optional[torch.Tensor]) -> torch.Tensor:
    if ws is not None and ws.numel() * ws.element_size() >= nbytes:
        return ws
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# workspace sizes
# ---------------------------------------------------------------------------

def flarepp_project_workspace_bytes(dtype: int, C: int) -> int:
    return int(load().flarepp_project_workspace_bytes(dtype, C))


def flarepp_route_workspace_bytes(kind: int, dtype: int, B: int, H: int, N: int, M: int, D: int) -> int:
    return int(load().flarepp_route_workspace_bytes(kind, dtype, B, H, N, M, D))


def flarepp_mixer_workspace_bytes(dtype: int, B: int, N: int, C: int, H: int, M: int) -> int:
    return int(load().flarepp_mixer_workspace_bytes(dtype, B, N, C, H, M))


def flarepp_mixer_path(dtype: int, B: int, N: int, C: int, H: int, M: int) -> int:
    """PATH_FUSED or PATH_UNFUSED (the kernel sequence the mixer runs)."""
    rc = int(load().flarepp_mixer_path(dtype, B, N, C, H, M))
    _check(rc if rc < 0 else OK)
    return rc


# ---------------------------------------------------------------------------
# entry points on torch tensors
# ---------------------------------------------------------------------------

def flarepp_project(X: torch.Tensor, Wk=None, Wv=None, Wkt=None, Wvt=None, *, H: int,
                    ws: Optional[torch.Tensor] = None) -> Tuple[Optional[torch.Tensor], ...]:
    """K, V, K~, V~ = X W (heads split, [B, H, N, D]) for each weight given."""
    lib = load()
    B, N, C, _, D = _validate(X, H, mats=[(n, W) for n, W in (("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt))
                                          if W is not None], ws=ws)
    dt = _dtype_code(X)
    outs = [None if W is None else torch.empty((B, H, N, D), dtype=X.dtype, device=X.device)
            for W in (Wk, Wv, Wkt, Wvt)]
    w = _workspace(flarepp_project_workspace_bytes(dt, C), X.device, ws)
    rc = lib.flarepp_project(dt, B, N, C, H, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt), _ptr(Wvt),
                             *[_ptr(o) for o in outs], _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return tuple(outs)


def flarepp_route(kind: int, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, *,
                  shared_routes: bool = False, want_lse: bool = False,
                  ws: Optional[torch.Tensor] = None):
    """One routing SDPA call.

    ENCODE: q float32 [B|1, H, M, D] routes; k, v [B, H, N, D] tokens ->
    (out float32 [B, H, M, D], lse [B, H, M] or None).
    DECODE: q [B, H, N, D] tokens; k, v float32 [B|1, H, M, D] routes ->
    out [B, N, H*D] in the tokens' dtype.
    """
    lib = load()
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not isinstance(t, torch.Tensor) or t.dim() != 4:
            raise ValueError(f"{name} must be a 4-D tensor")
    tok, rt = (k, q) if kind == ENCODE else (q, k)
    B, H, N, D = tok.shape
    M = rt.shape[2]
    if kind == ENCODE:
        _same(v, "v", tok.shape, tok.dtype, tok.device)
        _same(q, "q", ((1 if shared_routes else B), H, M, D), torch.float32, tok.device)
    elif kind == DECODE:
        _same(k, "k", ((1 if shared_routes else B), H, M, D), torch.float32, tok.device)
        _same(v, "v", k.shape, torch.float32, tok.device)
    else:
        raise ValueError(f"kind={kind!r} is neither ENCODE nor DECODE")
    if ws is not None and (ws.dtype != torch.uint8 or ws.device != tok.device):
        raise TypeError("ws must be a uint8 tensor on the tokens' device")
    if kind == ENCODE:
        dt = _dtype_code(k)
        out = torch.empty((B, H, M, D), dtype=torch.float32, device=k.device)
        lse = torch.empty((B, H, M), dtype=torch.float32, device=k.device) if want_lse else None
    else:
        dt = _dtype_code(q)
        out = torch.empty((B, N, H * D), dtype=q.dtype, device=q.device)
        lse = None
    stride = 0 if shared_routes else H * M * D
    dev = out.device
    w = _workspace(flarepp_route_workspace_bytes(kind, dt, B, H, N, M, D), dev, ws)
    rc = lib.flarepp_route(kind, dt, B, H, N, M, D, _ptr(q), stride, _ptr(k), _ptr(v), _ptr(out),
                           _ptr(lse), _ptr(w), w.numel(), _stream(dev))
    _check(rc)
    return (out, lse) if kind == ENCODE else out


def flarepp_mixer_forward(X, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int,
                          out: Optional[torch.Tensor] = None,
                          ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The FLARE++ mixer forward: O [B, N, C] in X's dtype."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("out", out)], ws=ws)
    dt = _dtype_code(X)
    O = out if out is not None else torch.empty_like(X)
    w = _workspace(flarepp_mixer_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_mixer_forward(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt),
                                   _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(O), _ptr(w), w.numel(),
                                   _stream(X.device))
    _check(rc)
    return O


def flarepp_mixer_noalloc_max_bytes() -> int:
    return int(load().flarepp_mixer_noalloc_max_bytes())


def flarepp_mixer_forward_noalloc(X, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int,
                                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The FLARE++ mixer forward on the library's own scratch array (no
    workspace argument, nothing allocated by the library): O [B, N, C] in
    X's dtype, bitwise equal to flarepp_mixer_forward.  Calls on one device
    share the array and must not overlap."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)],
                              routes=("seeds", seeds), tokens=[("out", out)])
    dt = _dtype_code(X)
    O = out if out is not None else torch.empty_like(X)
    rc = lib.flarepp_mixer_forward_noalloc(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt), _ptr(Wvt),
                                           _ptr(Wo), _ptr(seeds), _ptr(O), _stream(X.device))
    _check(rc)
    return O


def flarepp_mixer_forward_debug(X, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int,
                                ws: Optional[torch.Tensor] = None):
    """Mixer forward that also returns the stage results: (O, Q, Z, Y)."""
    lib = load()
    B, N, C, M, D = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds), ws=ws)
    dt = _dtype_code(X)
    O = torch.empty_like(X)
    Q = torch.empty((B, H, M, D), dtype=torch.float32, device=X.device)
    Z = torch.empty_like(Q)
    Y = torch.empty_like(X)
    w = _workspace(flarepp_mixer_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_mixer_forward_debug(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt),
                                         _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(O), _ptr(Q), _ptr(Z),
                                         _ptr(Y), _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return O, Q, Z, Y


def flarepp_mixer_forward_profiled(X, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int, events,
                                   out: Optional[torch.Tensor] = None,
                                   ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Mixer forward that records ``events`` (PROFILE_EVENTS torch.cuda.Event
    objects with timing enabled) around its stages on the current stream."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("out", out)], ws=ws)
    dt = _dtype_code(X)
    if len(events) != PROFILE_EVENTS:
        raise ValueError(f"need {PROFILE_EVENTS} events")
    stream = torch.cuda.current_stream(X.device)
    for e in events:  # torch creates the underlying hipEvent_t on first record
        if e.cuda_event == 0:
            e.record(stream)
    handles = (ctypes.c_void_p * PROFILE_EVENTS)(*[e.cuda_event for e in events])
    O = out if out is not None else torch.empty_like(X)
    w = _workspace(flarepp_mixer_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_mixer_forward_profiled(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv),
                                            _ptr(Wkt), _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(O),
                                            _ptr(w), w.numel(), ctypes.c_void_p(stream.cuda_stream),
                                            handles, PROFILE_EVENTS)
    _check(rc)
    return O


def flarepp_mixer_stage(stage: int, X, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int, out: torch.Tensor,
                        ws: torch.Tensor) -> None:
    """Run stage ``stage`` (1-based, as PROFILE_STAGES) of the mixer alone.
    ``ws`` and ``out`` must be those of a complete mixer forward with the same
    arguments."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("out", out)], ws=ws)
    dt = _dtype_code(X)
    rc = lib.flarepp_mixer_stage(stage, dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt),
                                 _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(out), _ptr(ws), ws.numel(),
                                 _stream(X.device))
    _check(rc)


def flarepp_flare_workspace_bytes(dtype: int, B: int, N: int, C: int, H: int, M: int) -> int:
    return int(load().flarepp_flare_workspace_bytes(dtype, B, N, C, H, M))


def flarepp_flare_forward(X, Wk, Wv, Wo, queries, *, H: int,
                          out: Optional[torch.Tensor] = None,
                          ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The fixed-query FLARE mixer forward: O [B, N, C] in X's dtype;
    ``queries`` [H, M, D] are the learned routing queries."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wo", Wo)], routes=("queries", queries),
                              tokens=[("out", out)], ws=ws)
    dt = _dtype_code(X)
    O = out if out is not None else torch.empty_like(X)
    w = _workspace(flarepp_flare_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_flare_forward(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wo),
                                   _ptr(queries), _ptr(O), _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return O


def flarepp_flare_forward_debug(X, Wk, Wv, Wo, queries, *, H: int,
                                ws: Optional[torch.Tensor] = None):
    """Fixed-query FLARE forward that also returns the stage results: (O, Z, Y)."""
    lib = load()
    B, N, C, M, D = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wo", Wo)], routes=("queries", queries), ws=ws)
    dt = _dtype_code(X)
    O = torch.empty_like(X)
    Z = torch.empty((B, H, M, D), dtype=torch.float32, device=X.device)
    Y = torch.empty_like(X)
    w = _workspace(flarepp_flare_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_flare_forward_debug(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wo),
                                         _ptr(queries), _ptr(O), _ptr(Z), _ptr(Y), _ptr(w), w.numel(),
                                         _stream(X.device))
    _check(rc)
    return O, Z, Y


def flarepp_mixer_forward_shared(X, Wk, Wv, Wo, seeds, *, H: int,
                                 out: Optional[torch.Tensor] = None,
                                 ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """FLARE++ with the query-synthesis keys and values tied to K and V
    (K~ = K, V~ = V): O [B, N, C] in X's dtype."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("out", out)], ws=ws)
    dt = _dtype_code(X)
    O = out if out is not None else torch.empty_like(X)
    w = _workspace(flarepp_mixer_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_mixer_forward_shared(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wo), _ptr(seeds),
                                          _ptr(O), _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return O


def flarepp_mixer_backward_workspace_bytes(dtype: int, B: int, N: int, C: int, H: int, M: int) -> int:
    return int(load().flarepp_mixer_backward_workspace_bytes(dtype, B, N, C, H, M))


def _backward(debug, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, H, ws, out=None, saved=False):
    lib = load()
    B, N, C, M, D = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("dO", dO)], ws=ws,
                              f32_tokens=[("out['dX']", out["dX"])] if out else (),
                              f32_mats=[(f"out[{k!r}]", out[k]) for k in ("dWk", "dWv", "dWkt", "dWvt", "dWo")]
                              if out else (),
                              f32_routes=[("out['dseeds']", out["dseeds"])] if out else ())
    dt = _dtype_code(X)
    f32 = dict(dtype=torch.float32, device=X.device)
    if out is not None:
        g = dict(out)
    else:
        g = {"dX": torch.empty((B, N, C), **f32)}
        for k in ("dWk", "dWv", "dWkt", "dWvt", "dWo"):
            g[k] = torch.empty((C, C), **f32)
        g["dseeds"] = torch.empty((H, M, D), **f32)
    outs = [g[k] for k in ("dX", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dseeds")]
    if debug:
        g["dZ"] = torch.empty((B, H, M, D), **f32)
        g["dQ"] = torch.empty((B, H, M, D), **f32)
        outs += [g["dZ"], g["dQ"]]
    need = flarepp_mixer_backward_workspace_bytes(dt, B, N, C, H, M)
    if saved and (ws is None or ws.numel() * ws.element_size() < need):
        raise ValueError("backward_from_saved needs the workspace its training forward filled")
    w = _workspace(need, X.device, ws)
    if saved:
        rc = lib.flarepp_mixer_backward_from_saved(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt),
                                                   _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(dO),
                                                   *[_ptr(t) for t in outs], _ptr(w), w.numel(), _stream(X.device))
        _check(rc)
        return g
    fn = lib.flarepp_mixer_backward_debug if debug else lib.flarepp_mixer_backward
    rc = fn(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt), _ptr(Wvt), _ptr(Wo), _ptr(seeds),
            _ptr(dO), *[_ptr(t) for t in outs], _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return g


def flarepp_mixer_backward(X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, *, H: int,
                           ws: Optional[torch.Tensor] = None, out: Optional[dict] = None):
    """Gradients of <O, dO> for the FLARE++ mixer: a dict of fp32 tensors
    dX [B, N, C], dWk, dWv, dWkt, dWvt, dWo [C, C] and dseeds [H, M, D]
    (written into ``out``'s tensors when given)."""
    return _backward(False, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, H, ws, out)


def flarepp_mixer_forward_train(X, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int, ws: torch.Tensor,
                                out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Mixer forward that keeps in ``ws`` (at least
    flarepp_mixer_backward_workspace_bytes bytes) what
    flarepp_mixer_backward_from_saved reads: O [B, N, C] in X's dtype."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("out", out)], ws=ws)
    dt = _dtype_code(X)
    need = flarepp_mixer_backward_workspace_bytes(dt, B, N, C, H, M)
    if ws.numel() * ws.element_size() < need:
        raise ValueError(f"ws holds {ws.numel() * ws.element_size()} bytes, {need} needed")
    O = out if out is not None else torch.empty_like(X)
    rc = lib.flarepp_mixer_forward_train(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wkt), _ptr(Wvt),
                                         _ptr(Wo), _ptr(seeds), _ptr(O), _ptr(ws), ws.numel() * ws.element_size(),
                                         _stream(X.device))
    _check(rc)
    return O


def flarepp_mixer_backward_from_saved(X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, *, H: int, ws: torch.Tensor,
                                      out: Optional[dict] = None):
    """``flarepp_mixer_backward`` on the state a flarepp_mixer_forward_train
    with the same inputs left in ``ws`` (no forward is run again)."""
    return _backward(False, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, H, ws, out, saved=True)


def flarepp_mixer_backward_debug(X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, *, H: int,
                                 ws: Optional[torch.Tensor] = None):
    """``flarepp_mixer_backward`` plus the summed latent and query gradients
    dZ, dQ [B, H, M, D]."""
    return _backward(True, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, H, ws)


def flarepp_mixer_backward_shared(X, Wk, Wv, Wo, seeds, dO, *, H: int,
                                  ws: Optional[torch.Tensor] = None, out: Optional[dict] = None):
    """Gradients of <O, dO> for the shared-projection mixer (K~ = K, V~ = V):
    a dict of fp32 tensors dX [B, N, C], dWk, dWv, dWo [C, C] (the tied
    weights' gradients summed over both uses) and dseeds [H, M, D]."""
    lib = load()
    B, N, C, M, D = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("dO", dO)], ws=ws,
                              f32_tokens=[("out['dX']", out["dX"])] if out else (),
                              f32_mats=[(f"out[{k!r}]", out[k]) for k in ("dWk", "dWv", "dWo")] if out else (),
                              f32_routes=[("out['dseeds']", out["dseeds"])] if out else ())
    dt = _dtype_code(X)
    f32 = dict(dtype=torch.float32, device=X.device)
    if out is not None:
        g = dict(out)
    else:
        g = {"dX": torch.empty((B, N, C), **f32), "dWk": torch.empty((C, C), **f32),
             "dWv": torch.empty((C, C), **f32), "dWo": torch.empty((C, C), **f32),
             "dseeds": torch.empty((H, M, D), **f32)}
    w = _workspace(flarepp_mixer_backward_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_mixer_backward_shared(dt, B, N, C, H, M, _ptr(X), _ptr(Wk), _ptr(Wv), _ptr(Wo), _ptr(seeds),
                                           _ptr(dO), *[_ptr(g[k]) for k in ("dX", "dWk", "dWv", "dWo", "dseeds")],
                                           _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return g


def flarepp_block_workspace_bytes(dtype: int, B: int, N: int, C: int, H: int, M: int) -> int:
    return int(load().flarepp_block_workspace_bytes(dtype, B, N, C, H, M))


def flarepp_block_forward(X, gamma, beta, Wk, Wv, Wkt, Wvt, Wo, seeds, *, H: int, eps: float = 1e-5,
                          out: Optional[torch.Tensor] = None,
                          ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The pre-norm residual block X + mixer(LayerNorm(X)): O [B, N, C] in
    X's dtype; gamma, beta [C] in X's dtype."""
    lib = load()
    B, N, C, M, _ = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("out", out)], vecs=[("gamma", gamma), ("beta", beta)], ws=ws)
    dt = _dtype_code(X)
    O = out if out is not None else torch.empty_like(X)
    w = _workspace(flarepp_block_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_block_forward(dt, B, N, C, H, M, _ptr(X), _ptr(gamma), _ptr(beta), float(eps), _ptr(Wk),
                                   _ptr(Wv), _ptr(Wkt), _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(O), _ptr(w),
                                   w.numel(), _stream(X.device))
    _check(rc)
    return O


def flarepp_block_backward_workspace_bytes(dtype: int, B: int, N: int, C: int, H: int, M: int) -> int:
    return int(load().flarepp_block_backward_workspace_bytes(dtype, B, N, C, H, M))


def flarepp_block_backward(X, gamma, beta, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, *, H: int, eps: float = 1e-5,
                           ws: Optional[torch.Tensor] = None):
    """Gradients of <O, dO> for the pre-norm residual block: a dict of fp32
    tensors dX [B, N, C], dgamma, dbeta [C], dWk, dWv, dWkt, dWvt, dWo [C, C]
    and dseeds [H, M, D]."""
    lib = load()
    B, N, C, M, D = _validate(X, H, mats=[("Wk", Wk), ("Wv", Wv), ("Wkt", Wkt), ("Wvt", Wvt), ("Wo", Wo)], routes=("seeds", seeds),
                              tokens=[("dO", dO)], vecs=[("gamma", gamma), ("beta", beta)], ws=ws)
    dt = _dtype_code(X)
    f32 = dict(dtype=torch.float32, device=X.device)
    g = {"dX": torch.empty((B, N, C), **f32), "dgamma": torch.empty(C, **f32), "dbeta": torch.empty(C, **f32)}
    for k in ("dWk", "dWv", "dWkt", "dWvt", "dWo"):
        g[k] = torch.empty((C, C), **f32)
    g["dseeds"] = torch.empty((H, M, D), **f32)
    w = _workspace(flarepp_block_backward_workspace_bytes(dt, B, N, C, H, M), X.device, ws)
    rc = lib.flarepp_block_backward(dt, B, N, C, H, M, _ptr(X), _ptr(gamma), _ptr(beta), float(eps), _ptr(Wk),
                                    _ptr(Wv), _ptr(Wkt), _ptr(Wvt), _ptr(Wo), _ptr(seeds), _ptr(dO),
                                    *[_ptr(g[k]) for k in ("dX", "dgamma", "dbeta", "dWk", "dWv", "dWkt", "dWvt",
                                                            "dWo", "dseeds")],
                                    _ptr(w), w.numel(), _stream(X.device))
    _check(rc)
    return g


# short aliases
project = flarepp_project
route = flarepp_route
mixer_forward = flarepp_mixer_forward
mixer_forward_noalloc = flarepp_mixer_forward_noalloc
mixer_forward_debug = flarepp_mixer_forward_debug
flare_forward = flarepp_flare_forward
flare_forward_debug = flarepp_flare_forward_debug
mixer_forward_shared = flarepp_mixer_forward_shared
mixer_backward = flarepp_mixer_backward
mixer_backward_debug = flarepp_mixer_backward_debug
block_forward = flarepp_block_forward
mixer_backward_shared = flarepp_mixer_backward_shared
mixer_forward_train = flarepp_mixer_forward_train
mixer_backward_from_saved = flarepp_mixer_backward_from_saved
block_backward = flarepp_block_backward

"""C-ABI checks that need no GPU: the library loads, exports every function
include/flarepp.h declares, sizes workspaces, and rejects invalid arguments
before enqueuing anything (these calls never reach a HIP call)."""

import ctypes
import os
import re

import pytest

from paper_2608_11519_amd import flarepp as fp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flarepp.h")


def _lib():
    if not os.path.exists(fp.LIB_PATH):
        pytest.fail("libflarepp.so is not built (run __graft_entry__.build())")
    return fp.load()


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"FLAREPP_API\s+[\w\s\*]*?\b(flarepp_\w+)\s*\(", txt)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("flarepp_project", "flarepp_route", "flarepp_mixer_forward"):
        assert n in names
    assert set(names) == set(fp.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = _lib()
    for n in _declared():
        assert hasattr(lib, n), n
    assert "gfx950" in fp.version()


def test_workspace_sizes(monkeypatch):
    for dt in (fp.F32, fp.BF16):
        bs = 4 if dt == fp.F32 else 2
        assert fp.flarepp_project_workspace_bytes(dt, 128) >= 4 * 128 * 128 * bs
        n = fp.flarepp_mixer_workspace_bytes(dt, 4, 16384, 128, 8, 128)
        assert n >= 5 * 128 * 128 * bs + 2 * 4 * 8 * 128 * 16 * bs  # weights, Q and Z operands
        monkeypatch.setenv("FLAREPP_UNFUSED", "1")
        nu = fp.flarepp_mixer_workspace_bytes(dt, 4, 16384, 128, 8, 128)
        monkeypatch.delenv("FLAREPP_UNFUSED")
        assert nu >= 5 * 4 * 16384 * 128 * bs  # K, K~, V, V~, Y
        if dt == fp.BF16:  # the fused path never materialises K, V, K~, V~ or Y
            assert n < nu - 4 * 4 * 16384 * 128 * bs
        assert fp.flarepp_route_workspace_bytes(fp.ENCODE, dt, 2, 8, 1000, 64, 16) > 0
        assert fp.flarepp_route_workspace_bytes(fp.DECODE, dt, 2, 8, 1000, 64, 16) > 0
    # invalid shapes size to zero
    assert fp.flarepp_mixer_workspace_bytes(fp.BF16, 1, 10, 100, 3, 4) == 0
    assert fp.flarepp_mixer_workspace_bytes(7, 1, 10, 64, 4, 4) == 0
    assert fp.flarepp_route_workspace_bytes(5, fp.BF16, 1, 1, 10, 4, 16) == 0


@pytest.mark.parametrize("name", ["tiny", "grid2d", "mesh", "lra", "mesh3d"])
def test_workloads_take_the_fused_path(name):
    from paper_2608_11519_amd import inputs as inp
    w = inp.workload(name)
    dt = fp.F32 if w.dtype == "f32" else fp.BF16
    assert fp.flarepp_mixer_path(dt, w.B, w.N, w.C, w.H, w.M) == fp.PATH_FUSED


def test_unfused_path_for_other_widths(monkeypatch):
    assert fp.flarepp_mixer_path(fp.BF16, 1, 100, 32, 2, 16) == fp.PATH_UNFUSED   # C = 32
    assert fp.flarepp_mixer_path(fp.BF16, 1, 100, 512, 8, 16) == fp.PATH_UNFUSED  # C = 512
    assert fp.flarepp_mixer_path(fp.F32, 1, 100, 128, 2, 16) == fp.PATH_UNFUSED   # fp32, D = 64
    monkeypatch.setenv("FLAREPP_UNFUSED", "1")
    assert fp.flarepp_mixer_path(fp.BF16, 4, 16384, 128, 8, 128) == fp.PATH_UNFUSED
    with pytest.raises(fp.FlareppError):
        fp.flarepp_mixer_path(fp.BF16, 1, 100, 100, 3, 16)


def test_forced_chunk_count_changes_encode_workspace(monkeypatch):
    base = fp.flarepp_route_workspace_bytes(fp.ENCODE, fp.BF16, 1, 1, 4096, 64, 16)
    monkeypatch.setenv("FLAREPP_FORCE_CHUNKS", "200")
    forced = fp.flarepp_route_workspace_bytes(fp.ENCODE, fp.BF16, 1, 1, 4096, 64, 16)
    assert forced > base


_P = ctypes.c_void_p(4096)  # aligned, never dereferenced: validation fails first


def _mixer(dtype=fp.BF16, B=1, N=64, C=64, H=4, M=32, ptrs=None, ws=_P, ws_bytes=1 << 30):
    lib = _lib()
    p = ptrs or [_P] * 8
    return lib.flarepp_mixer_forward(dtype, B, N, C, H, M, *p, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), fp.ERR_INVALID_ARG),
    (dict(N=0), fp.ERR_INVALID_ARG),
    (dict(M=0), fp.ERR_INVALID_ARG),
    (dict(H=0), fp.ERR_INVALID_ARG),
    (dict(C=100, H=3), fp.ERR_INVALID_ARG),
    (dict(C=96, H=2), fp.ERR_UNSUPPORTED),     # D = 48
    (dict(C=32, H=4), fp.ERR_UNSUPPORTED),     # D = 8
    (dict(C=48, H=3), fp.ERR_UNSUPPORTED),     # C not a multiple of 32
    (dict(dtype=3), fp.ERR_UNSUPPORTED),
    (dict(ws=None), fp.ERR_WORKSPACE),
    (dict(ws_bytes=100), fp.ERR_WORKSPACE),
])
def test_mixer_rejects_invalid_arguments(kw, code):
    assert _mixer(**kw) == code
    assert fp.last_error() != ""


def test_mixer_rejects_null_and_misaligned_pointers():
    for i in range(8):
        ptrs = [_P] * 8
        ptrs[i] = None
        assert _mixer(ptrs=ptrs) == fp.ERR_INVALID_ARG
        ptrs[i] = ctypes.c_void_p(4096 + 8)
        assert _mixer(ptrs=ptrs) == fp.ERR_INVALID_ARG
        assert "aligned" in fp.last_error()


def test_route_rejects_invalid_arguments():
    lib = _lib()

    def call(kind=fp.ENCODE, dtype=fp.BF16, B=1, H=2, N=64, M=32, D=16, stride=0, lse=None,
             ws=_P, wsb=1 << 30):
        return lib.flarepp_route(kind, dtype, B, H, N, M, D, _P, stride, _P, _P, _P, lse, ws, wsb, None)

    assert call(kind=2) == fp.ERR_UNSUPPORTED
    assert call(D=24) == fp.ERR_UNSUPPORTED
    assert call(N=0) == fp.ERR_INVALID_ARG
    assert call(M=-1) == fp.ERR_INVALID_ARG
    assert call(stride=5) == fp.ERR_INVALID_ARG
    assert call(kind=fp.DECODE, lse=_P) == fp.ERR_INVALID_ARG
    assert call(ws=None) == fp.ERR_WORKSPACE
    assert call(wsb=16) == fp.ERR_WORKSPACE


def test_project_rejects_unpaired_weights():
    lib = _lib()
    p = [_P, _P, None, None, _P, None, None, None]  # Wk, Wv given; outputs K only
    rc = lib.flarepp_project(fp.BF16, 1, 64, 64, 4, _P, *p, _P, 1 << 20, None)
    assert rc == fp.ERR_INVALID_ARG
    rc = lib.flarepp_project(fp.BF16, 1, 64, 64, 4, _P, *([None] * 8), _P, 1 << 20, None)
    assert rc == fp.ERR_INVALID_ARG
    rc = lib.flarepp_project(fp.BF16, 1, 64, 64, 4, _P, _P, None, None, None, _P, None, None, None,
                             _P, 16, None)
    assert rc == fp.ERR_WORKSPACE


def _flare(dtype=fp.BF16, B=1, N=64, C=64, H=4, M=32, ptrs=None, ws=_P, ws_bytes=1 << 30):
    lib = _lib()
    p = ptrs or [_P] * 6  # X, Wk, Wv, Wo, queries, O
    return lib.flarepp_flare_forward(dtype, B, N, C, H, M, *p, ws, ws_bytes, None)


def test_flare_workspace_is_smaller_than_the_mixer_one(monkeypatch):
    for dt in (fp.F32, fp.BF16):
        for unfused in (False, True):
            if unfused:
                monkeypatch.setenv("FLAREPP_UNFUSED", "1")
            f = fp.flarepp_flare_workspace_bytes(dt, 4, 16384, 128, 8, 128)
            m = fp.flarepp_mixer_workspace_bytes(dt, 4, 16384, 128, 8, 128)
            monkeypatch.delenv("FLAREPP_UNFUSED", raising=False)
            assert 0 < f < m
    assert fp.flarepp_flare_workspace_bytes(fp.BF16, 1, 10, 100, 3, 4) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), fp.ERR_INVALID_ARG),
    (dict(M=0), fp.ERR_INVALID_ARG),
    (dict(C=96, H=2), fp.ERR_UNSUPPORTED),
    (dict(dtype=3), fp.ERR_UNSUPPORTED),
    (dict(ws=None), fp.ERR_WORKSPACE),
    (dict(ws_bytes=100), fp.ERR_WORKSPACE),
])
def test_flare_rejects_invalid_arguments(kw, code):
    assert _flare(**kw) == code
    assert fp.last_error() != ""


def test_flare_rejects_null_and_misaligned_pointers():
    for i in range(6):
        ptrs = [_P] * 6
        ptrs[i] = None
        assert _flare(ptrs=ptrs) == fp.ERR_INVALID_ARG
        ptrs[i] = ctypes.c_void_p(4096 + 4)
        assert _flare(ptrs=ptrs) == fp.ERR_INVALID_ARG


def _backward(dtype=fp.BF16, B=1, N=64, C=64, H=4, M=32, ptrs=None, ws=_P, ws_bytes=1 << 40):
    lib = _lib()
    p = ptrs or [_P] * 15  # X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, dX, dWk, dWv, dWkt, dWvt, dWo, dseeds
    return lib.flarepp_mixer_backward(dtype, B, N, C, H, M, *p, ws, ws_bytes, None)


def test_backward_workspace_sizes():
    for dt in (fp.F32, fp.BF16):
        bs = 4 if dt == fp.F32 else 2
        n = fp.flarepp_mixer_backward_workspace_bytes(dt, 4, 16384, 128, 8, 128)
        # K, K~, V, V~, Y and the five token gradients dY, dK, dV, dK~, dV~
        assert n >= 4 * 16384 * 128 * 10 * bs
    # every route count is covered (the kernel walks the routes in windows)
    assert fp.flarepp_mixer_backward_workspace_bytes(fp.BF16, 1, 100, 128, 2, 512) > 0
    assert fp.flarepp_mixer_backward_workspace_bytes(fp.BF16, 1, 100, 128, 2, 256) > 0
    assert fp.flarepp_mixer_backward_workspace_bytes(fp.BF16, 1, 100, 128, 8, 512) > 0
    assert fp.flarepp_mixer_backward_workspace_bytes(fp.BF16, 1, 10, 100, 3, 4) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), fp.ERR_INVALID_ARG),
    (dict(N=0), fp.ERR_INVALID_ARG),
    (dict(C=96, H=2), fp.ERR_UNSUPPORTED),
    (dict(dtype=3), fp.ERR_UNSUPPORTED),
    (dict(ws=None), fp.ERR_WORKSPACE),
    (dict(ws_bytes=100), fp.ERR_WORKSPACE),
])
def test_backward_rejects_invalid_arguments(kw, code):
    assert _backward(**kw) == code
    assert fp.last_error() != ""


def test_backward_rejects_null_and_misaligned_pointers():
    for i in range(15):
        ptrs = [_P] * 15
        ptrs[i] = None
        assert _backward(ptrs=ptrs) == fp.ERR_INVALID_ARG
        ptrs[i] = ctypes.c_void_p(4096 + 4)
        assert _backward(ptrs=ptrs) == fp.ERR_INVALID_ARG


def test_shared_variant_rejects_invalid_arguments():
    lib = _lib()
    assert lib.flarepp_mixer_forward_shared(fp.BF16, 0, 64, 64, 4, 32, *([_P] * 6), _P, 1 << 30, None) == fp.ERR_INVALID_ARG
    assert lib.flarepp_mixer_forward_shared(fp.BF16, 1, 64, 64, 4, 32, None, *([_P] * 5), _P, 1 << 30, None) == fp.ERR_INVALID_ARG
    assert lib.flarepp_mixer_forward_shared(fp.BF16, 1, 64, 64, 4, 32, *([_P] * 6), _P, 16, None) == fp.ERR_WORKSPACE


def _block(dtype=fp.BF16, B=1, N=64, C=64, H=4, M=32, eps=1e-5, ptrs=None, ws=_P, ws_bytes=1 << 30):
    # X, gamma, beta, Wk, Wv, Wkt, Wvt, Wo, seeds, O: O differs from X unless
    # a test makes them alias
    ptrs = ptrs if ptrs is not None else [_P] * 9 + [ctypes.c_void_p(8192)]
    return _lib().flarepp_block_forward(dtype, B, N, C, H, M, *ptrs[:3], eps, *ptrs[3:], ws, ws_bytes, None)


def test_block_workspace_adds_the_normalised_input():
    for dt, bs in ((fp.F32, 4), (fp.BF16, 2)):
        m = fp.flarepp_mixer_workspace_bytes(dt, 2, 1000, 128, 8, 64)
        assert fp.flarepp_block_workspace_bytes(dt, 2, 1000, 128, 8, 64) >= m + 2 * 1000 * 128 * bs
    assert fp.flarepp_block_workspace_bytes(fp.BF16, 1, 10, 100, 3, 4) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), fp.ERR_INVALID_ARG),
    (dict(C=96, H=2), fp.ERR_UNSUPPORTED),
    (dict(dtype=3), fp.ERR_UNSUPPORTED),
    (dict(eps=0.0), fp.ERR_INVALID_ARG),
    (dict(eps=-1.0), fp.ERR_INVALID_ARG),
    (dict(eps=float("nan")), fp.ERR_INVALID_ARG),
    (dict(ws=None), fp.ERR_WORKSPACE),
    (dict(ws_bytes=100), fp.ERR_WORKSPACE),
    (dict(ptrs=[_P] * 10), fp.ERR_INVALID_ARG),  # O aliases X
])
def test_block_rejects_invalid_arguments(kw, code):
    assert _block(**kw) == code
    assert fp.last_error() != ""


def test_block_rejects_null_and_misaligned_pointers():
    for i in range(10):
        ptrs = [_P] * 9 + [ctypes.c_void_p(8192)]
        ptrs[i] = None
        assert _block(ptrs=ptrs) == fp.ERR_INVALID_ARG
        ptrs[i] = ctypes.c_void_p(4096 + 4 if i != 9 else 8192 + 4)
        assert _block(ptrs=ptrs) == fp.ERR_INVALID_ARG


def test_shared_backward_rejects_invalid_arguments():
    lib = _lib()
    args = lambda B=1, ptrs=None, ws=_P, nbytes=1 << 30: lib.flarepp_mixer_backward_shared(
        fp.BF16, B, 64, 64, 4, 32, *(ptrs or [_P] * 11), ws, nbytes, None)
    assert args(B=0) == fp.ERR_INVALID_ARG
    assert args(ws=None) == fp.ERR_WORKSPACE
    assert args(nbytes=16) == fp.ERR_WORKSPACE
    for i in range(11):
        ptrs = [_P] * 11
        ptrs[i] = None
        assert args(ptrs=ptrs) == fp.ERR_INVALID_ARG


def test_training_pair_rejects_invalid_arguments():
    lib = _lib()
    fwd = lambda B=1, ptrs=None, ws=_P, nbytes=1 << 30: lib.flarepp_mixer_forward_train(
        fp.BF16, B, 64, 64, 4, 32, *(ptrs or [_P] * 8), ws, nbytes, None)
    assert fwd(B=0) == fp.ERR_INVALID_ARG
    assert fwd(ws=None) == fp.ERR_WORKSPACE
    assert fwd(nbytes=16) == fp.ERR_WORKSPACE
    for i in range(8):
        ptrs = [_P] * 8
        ptrs[i] = None
        assert fwd(ptrs=ptrs) == fp.ERR_INVALID_ARG
    bwd = lambda B=1, ptrs=None, ws=_P, nbytes=1 << 30: lib.flarepp_mixer_backward_from_saved(
        fp.BF16, B, 64, 64, 4, 32, *(ptrs or [_P] * 15), ws, nbytes, None)
    assert bwd(B=0) == fp.ERR_INVALID_ARG
    assert bwd(nbytes=16) == fp.ERR_WORKSPACE
    for i in range(15):
        ptrs = [_P] * 15
        ptrs[i] = None
        assert bwd(ptrs=ptrs) == fp.ERR_INVALID_ARG


def test_block_backward_rejects_invalid_arguments():
    lib = _lib()
    call = lambda B=1, eps=1e-5, ptrs=None, ws=_P, nbytes=1 << 30: lib.flarepp_block_backward(
        fp.BF16, B, 64, 64, 4, 32, *([_P] * 3 if ptrs is None else ptrs[:3]), eps, *([_P] * 7 if ptrs is None else ptrs[3:10]),
        *([_P] * 9 if ptrs is None else ptrs[10:]), ws, nbytes, None)
    assert call(B=0) == fp.ERR_INVALID_ARG
    assert call(eps=0.0) == fp.ERR_INVALID_ARG
    assert call(ws=None) == fp.ERR_WORKSPACE
    assert call(nbytes=16) == fp.ERR_WORKSPACE
    for i in range(19):
        ptrs = [_P] * 19
        ptrs[i] = None
        assert call(ptrs=ptrs) == fp.ERR_INVALID_ARG
    n = fp.flarepp_block_backward_workspace_bytes(fp.BF16, 2, 1000, 128, 8, 64)
    assert n > fp.flarepp_mixer_backward_workspace_bytes(fp.BF16, 2, 1000, 128, 8, 64) + 4 * 2 * 1000 * 128


def test_noalloc_rejects_shapes_beyond_its_scratch_array_before_any_hip_call():
    lib = _lib()
    cap = fp.flarepp_mixer_noalloc_max_bytes()
    assert cap == 32 << 20
    p = ctypes.c_void_p(256)  # aligned, never dereferenced: the checks come first
    ptrs = [p] * 8
    # a fused shape whose workspace exceeds the array
    B, N, C, H, M = 64, 4096, 128, 8, 512
    assert fp.flarepp_mixer_path(fp.BF16, B, N, C, H, M) == fp.PATH_FUSED
    assert fp.flarepp_mixer_workspace_bytes(fp.BF16, B, N, C, H, M) > cap
    rc = lib.flarepp_mixer_forward_noalloc(fp.BF16, B, N, C, H, M, *ptrs, None)
    assert rc == fp.ERR_WORKSPACE and "scratch" in fp.last_error()
    # a shape on the unfused path (C = 512)
    assert fp.flarepp_mixer_path(fp.BF16, 1, 100, 512, 8, 32) == fp.PATH_UNFUSED
    rc = lib.flarepp_mixer_forward_noalloc(fp.BF16, 1, 100, 512, 8, 32, *ptrs, None)
    assert rc == fp.ERR_UNSUPPORTED
    # invalid shapes as for the mixer
    assert lib.flarepp_mixer_forward_noalloc(fp.BF16, 1, 100, 100, 3, 32, *ptrs, None) == fp.ERR_INVALID_ARG

"""libkvr_model without a GPU: the library loads next to libkvr, exports what
include/kvr_model.h declares, and rejects invalid arguments on the host
before any HIP call (fake, never dereferenced pointers)."""
import ctypes
import os

import pytest

from paper_2606_13361_amd import kvr
from paper_2606_13361_amd import kvr_model as M

from test_abi_cpu import A, MIS, desc, exported_symbols, lib  # noqa: F401  (lib: builds if needed)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SZ_MAX = ctypes.c_size_t(-1).value


@pytest.fixture(scope="module")
def mlib(lib):   # noqa: F811
    if not os.path.exists(M.LIB_PATH):
        from paper_2606_13361_amd import build
        build.build()
    return M.load()


def test_exports_match_header(mlib):
    import re
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "kvr_model.h")).read(), flags=re.S)
    declared = sorted(set(re.findall(r"\b(kvr_[a-z0-9_]+)\s*\(", text)))
    assert set(declared) == set(M.EXPORTS)
    assert set(declared) <= exported_symbols(M.LIB_PATH)
    assert mlib.kvr_model_abi_version() == 1


def shape(**kw):
    s = dict(hidden=2560, intermediate=9728, eps=1e-6, reserved=0)
    s.update(kw)
    return M.kvr_layer_shape(s["hidden"], s["intermediate"], s["eps"], s["reserved"])


def weights(**kw):
    w = M.kvr_layer_weights(*([A] * 8))
    for k, v in kw.items():
        setattr(w, k, v)
    return w


def fwd(mlib, d=None, sh=None, w=None, rope=None, blas=A, h=A, T=8, Lp=0, kc=A, vc=A, ws=A, wsb=1 << 40):
    d = d or desc(capacity=4096)
    sh = sh or shape()
    w = w or weights()
    rope = rope if rope is not None else kvr.kvr_rope(A, 4096)
    return mlib.kvr_layer_forward(ctypes.byref(d), ctypes.byref(sh), ctypes.byref(w) if w != "null" else None,
                                  ctypes.byref(rope) if rope != "null" else None, blas, h, T, Lp, kc, vc, ws, wsb,
                                  None)


def test_layer_forward_errors(mlib):
    assert fwd(mlib, d=desc(dtype=kvr.KVR_F32)) == kvr.KVR_ERR_DTYPE
    assert fwd(mlib, d=desc(head_dim=96)) == kvr.KVR_ERR_SHAPE
    assert fwd(mlib, sh=shape(hidden=100)) == kvr.KVR_ERR_SHAPE
    assert fwd(mlib, sh=shape(intermediate=0)) == kvr.KVR_ERR_SHAPE
    assert fwd(mlib, sh=shape(reserved=1)) == kvr.KVR_ERR_SHAPE
    assert fwd(mlib, sh=shape(eps=-1.0)) == kvr.KVR_ERR_SHAPE
    assert fwd(mlib, T=-1) == kvr.KVR_ERR_SHAPE
    # (token, head) waves beyond a 32-bit grid
    assert fwd(mlib, d=desc(n_q_heads=4096, n_kv_heads=8, capacity=1 << 24), T=1 << 19) == kvr.KVR_ERR_SHAPE
    assert fwd(mlib, d=desc(capacity=100), T=50, Lp=60) == kvr.KVR_ERR_CAPACITY
    assert fwd(mlib, T=0, w="null", rope="null", blas=None, h=None) == kvr.KVR_OK
    assert fwd(mlib, w="null") == kvr.KVR_ERR_NULL
    assert fwd(mlib, w=weights(wd=None)) == kvr.KVR_ERR_NULL
    assert fwd(mlib, rope="null") == kvr.KVR_ERR_NULL
    for kw in ("blas", "h", "kc", "vc", "ws"):
        assert fwd(mlib, **{kw: None}) == kvr.KVR_ERR_NULL, kw
    assert fwd(mlib, rope=kvr.kvr_rope(A, 100), T=8, Lp=95) == kvr.KVR_ERR_POSITION
    need = mlib.kvr_layer_workspace_bytes(ctypes.byref(desc(capacity=4096)), ctypes.byref(shape()), 8, 0)
    assert fwd(mlib, wsb=need - 1) == kvr.KVR_ERR_WORKSPACE
    assert fwd(mlib, h=MIS) == kvr.KVR_ERR_ALIGN
    assert fwd(mlib, w=weights(wqkv=MIS)) == kvr.KVR_ERR_ALIGN


def test_workspace_bytes(mlib):
    d, sh = desc(capacity=1 << 16), shape()
    f = lambda T, L: mlib.kvr_layer_workspace_bytes(ctypes.byref(d), ctypes.byref(sh), T, L)   # noqa: E731
    up = lambda b: (b + 255) // 256 * 256                                                        # noqa: E731
    T = 24
    acts = [T * 2560, T * 6144, T * 4096, T * 1024, T * 1024, T * 4096, T * 19456, T * 9728]
    base = sum(up(2 * a) for a in acts) + (32 << 20)
    assert f(T, 0) == base + up(kvr.kvr_workspace_bytes(d, 0, T))
    assert f(T, 32768) == base + up(kvr.kvr_workspace_bytes(d, 32768, T))
    assert f(T, 32768) >= f(T, 4096) >= f(T, 0)
    assert f(-1, 0) == SZ_MAX
    assert mlib.kvr_layer_workspace_bytes(ctypes.byref(desc(dtype=kvr.KVR_F32)), ctypes.byref(sh), 4, 0) == SZ_MAX


def test_linear_and_rmsnorm_errors(mlib):
    lin = lambda blas=A, dt=kvr.KVR_BF16, x=A, w=A, rows=4, ni=64, no=64, beta=0.0, y=A, ws=A, wsb=32 << 20: \
        mlib.kvr_linear(blas, dt, x, w, rows, ni, no, beta, y, ws, wsb, None)   # noqa: E731
    assert lin(dt=kvr.KVR_F32) == kvr.KVR_ERR_DTYPE
    assert lin(ni=60) == kvr.KVR_ERR_SHAPE
    assert lin(rows=-1) == kvr.KVR_ERR_SHAPE
    assert lin(beta=0.5) == kvr.KVR_ERR_SHAPE
    assert lin(rows=0, blas=None, x=None) == kvr.KVR_OK
    for kw in ("blas", "x", "w", "y", "ws"):
        assert lin(**{kw: None}) == kvr.KVR_ERR_NULL, kw
    assert lin(wsb=(32 << 20) - 1) == kvr.KVR_ERR_WORKSPACE
    assert lin(y=MIS) == kvr.KVR_ERR_ALIGN
    rms = lambda dt=kvr.KVR_BF16, x=A, w=A, rows=4, n=64, eps=1e-6, y=A: \
        mlib.kvr_rmsnorm(dt, x, w, rows, n, eps, y, None)   # noqa: E731
    assert rms(dt=kvr.KVR_F32) == kvr.KVR_ERR_DTYPE
    assert rms(n=12) == kvr.KVR_ERR_SHAPE
    assert rms(eps=float("nan")) == kvr.KVR_ERR_SHAPE
    assert rms(rows=0, x=None) == kvr.KVR_OK
    assert rms(w=None) == kvr.KVR_ERR_NULL
    assert rms(x=MIS) == kvr.KVR_ERR_ALIGN
    assert mlib.kvr_blas_create(None) == kvr.KVR_ERR_NULL
    assert mlib.kvr_blas_destroy(None) == kvr.KVR_ERR_NULL

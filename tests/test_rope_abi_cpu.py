"""Host-side validation of the RoPE entry points (no GPU: fake, never
dereferenced pointers; every error returns before any HIP call)."""
import ctypes

import pytest

from paper_2606_13361_amd import kvr

from test_abi_cpu import A, MIS, desc, lib  # noqa: F401  (the fixture)

SZ_MAX = ctypes.c_size_t(-1).value


def rope(n_pos=4096, cs=A):
    return kvr.kvr_rope(cs, n_pos)


def table(lib, d=128, base=1e6, n=16, cs=A):
    return lib.kvr_rope_table(d, base, n, cs, None)


def apply_(lib, d, r, n_tok=4, n_heads=8, pos0=0, x=A, y=A):
    return lib.kvr_rope_apply(ctypes.byref(d), ctypes.byref(r) if r is not None else None, x, n_tok, n_heads,
                              pos0, y, None)


def prefill(lib, d, r, L=16, Q=A, K=A, V=A, out=A, kc=A, vc=A):
    return lib.kvr_prefill_rope(ctypes.byref(d), ctypes.byref(r) if r is not None else None, Q, K, V, L, out,
                                kc, vc, None)


def cont(lib, d, r, Lp=64, S=8, append=0, Q=A, K=A, V=A, kc=A, vc=A, out=A, ws=A, wsb=1 << 30):
    return lib.kvr_continue_rope(ctypes.byref(d), ctypes.byref(r) if r is not None else None, Q, K, V, kc, vc,
                                 Lp, S, append, out, ws, wsb, None)


def batched(lib, d, r, cu, Lp=64, Q=A, K=A, V=A, kc=A, vc=A, out=A, ws=A, wsb=1 << 30):
    arr = (ctypes.c_int32 * len(cu))(*cu)
    return lib.kvr_continue_batched_rope(ctypes.byref(d), ctypes.byref(r) if r is not None else None, Q, K, V,
                                         arr, len(cu) - 1, kc, vc, Lp, out, ws, wsb, None)


def test_table_errors(lib):
    assert table(lib, d=96) == kvr.KVR_ERR_SHAPE
    for base in (0.0, -2.0, float("inf"), float("nan")):
        assert table(lib, base=base) == kvr.KVR_ERR_POSITION, base
    assert table(lib, n=-1) == kvr.KVR_ERR_POSITION
    assert table(lib, n=0, cs=None) == kvr.KVR_OK
    assert table(lib, cs=None) == kvr.KVR_ERR_NULL
    assert table(lib, cs=MIS) == kvr.KVR_ERR_ALIGN


def test_apply_errors(lib):
    d = desc()
    assert apply_(lib, d, rope(), n_tok=-1) == kvr.KVR_ERR_SHAPE
    assert apply_(lib, d, rope(), n_heads=0) == kvr.KVR_ERR_SHAPE
    assert apply_(lib, d, rope(), pos0=-1) == kvr.KVR_ERR_POSITION
    assert apply_(lib, d, rope(), n_tok=0, x=None, y=None) == kvr.KVR_OK
    assert apply_(lib, d, None) == kvr.KVR_ERR_NULL
    assert apply_(lib, d, rope(cs=None)) == kvr.KVR_ERR_NULL
    assert apply_(lib, d, rope(n_pos=10), n_tok=4, pos0=7) == kvr.KVR_ERR_POSITION   # needs positions 7..10
    assert apply_(lib, d, rope(cs=MIS)) == kvr.KVR_ERR_ALIGN
    assert apply_(lib, d, rope(), x=MIS) == kvr.KVR_ERR_ALIGN
    assert apply_(lib, desc(dtype=7), rope()) == kvr.KVR_ERR_DTYPE


def test_prefill_errors(lib):
    d = desc(capacity=100)
    assert prefill(lib, d, rope(), L=101) == kvr.KVR_ERR_CAPACITY
    assert prefill(lib, d, None, L=0) == kvr.KVR_OK
    assert prefill(lib, d, None) == kvr.KVR_ERR_NULL
    assert prefill(lib, d, rope(n_pos=15), L=16) == kvr.KVR_ERR_POSITION
    for kw in ("Q", "K", "V", "out", "kc", "vc"):
        assert prefill(lib, d, rope(), **{kw: None}) == kvr.KVR_ERR_NULL, kw
        assert prefill(lib, d, rope(), **{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw


def test_continue_errors(lib):
    d = desc(capacity=100)
    assert cont(lib, d, rope(), Lp=101) == kvr.KVR_ERR_CAPACITY
    assert cont(lib, d, rope(), Lp=95, S=8, append=1) == kvr.KVR_ERR_CAPACITY   # rows 95..102
    assert cont(lib, d, rope(), S=0, Q=None, K=None, V=None, out=None, ws=None) == kvr.KVR_OK
    assert cont(lib, d, rope(n_pos=71), Lp=64, S=8) == kvr.KVR_ERR_POSITION    # positions 64..71
    assert cont(lib, d, None) == kvr.KVR_ERR_NULL
    assert cont(lib, d, rope(), Lp=0, kc=None, vc=None, append=1) == kvr.KVR_ERR_NULL
    need = lib.kvr_workspace_bytes_rope(ctypes.byref(d), 64, 8, 1)
    assert cont(lib, d, rope(), wsb=need - 1) == kvr.KVR_ERR_WORKSPACE
    for kw in ("Q", "K", "V", "out", "kc", "vc", "ws"):
        assert cont(lib, d, rope(), **{kw: None}) == kvr.KVR_ERR_NULL, kw
        assert cont(lib, d, rope(), **{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw


def test_batched_errors(lib):
    d = desc(capacity=100)
    assert batched(lib, d, rope(), [0, 4, 3]) == kvr.KVR_ERR_SHAPE
    assert batched(lib, d, None, [0, 0, 0]) == kvr.KVR_OK                 # only empty readers
    assert batched(lib, d, rope(n_pos=64 + 9), [0, 4, 14], Lp=64) == kvr.KVR_ERR_POSITION   # longest reader: 10
    assert batched(lib, d, rope(n_pos=64 + 10), [0, 4, 14], Lp=64, ws=None) == kvr.KVR_ERR_NULL
    need = lib.kvr_workspace_bytes_rope(ctypes.byref(d), 64, 14, 2)
    assert batched(lib, d, rope(), [0, 4, 14], wsb=need - 1) == kvr.KVR_ERR_WORKSPACE
    assert batched(lib, d, rope(), [0, 4, 14], ws=MIS) == kvr.KVR_ERR_ALIGN


@pytest.mark.parametrize("dtype,elt", [(kvr.KVR_BF16, 2), (kvr.KVR_F16, 2), (kvr.KVR_F32, 4)])
def test_workspace_bytes(lib, dtype, elt):
    d = desc(dtype=dtype, capacity=1 << 16)
    f = lambda Lp, S, n=1: lib.kvr_workspace_bytes_rope(ctypes.byref(d), Lp, S, n)   # noqa: E731
    g = lambda Lp, S, n=1: lib.kvr_workspace_bytes(ctypes.byref(d), Lp, S, n)        # noqa: E731
    up = lambda b: (b + 255) // 256 * 256                                              # noqa: E731
    for Lp, S in ((0, 24), (4096, 24), (32768, 1), (32768, 300)):
        # the plain split partials, then rotated Q rows and rotated K rows
        assert f(Lp, S) == up(g(Lp, S)) + up(S * 32 * 128 * elt) + up(S * 8 * 128 * elt)
    # readers: the split partials of their last tiles (bf16 / fp16), then the rotated keys
    assert f(3774, 8424, 64) == up(g(3774, 8424, 64)) + up(8424 * 8 * 128 * elt)
    assert (g(3774, 8424, 64) > 0) == (dtype != kvr.KVR_F32)
    assert f(-1, 3) == SZ_MAX
    sizes = [f(L, 24) for L in range(0, 40000, 211)]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))

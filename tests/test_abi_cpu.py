"""The C ABI without a GPU: the library loads, exports what include/kvr.h
declares, and rejects every invalid argument on the host before any HIP call.

Pointers here are fake integers (never dereferenced): validation returns
before any launch, so no device is touched.
"""
import ctypes
import os
import re

import pytest

from paper_2606_13361_amd import kvr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvr.h")

A = 0x1000          # a 16-byte-aligned fake device pointer
MIS = 0x1008        # 8-byte aligned only


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(kvr.LIB_PATH):
        from paper_2606_13361_amd import build
        build.build()
    return kvr.load()


def desc(**kw):
    d = dict(n_q_heads=32, n_kv_heads=8, head_dim=128, dtype=kvr.KVR_BF16, capacity=4096, scale=0.0)
    d.update(kw)
    return kvr.make_desc(d["n_q_heads"], d["n_kv_heads"], d["head_dim"], d["dtype"], d["capacity"], d["scale"])


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvr_[a-z0-9_]+)\s*\(", text)))


def exported_symbols(path):
    """Dynamic symbol names of the shared library, read from its ELF tables."""
    import struct
    data = open(path, "rb").read()
    assert data[:4] == b"\x7fELF" and data[4] == 2    # 64-bit
    shoff, = struct.unpack_from("<Q", data, 0x28)
    shentsize, shnum, _ = struct.unpack_from("<HHH", data, 0x3A)
    secs = [struct.unpack_from("<IIQQQQIIQQ", data, shoff + i * shentsize) for i in range(shnum)]
    names = set()
    for s in secs:
        if s[1] == 11:                         # SHT_DYNSYM
            strtab = secs[s[6]]
            off, size, ent = s[4], s[5], s[9]
            for k in range(size // ent):
                st_name, st_info, _, st_shndx, _, _ = struct.unpack_from("<IBBHQQ", data, off + k * ent)
                if st_shndx != 0 and (st_info >> 4) == 1:   # defined, global
                    nm = data[strtab[4] + st_name: data.index(b"\0", strtab[4] + st_name)]
                    names.add(nm.decode())
    return names


def test_exports_match_header(lib):
    declared = header_functions()
    assert set(declared) == set(kvr.EXPORTS)
    syms = exported_symbols(kvr.LIB_PATH)
    for name in declared:
        assert name in syms, name
        assert hasattr(lib, name)


def test_abi_version_and_strerror(lib):
    assert lib.kvr_abi_version() == 4
    for code in range(11):
        assert len(lib.kvr_strerror(code)) > 0
    assert b"unknown" in lib.kvr_strerror(99)


def prefill(lib, d, L=16, Q=A, K=A, V=A, out=A, kc=A, vc=A):
    return lib.kvr_prefill(ctypes.byref(d), Q, K, V, L, out, kc, vc, None)


def cont(lib, d, Lp=64, S=8, Q=A, K=A, V=A, kc=A, vc=A, out=A, ws=A, wsb=1 << 30):
    return lib.kvr_continue(ctypes.byref(d), Q, K, V, kc, vc, Lp, S, out, ws, wsb, None)


def append(lib, d, S=4, Lc=0, K=A, V=A, kc=A, vc=A):
    return lib.kvr_cache_append(ctypes.byref(d), K, V, S, kc, vc, Lc, None)


def batched(lib, d, cu, Lp=64, Q=A, K=A, V=A, kc=A, vc=A, out=A):
    arr = (ctypes.c_int32 * len(cu))(*cu)
    return lib.kvr_continue_batched(ctypes.byref(d), Q, K, V, arr, len(cu) - 1, kc, vc, Lp, out, None, 0, None)


@pytest.mark.parametrize("bad,code", [
    (dict(n_q_heads=30, n_kv_heads=8), kvr.KVR_ERR_SHAPE),   # Hq % Hkv != 0
    (dict(n_q_heads=0), kvr.KVR_ERR_SHAPE),
    (dict(n_kv_heads=0), kvr.KVR_ERR_SHAPE),
    (dict(head_dim=96), kvr.KVR_ERR_SHAPE),
    (dict(head_dim=256), kvr.KVR_ERR_SHAPE),
    (dict(dtype=7), kvr.KVR_ERR_DTYPE),
    (dict(dtype=3), kvr.KVR_ERR_DTYPE),
    (dict(capacity=-1), kvr.KVR_ERR_SHAPE),
    (dict(scale=float("nan")), kvr.KVR_ERR_SHAPE),
])
def test_descriptor_errors(lib, bad, code):
    d = desc(**bad)
    assert prefill(lib, d) == code
    assert cont(lib, d) == code
    assert append(lib, d) == code
    assert batched(lib, d, [0, 4]) == code
    assert lib.kvr_workspace_bytes(ctypes.byref(d), 64, 8, 1) == ctypes.c_size_t(-1).value


def test_fp16_descriptor(lib):
    """fp16 (the paper's precision) is a valid dtype everywhere bf16 is, with the
    same workspace; the int8 artifact is a bf16 model's only."""
    d16, db = desc(dtype=kvr.KVR_F16), desc()
    assert prefill(lib, d16, L=0, Q=None, K=None, V=None, out=None, kc=None, vc=None) == kvr.KVR_OK
    assert cont(lib, d16, Lp=0, S=0) == kvr.KVR_OK
    assert prefill(lib, d16, L=-1) == kvr.KVR_ERR_SHAPE
    for Lp, S in ((3774, 24), (32768, 1), (100, 200)):
        assert lib.kvr_workspace_bytes(ctypes.byref(d16), Lp, S, 1) == lib.kvr_workspace_bytes(ctypes.byref(db), Lp, S, 1)
    assert quant(lib, d16) == kvr.KVR_ERR_DTYPE
    assert cont_q8(lib, d16) == kvr.KVR_ERR_DTYPE
    assert lib.kvr_artifact_bytes(ctypes.byref(d16), 36, 3774) == lib.kvr_artifact_bytes(ctypes.byref(db), 36, 3774)


def test_null_descriptor(lib):
    assert lib.kvr_prefill(None, A, A, A, 4, A, A, A, None) == kvr.KVR_ERR_NULL
    assert lib.kvr_cache_append(None, A, A, 4, A, A, 0, None) == kvr.KVR_ERR_NULL


def test_reserved_field_must_be_zero(lib):
    d = desc()
    d.reserved = 1
    assert prefill(lib, d) == kvr.KVR_ERR_SHAPE


def test_prefill_errors(lib):
    d = desc(capacity=100)
    assert prefill(lib, d, L=-1) == kvr.KVR_ERR_SHAPE
    assert prefill(lib, d, L=101) == kvr.KVR_ERR_CAPACITY
    assert prefill(lib, d, L=0, Q=None, K=None, V=None, out=None, kc=None, vc=None) == kvr.KVR_OK
    for kw in ("Q", "K", "V", "out", "kc", "vc"):
        assert prefill(lib, d, **{kw: None}) == kvr.KVR_ERR_NULL, kw
        assert prefill(lib, d, **{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw


def test_continue_errors(lib):
    d = desc(capacity=100)
    assert cont(lib, d, Lp=-1) == kvr.KVR_ERR_SHAPE
    assert cont(lib, d, S=-2) == kvr.KVR_ERR_SHAPE
    assert cont(lib, d, Lp=101) == kvr.KVR_ERR_CAPACITY
    assert cont(lib, d, S=0, Q=None, K=None, V=None, out=None) == kvr.KVR_OK
    for kw in ("Q", "K", "V", "out", "kc", "vc"):
        assert cont(lib, d, **{kw: None}) == kvr.KVR_ERR_NULL, kw
        assert cont(lib, d, **{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw


def test_continue_workspace(lib):
    d = desc(capacity=8192)
    need = lib.kvr_workspace_bytes(ctypes.byref(d), 4096, 24, 1)
    assert need > 0
    assert cont(lib, d, Lp=4096, S=24, wsb=need - 1) == kvr.KVR_ERR_WORKSPACE
    assert cont(lib, d, Lp=4096, S=24, ws=None, wsb=need) == kvr.KVR_ERR_NULL
    assert cont(lib, d, Lp=4096, S=24, ws=MIS, wsb=need) == kvr.KVR_ERR_ALIGN


def test_workspace_bytes_is_a_pure_plan(lib):
    d = desc(capacity=1 << 16)
    f = lambda Lp, S, n=1, dd=d: lib.kvr_workspace_bytes(ctypes.byref(dd), Lp, S, n)
    assert f(0, 24) == 0                       # nothing cached: no split
    assert f(100, 24) == 0                     # short prefix: one split
    assert f(32768, 24) > f(4096, 24) > 0      # longer prefix: more splits
    assert f(32768, 24) == f(32768, 24)        # deterministic
    assert f(32768, 1) % (8 * 4 * (128 + 2) * 4) == 0   # whole partial rows of fp32
    assert f(32768, 24, 1, desc(dtype=kvr.KVR_F32, capacity=1 << 16)) == 0
    assert f(-1, 3) == ctypes.c_size_t(-1).value
    # never decreases with the prefix length (one buffer for a whole decode chain)
    for S in (1, 24, 100):
        sizes = [f(L, S) for L in range(0, 40000, 97)]
        assert all(a <= b for a, b in zip(sizes, sizes[1:])), S


def test_readers_workspace_plan(lib):
    """Many readers (n >= 2) on the two-group kernel: rows packed across
    readers into tiles of 256, 8 kv heads -> 32 tiles per round of 256
    workgroups; the tiles of a last partial round split over the keys into the
    ns <= min(16, L_prefix // 256) parts whose rounds cost least (a split
    workgroup: 1/ns + 0.07 of a whole one of 2 us per key tile; the merge
    launch: 0.04; the fp32 (O, m, l) records written and read back at 5 TB/s)."""
    d = desc(capacity=1 << 16)
    f = lambda Lp, S, n, dd=d: lib.kvr_workspace_bytes(ctypes.byref(dd), Lp, S, n)
    # 64 readers, 8424 tokens over 3774: 132 tiles, 4 in the last round -> 8 splits
    # of the 8424 * 4 - 128 * 256 = 928 rows per kv head from tile 128 on
    assert f(3774, 8424, 64) == 8 * 8 * 928 * (128 + 2) * 4
    # 3 readers, 301 tokens over 3774: 5 tiles, all split 6 ways
    assert f(3774, 301, 3) == 6 * 8 * 1204 * (128 + 2) * 4
    # 16 readers, 2058 tokens: 33 tiles, one in the last round -> 14 splits (the
    # most with four key tiles each) of 8232 - 32 * 256 = 40 rows
    assert f(3774, 2058, 16) == 14 * 8 * 40 * (128 + 2) * 4
    # 8 readers, 1391 tokens: 22 tiles, one partial round of 176 workgroups; 4
    # splits would take 3 rounds (0.96) but 185 MB of records (0.31): whole
    assert f(3774, 1391, 8) == 0
    assert f(3774, 8192, 64) == 0              # 128 tiles: four full rounds
    assert f(3774, 6000, 64) == 0              # 94 tiles: 30 in the last round
    assert f(511, 301, 3) == 0                 # fewer than 2 x 4 key tiles per split
    assert f(512, 301, 3) == 2 * 8 * 1204 * (128 + 2) * 4
    assert f(3774, 8424, 129) == 0             # more than one launch: no split
    assert f(3774, 8424, 64, desc(n_q_heads=24, capacity=1 << 16)) == 0   # G = 3
    assert f(3774, 8424, 64, desc(head_dim=64, capacity=1 << 16)) == 0    # other kernel
    assert f(3774, 8424, 64, desc(dtype=kvr.KVR_F32, capacity=1 << 16)) == 0
    sizes = [f(L, 301, 3) for L in range(0, 5000, 37)]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))
    # the batched call checks the workspace the plan needs
    need = f(3774, 301, 3)
    cu = [0, 24, 224, 301]
    arr = (ctypes.c_int32 * 4)(*cu)
    call = lambda ws, wsb: lib.kvr_continue_batched(ctypes.byref(d), A, A, A, arr, 3, A, A, 3774, A, ws, wsb, None)
    assert call(A, need - 1) == kvr.KVR_ERR_WORKSPACE
    assert call(None, need) == kvr.KVR_ERR_NULL
    assert call(MIS, need) == kvr.KVR_ERR_ALIGN
    # with RoPE: the partials, then the rotated keys
    rot = 301 * 8 * 128 * 2
    assert lib.kvr_workspace_bytes_rope(ctypes.byref(d), 3774, 301, 3) == (need + 255) // 256 * 256 + \
        (rot + 255) // 256 * 256


def test_append_errors(lib):
    d = desc(capacity=50)
    assert append(lib, d, S=-1) == kvr.KVR_ERR_SHAPE
    assert append(lib, d, Lc=-1) == kvr.KVR_ERR_SHAPE
    assert append(lib, d, S=10, Lc=41) == kvr.KVR_ERR_CAPACITY
    assert append(lib, d, S=0, K=None, V=None, kc=None, vc=None) == kvr.KVR_OK
    for kw in ("K", "V", "kc", "vc"):
        assert append(lib, d, **{kw: None}) == kvr.KVR_ERR_NULL
        assert append(lib, d, **{kw: MIS}) == kvr.KVR_ERR_ALIGN


def test_batched_errors(lib):
    d = desc(capacity=100)
    assert batched(lib, d, [1, 4]) == kvr.KVR_ERR_SHAPE       # cu[0] != 0
    assert batched(lib, d, [0, 4, 3]) == kvr.KVR_ERR_SHAPE    # decreasing
    assert batched(lib, d, [0, 4], Lp=101) == kvr.KVR_ERR_CAPACITY
    assert batched(lib, d, [0]) == kvr.KVR_OK                  # no readers
    assert batched(lib, d, [0, 0, 0], Q=None) == kvr.KVR_OK    # only empty readers
    assert lib.kvr_continue_batched(ctypes.byref(d), A, A, A, None, 2, A, A, 4, A, None, 0, None) == kvr.KVR_ERR_NULL
    assert batched(lib, d, [0, 4], out=MIS) == kvr.KVR_ERR_ALIGN
    assert batched(lib, d, [0, 4], kc=None) == kvr.KVR_ERR_NULL
    # packed rows of one launch (two-group kernel: bf16, d = 128) must fit 32-bit
    # row indices even when each reader's do: G = 4096 (4096 q heads, 1 kv head)
    big = desc(n_q_heads=4096, n_kv_heads=1, capacity=100)
    assert batched(lib, big, [0, 300000, 600000]) == kvr.KVR_ERR_SHAPE        # 4096 x 600000 > 2^31
    assert batched(lib, big, [0, 300000, 600000], Lp=0, Q=None) == kvr.KVR_ERR_SHAPE
    assert batched(lib, big, [0, 200000, 400000], Q=None) == kvr.KVR_ERR_NULL  # 4096 x 400000 < 2^31


def test_python_binding_rejects_metadata_mismatch():
    """The binding refuses tensors whose dtype or shape disagree with the descriptor."""
    import torch
    d = desc(n_q_heads=4, n_kv_heads=2, head_dim=64, capacity=8)
    x = torch.zeros((2, 4, 64), dtype=torch.float32)
    with pytest.raises(ValueError):
        kvr._check(x, "Q", d, (2, 4, 64))       # CPU tensor and fp32 vs bf16


def quant(lib, d, L=64, kc=A, vc=A, kq=A, vq=A, sc=A):
    return lib.kvr_quantize_cache(ctypes.byref(d), kc, vc, L, kq, vq, sc, None)


def cont_q8(lib, d, Lp=64, S=8, Q=A, K=A, V=A, kq=A, vq=A, sc=A, out=A, ws=A, wsb=1 << 30):
    return lib.kvr_continue_q8(ctypes.byref(d), Q, K, V, kq, vq, sc, Lp, S, out, ws, wsb, None)


def test_q8_bytes(lib):
    assert lib.kvr_q8_bytes(ctypes.byref(desc(capacity=4096))) == 8 * 4096 * 128
    assert lib.kvr_q8_bytes(ctypes.byref(desc(capacity=33))) == 8 * 64 * 128      # rows padded to 32
    assert lib.kvr_q8_bytes(ctypes.byref(desc(capacity=0))) == 0
    assert lib.kvr_q8_bytes(ctypes.byref(desc(head_dim=96))) == ctypes.c_size_t(-1).value


def test_quantize_errors(lib):
    d = desc(capacity=100)
    assert quant(lib, desc(dtype=kvr.KVR_F32)) == kvr.KVR_ERR_DTYPE
    assert quant(lib, desc(head_dim=64)) == kvr.KVR_ERR_SHAPE
    assert quant(lib, d, L=-1) == kvr.KVR_ERR_SHAPE
    assert quant(lib, d, L=101) == kvr.KVR_ERR_CAPACITY
    assert quant(lib, d, L=0, kc=None, vc=None, kq=None, vq=None, sc=None) == kvr.KVR_OK
    for kw in ("kc", "vc", "kq", "vq", "sc"):
        assert quant(lib, d, **{kw: None}) == kvr.KVR_ERR_NULL, kw
    for kw in ("kc", "vc", "kq", "vq"):
        assert quant(lib, d, **{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw
    assert quant(lib, d, sc=A + 2) == kvr.KVR_ERR_ALIGN


def test_continue_q8_errors(lib):
    d = desc(capacity=100)
    assert cont_q8(lib, desc(dtype=kvr.KVR_F32)) == kvr.KVR_ERR_DTYPE
    assert cont_q8(lib, desc(head_dim=64)) == kvr.KVR_ERR_SHAPE
    assert cont_q8(lib, d, S=25) == kvr.KVR_ERR_SHAPE           # G * S = 100 > 96 rows
    assert cont_q8(lib, d, Lp=-1) == kvr.KVR_ERR_SHAPE
    assert cont_q8(lib, d, Lp=101) == kvr.KVR_ERR_CAPACITY
    assert cont_q8(lib, d, S=0, Q=None, K=None, V=None, out=None) == kvr.KVR_OK
    for kw in ("Q", "K", "V", "out", "kq", "vq", "sc"):
        assert cont_q8(lib, d, **{kw: None}) == kvr.KVR_ERR_NULL, kw
    for kw in ("Q", "K", "V", "out", "kq", "vq"):
        assert cont_q8(lib, d, **{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw
    d2 = desc(capacity=8192)
    need = lib.kvr_workspace_bytes(ctypes.byref(d2), 4096, 24, 1)
    assert cont_q8(lib, d2, Lp=4096, S=24, wsb=need - 1) == kvr.KVR_ERR_WORKSPACE


def test_continue_append_errors(lib):
    d = desc(capacity=100)
    f = lambda Lp=64, S=8, Q=A, K=A, V=A, kc=A, vc=A, out=A, ws=A, wsb=1 << 30: lib.kvr_continue_append(  # noqa: E731
        ctypes.byref(d), Q, K, V, kc, vc, Lp, S, out, ws, wsb, None)
    assert f(Lp=-1) == kvr.KVR_ERR_SHAPE
    assert f(Lp=95, S=8) == kvr.KVR_ERR_CAPACITY          # the update needs rows 95..102
    assert f(S=0, Q=None, K=None, V=None, kc=None, vc=None, out=None) == kvr.KVR_OK
    for kw in ("Q", "K", "V", "out", "kc", "vc"):
        assert f(**{kw: None}) == kvr.KVR_ERR_NULL, kw    # the caches are written: always needed
        assert f(**{kw: MIS}) == kvr.KVR_ERR_ALIGN, kw


def noalloc(lib, d, Lp=64, S=8, Q=A, K=A, V=A, kc=A, vc=A, out=A):
    return lib.kvr_continue_noalloc(ctypes.byref(d), Q, K, V, kc, vc, Lp, S, out, None)


def test_noalloc_rejections(lib):
    """kvr_continue_noalloc: kvr_continue's argument checks, and a plan whose split
    partials exceed the fixed buffer is KVR_ERR_TOO_LARGE -- all before any HIP call."""
    d = desc(capacity=1 << 20)
    assert noalloc(lib, desc(n_q_heads=30)) == kvr.KVR_ERR_SHAPE
    assert noalloc(lib, desc(dtype=7)) == kvr.KVR_ERR_DTYPE
    assert noalloc(lib, d, Lp=-1) == kvr.KVR_ERR_SHAPE
    assert noalloc(lib, desc(capacity=100), Lp=101) == kvr.KVR_ERR_CAPACITY
    assert noalloc(lib, d, Q=None) == kvr.KVR_ERR_NULL
    assert noalloc(lib, d, kc=None) == kvr.KVR_ERR_NULL
    assert noalloc(lib, d, out=MIS) == kvr.KVR_ERR_ALIGN
    assert noalloc(lib, d, S=0, Q=None, K=None, V=None, out=None) == kvr.KVR_OK
    Lp, S = 20000, 256
    assert lib.kvr_workspace_bytes(ctypes.byref(d), Lp, S, 1) > kvr.KVR_NOALLOC_SCRATCH_BYTES
    assert noalloc(lib, d, Lp=Lp, S=S) == kvr.KVR_ERR_TOO_LARGE
    # the Qwen-shaped 24-token continuation and every decode step fit
    for Lp, S in ((32768, 24), (32768, 1), (1 << 19, 1), (3774, 24)):
        assert lib.kvr_workspace_bytes(ctypes.byref(d), Lp, S, 1) <= kvr.KVR_NOALLOC_SCRATCH_BYTES

"""Python binding of libkvr (include/kvr.h): argument marshalling only.

Every function has the name of the C entry point it calls.  Tensors are torch
tensors on the GPU (PyTorch provides device memory and streams); their
dtype, device, contiguity and shape are checked against the layer descriptor
before the call -- the consumer-side metadata check of the paper's Alg. 2 --
and a ValueError is raised on a mismatch.  A nonzero kvr_status raises
KvrError.  There is no fallback: without the built library every call fails.
"""
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkvr.so")

KVR_OK, KVR_ERR_NULL, KVR_ERR_SHAPE, KVR_ERR_DTYPE = 0, 1, 2, 3
KVR_ERR_CAPACITY, KVR_ERR_WORKSPACE, KVR_ERR_ALIGN, KVR_ERR_DEVICE = 4, 5, 6, 7
KVR_ERR_MISMATCH, KVR_ERR_POSITION, KVR_ERR_TOO_LARGE = 8, 9, 10
KVR_NOALLOC_SCRATCH_BYTES = 16 << 20
KVR_ARTIFACT_HEADER_BYTES = 256
KVR_BF16, KVR_F32, KVR_F16 = 0, 1, 2

EXPORTS = ("kvr_prefill", "kvr_continue", "kvr_continue_append", "kvr_continue_noalloc", "kvr_continue_batched",
           "kvr_cache_append",
           "kvr_workspace_bytes", "kvr_strerror", "kvr_abi_version",
           "kvr_q8_bytes", "kvr_quantize_cache", "kvr_continue_q8",
           "kvr_artifact_bytes", "kvr_artifact_save", "kvr_artifact_load",
           "kvr_rope_table", "kvr_rope_apply", "kvr_prefill_rope", "kvr_continue_rope",
           "kvr_continue_batched_rope", "kvr_workspace_bytes_rope")

_TORCH_DTYPE = {KVR_BF16: torch.bfloat16, KVR_F32: torch.float32, KVR_F16: torch.float16}


class kvr_desc(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float), ("reserved", ctypes.c_int32),
                ("capacity", ctypes.c_int64)]


class kvr_rope(ctypes.Structure):
    _fields_ = [("cos_sin", ctypes.c_void_p), ("n_pos", ctypes.c_int64)]


class KvrError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, strerror(status), status))


_lib = None


def load():
    """Load the in-tree libkvr.so; raise if it was not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libkvr.so is not built (run __graft_entry__.build() or "
                           "python -m paper_2606_13361_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    D = ctypes.POINTER(kvr_desc)
    lib.kvr_prefill.argtypes = [D, P, P, P, I64, P, P, P, P]
    lib.kvr_continue.argtypes = [D, P, P, P, P, P, I64, I64, P, P, SZ, P]
    lib.kvr_continue_append.argtypes = [D, P, P, P, P, P, I64, I64, P, P, SZ, P]
    lib.kvr_continue_noalloc.argtypes = [D, P, P, P, P, P, I64, I64, P, P]
    lib.kvr_continue_batched.argtypes = [D, P, P, P, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                         P, P, I64, P, P, SZ, P]
    lib.kvr_cache_append.argtypes = [D, P, P, I64, P, P, I64, P]
    lib.kvr_workspace_bytes.argtypes = [D, I64, I64, ctypes.c_int32]
    lib.kvr_workspace_bytes.restype = SZ
    lib.kvr_q8_bytes.argtypes = [D]
    lib.kvr_q8_bytes.restype = SZ
    lib.kvr_quantize_cache.argtypes = [D, P, P, I64, P, P, P, P]
    lib.kvr_continue_q8.argtypes = [D, P, P, P, P, P, P, I64, I64, P, P, SZ, P]
    PP = ctypes.POINTER(ctypes.c_void_p)
    lib.kvr_artifact_bytes.argtypes = [D, ctypes.c_int32, I64]
    lib.kvr_artifact_bytes.restype = SZ
    lib.kvr_artifact_save.argtypes = [D, ctypes.c_char_p, ctypes.c_int32, I64, PP, PP, P, SZ, P]
    lib.kvr_artifact_load.argtypes = [D, ctypes.c_char_p, ctypes.c_int32, P, SZ, PP, PP,
                                      ctypes.POINTER(ctypes.c_int64), P]
    R = ctypes.POINTER(kvr_rope)
    lib.kvr_rope_table.argtypes = [ctypes.c_int32, ctypes.c_double, I64, P, P]
    lib.kvr_rope_apply.argtypes = [D, R, P, I64, ctypes.c_int32, I64, P, P]
    lib.kvr_prefill_rope.argtypes = [D, R, P, P, P, I64, P, P, P, P]
    lib.kvr_continue_rope.argtypes = [D, R, P, P, P, P, P, I64, I64, ctypes.c_int32, P, P, SZ, P]
    lib.kvr_continue_batched_rope.argtypes = [D, R, P, P, P, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                              P, P, I64, P, P, SZ, P]
    lib.kvr_workspace_bytes_rope.argtypes = [D, I64, I64, ctypes.c_int32]
    lib.kvr_workspace_bytes_rope.restype = SZ
    lib.kvr_strerror.argtypes = [ctypes.c_int]
    lib.kvr_strerror.restype = ctypes.c_char_p
    lib.kvr_abi_version.argtypes = []
    for f in (lib.kvr_prefill, lib.kvr_continue, lib.kvr_continue_append, lib.kvr_continue_noalloc,
              lib.kvr_continue_batched,
              lib.kvr_cache_append,
              lib.kvr_abi_version, lib.kvr_quantize_cache, lib.kvr_continue_q8, lib.kvr_artifact_save,
              lib.kvr_artifact_load, lib.kvr_rope_table, lib.kvr_rope_apply, lib.kvr_prefill_rope,
              lib.kvr_continue_rope, lib.kvr_continue_batched_rope):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def strerror(status):
    return load().kvr_strerror(int(status)).decode()


def kvr_abi_version():
    return load().kvr_abi_version()


def make_desc(n_q_heads, n_kv_heads, head_dim, dtype, capacity, scale=0.0):
    """dtype: torch.bfloat16 / torch.float16 / torch.float32 or KVR_BF16 / KVR_F16 / KVR_F32."""
    if isinstance(dtype, torch.dtype):
        dtype = {torch.bfloat16: KVR_BF16, torch.float16: KVR_F16, torch.float32: KVR_F32}.get(dtype, -1)
    return kvr_desc(int(n_q_heads), int(n_kv_heads), int(head_dim), int(dtype), float(scale), 0,
                    int(capacity))


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(t, name, desc, shape):
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a torch tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be on the GPU" % name)
    want = _TORCH_DTYPE.get(desc.dtype)
    if t.dtype != want:
        raise ValueError("%s has dtype %s, the layer descriptor says %s" % (name, t.dtype, want))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return t.data_ptr()


def _cache_ptrs(desc, kcache, vcache, required):
    if kcache is None and vcache is None and not required:
        return None, None
    shape = (desc.n_kv_heads, desc.capacity, desc.head_dim)
    return _check(kcache, "kcache", desc, shape), _check(vcache, "vcache", desc, shape)


def _raise(st, where):
    if st != KVR_OK:
        raise KvrError(st, where)


def kvr_workspace_bytes(desc, L_prefix, total_S, n=1):
    return load().kvr_workspace_bytes(ctypes.byref(desc), int(L_prefix), int(total_S), int(n))


def kvr_prefill(desc, Q, K, V, L, out, kcache, vcache, stream=None):
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Q, "Q", desc, (L, Hq, d))
    k = _check(K, "K", desc, (L, Hkv, d))
    v = _check(V, "V", desc, (L, Hkv, d))
    o = _check(out, "out", desc, (L, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, True)
    _raise(load().kvr_prefill(ctypes.byref(desc), q, k, v, int(L), o, kc, vc, _stream(stream)),
           "kvr_prefill")


def kvr_continue(desc, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out, ws=None, stream=None):
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Qs, "Qs", desc, (S, Hq, d))
    k = _check(Ks, "Ks", desc, (S, Hkv, d))
    v = _check(Vs, "Vs", desc, (S, Hkv, d))
    o = _check(out, "out", desc, (S, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, L_prefix > 0)
    wp, wn = _workspace(ws)
    _raise(load().kvr_continue(ctypes.byref(desc), q, k, v, kc, vc, int(L_prefix), int(S), o, wp, wn,
                               _stream(stream)), "kvr_continue")


def kvr_continue_noalloc(desc, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out, stream=None):
    """kvr_continue with its split partials in the library's fixed per-device buffer."""
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Qs, "Qs", desc, (S, Hq, d))
    k = _check(Ks, "Ks", desc, (S, Hkv, d))
    v = _check(Vs, "Vs", desc, (S, Hkv, d))
    o = _check(out, "out", desc, (S, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, L_prefix > 0)
    _raise(load().kvr_continue_noalloc(ctypes.byref(desc), q, k, v, kc, vc, int(L_prefix), int(S), o,
                                       _stream(stream)), "kvr_continue_noalloc")


def kvr_continue_append(desc, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out, ws=None, stream=None):
    """kvr_continue plus the cache update of the S tokens at rows L_prefix.. ."""
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Qs, "Qs", desc, (S, Hq, d))
    k = _check(Ks, "Ks", desc, (S, Hkv, d))
    v = _check(Vs, "Vs", desc, (S, Hkv, d))
    o = _check(out, "out", desc, (S, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, True)
    wp, wn = _workspace(ws)
    _raise(load().kvr_continue_append(ctypes.byref(desc), q, k, v, kc, vc, int(L_prefix), int(S), o, wp, wn,
                                      _stream(stream)), "kvr_continue_append")


def kvr_continue_batched(desc, Qs, Ks, Vs, cu_seqlens, kcache, vcache, L_prefix, out, ws=None,
                         stream=None):
    """cu_seqlens: host sequence of n+1 ints (a list or a CPU tensor).  ws: the
    workspace of workspace_for(desc, L_prefix, cu_seqlens[-1], n) (None when
    that is None: the call's plan splits no row tile over the keys)."""
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    cu = [int(x) for x in (cu_seqlens.tolist() if isinstance(cu_seqlens, torch.Tensor) else cu_seqlens)]
    n = len(cu) - 1
    if n < 0:
        raise ValueError("cu_seqlens needs at least one entry")
    total = cu[-1]
    q = _check(Qs, "Qs", desc, (total, Hq, d))
    k = _check(Ks, "Ks", desc, (total, Hkv, d))
    v = _check(Vs, "Vs", desc, (total, Hkv, d))
    o = _check(out, "out", desc, (total, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, L_prefix > 0)
    arr = (ctypes.c_int32 * len(cu))(*cu)
    wp, wn = _workspace(ws)
    _raise(load().kvr_continue_batched(ctypes.byref(desc), q, k, v, arr, n, kc, vc, int(L_prefix), o,
                                       wp, wn, _stream(stream)), "kvr_continue_batched")


def kvr_cache_append(desc, Ks, Vs, S, kcache, vcache, L_cur, stream=None):
    Hkv, d = desc.n_kv_heads, desc.head_dim
    k = _check(Ks, "Ks", desc, (S, Hkv, d))
    v = _check(Vs, "Vs", desc, (S, Hkv, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, True)
    _raise(load().kvr_cache_append(ctypes.byref(desc), k, v, int(S), kc, vc, int(L_cur), _stream(stream)),
           "kvr_cache_append")


def kvr_q8_bytes(desc):
    """Bytes of each int8 artifact tensor (kq, vq) for this descriptor."""
    nb = load().kvr_q8_bytes(ctypes.byref(desc))
    if nb == ctypes.c_size_t(-1).value:
        raise ValueError("invalid layer descriptor")
    return nb


def q8_artifact(desc, device="cuda"):
    """Allocate (with torch) an int8 artifact: (kq, vq, scales)."""
    nb = kvr_q8_bytes(desc)
    return (torch.empty(nb, dtype=torch.int8, device=device), torch.empty(nb, dtype=torch.int8, device=device),
            torch.empty(2, dtype=torch.float32, device=device))


def _check_q8(desc, kq, vq, scales):
    nb = kvr_q8_bytes(desc)
    for t, name in ((kq, "kq"), (vq, "vq")):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.int8 or not t.is_contiguous():
            raise ValueError("%s must be a contiguous int8 GPU tensor" % name)
        if t.numel() != nb:
            raise ValueError("%s holds %d bytes, the descriptor needs %d" % (name, t.numel(), nb))
    if (not isinstance(scales, torch.Tensor) or not scales.is_cuda or scales.dtype != torch.float32
            or scales.numel() != 2 or not scales.is_contiguous()):
        raise ValueError("scales must be a contiguous float32 GPU tensor of 2 values")
    return kq.data_ptr(), vq.data_ptr(), scales.data_ptr()


def kvr_quantize_cache(desc, kcache, vcache, L, kq, vq, scales, stream=None):
    kc, vc = _cache_ptrs(desc, kcache, vcache, True)
    a, b, sc = _check_q8(desc, kq, vq, scales)
    _raise(load().kvr_quantize_cache(ctypes.byref(desc), kc, vc, int(L), a, b, sc, _stream(stream)),
           "kvr_quantize_cache")


def kvr_continue_q8(desc, Qs, Ks, Vs, kq, vq, scales, L_prefix, S, out, ws=None, stream=None):
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Qs, "Qs", desc, (S, Hq, d))
    k = _check(Ks, "Ks", desc, (S, Hkv, d))
    v = _check(Vs, "Vs", desc, (S, Hkv, d))
    o = _check(out, "out", desc, (S, Hq, d))
    a, b, sc = _check_q8(desc, kq, vq, scales)
    wp, wn = _workspace(ws)
    _raise(load().kvr_continue_q8(ctypes.byref(desc), q, k, v, a, b, sc, int(L_prefix), int(S), o, wp, wn,
                                  _stream(stream)), "kvr_continue_q8")


def kvr_artifact_bytes(desc, n_layers, L):
    nb = load().kvr_artifact_bytes(ctypes.byref(desc), int(n_layers), int(L))
    if nb == ctypes.c_size_t(-1).value:
        raise ValueError("invalid descriptor, layer count or length")
    return nb


def _host_buffer(host, name):
    if not isinstance(host, torch.Tensor) or host.is_cuda or host.dtype != torch.uint8 or not host.is_contiguous():
        raise ValueError("%s must be a contiguous uint8 CPU tensor (pinned for asynchronous copies)" % name)
    return host.data_ptr(), host.numel()


def _layer_ptrs(desc, caches, name):
    arr = (ctypes.c_void_p * len(caches))()
    shape = (desc.n_kv_heads, desc.capacity, desc.head_dim)
    for i, c in enumerate(caches):
        arr[i] = _check(c, "%s[%d]" % (name, i), desc, shape)
    return arr


def kvr_artifact_save(desc, model_id, kcaches, vcaches, L, host, stream=None):
    """Serialize rows [0, L) of every layer's caches into the host tensor (Alg. 1)."""
    if len(kcaches) != len(vcaches) or not kcaches:
        raise ValueError("one K and one V cache per layer")
    hp, hn = _host_buffer(host, "host")
    _raise(load().kvr_artifact_save(ctypes.byref(desc), model_id.encode(), len(kcaches), int(L),
                                    _layer_ptrs(desc, kcaches, "kcaches"), _layer_ptrs(desc, vcaches, "vcaches"),
                                    hp, hn, _stream(stream)), "kvr_artifact_save")


def kvr_artifact_load(desc, model_id, host, kcaches, vcaches, stream=None):
    """Check the artifact's metadata against (model_id, desc, layer count) and load it
    into the caches (Alg. 2); returns L, where the continuation starts."""
    if len(kcaches) != len(vcaches) or not kcaches:
        raise ValueError("one K and one V cache per layer")
    hp, hn = _host_buffer(host, "host")
    L = ctypes.c_int64(-1)
    _raise(load().kvr_artifact_load(ctypes.byref(desc), model_id.encode(), len(kcaches), hp, hn,
                                    _layer_ptrs(desc, kcaches, "kcaches"), _layer_ptrs(desc, vcaches, "vcaches"),
                                    ctypes.byref(L), _stream(stream)), "kvr_artifact_load")
    return L.value


def _workspace(ws):
    if ws is None:
        return None, 0
    if not isinstance(ws, torch.Tensor) or not ws.is_cuda or not ws.is_contiguous():
        raise ValueError("ws must be a contiguous GPU tensor")
    return ws.data_ptr(), ws.numel() * ws.element_size()


def workspace_for(desc, L_prefix, total_S, n=1, device="cuda"):
    """Allocate (with torch) the workspace a continuation needs, or None."""
    nb = kvr_workspace_bytes(desc, L_prefix, total_S, n)
    if nb == ctypes.c_size_t(-1).value:
        raise ValueError("invalid layer descriptor")
    if nb == 0:
        return None
    return torch.empty(nb, dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- RoPE
QWEN3_ROPE_BASE = 1.0e6


class RopeTable:
    """A device cos/sin table (float [n_pos][head_dim/2][2], torch-allocated)
    filled by kvr_rope_table; pass it to the *_rope entry points."""

    def __init__(self, head_dim, n_pos, base=QWEN3_ROPE_BASE, device="cuda", stream=None):
        self.head_dim, self.n_pos, self.base = int(head_dim), int(n_pos), float(base)
        self.cos_sin = torch.empty((max(self.n_pos, 1), self.head_dim // 2, 2), dtype=torch.float32, device=device)
        kvr_rope_table(self.head_dim, self.base, self.n_pos, self.cos_sin, stream)

    def c(self):
        return kvr_rope(self.cos_sin.data_ptr(), self.n_pos)


def kvr_rope_table(head_dim, base, n_pos, cos_sin, stream=None):
    if (not isinstance(cos_sin, torch.Tensor) or not cos_sin.is_cuda or cos_sin.dtype != torch.float32
            or not cos_sin.is_contiguous() or cos_sin.numel() < int(n_pos) * int(head_dim)):
        raise ValueError("cos_sin must be a contiguous float32 GPU tensor of n_pos * head_dim values")
    _raise(load().kvr_rope_table(int(head_dim), float(base), int(n_pos), cos_sin.data_ptr(), _stream(stream)),
           "kvr_rope_table")


def _rope(rope, desc):
    if not isinstance(rope, RopeTable):
        raise ValueError("rope must be a RopeTable")
    if rope.head_dim != desc.head_dim:
        raise ValueError("RoPE table head_dim %d, descriptor %d" % (rope.head_dim, desc.head_dim))
    return ctypes.byref(rope.c())


def kvr_rope_apply(desc, rope, x, pos0, y=None, stream=None):
    """Rotate rows x [n_tok, n_heads, head_dim] at positions pos0.. into y (default: in place)."""
    if x.dim() != 3:
        raise ValueError("x must be [n_tok, n_heads, head_dim]")
    n_tok, n_heads = x.shape[0], x.shape[1]
    y = x if y is None else y
    xp = _check(x, "x", desc, (n_tok, n_heads, desc.head_dim))
    yp = _check(y, "y", desc, (n_tok, n_heads, desc.head_dim))
    _raise(load().kvr_rope_apply(ctypes.byref(desc), _rope(rope, desc), xp, int(n_tok), int(n_heads), int(pos0),
                                 yp, _stream(stream)), "kvr_rope_apply")
    return y


def kvr_prefill_rope(desc, rope, Q, K, V, L, out, kcache, vcache, stream=None):
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Q, "Q", desc, (L, Hq, d))
    k = _check(K, "K", desc, (L, Hkv, d))
    v = _check(V, "V", desc, (L, Hkv, d))
    o = _check(out, "out", desc, (L, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, True)
    _raise(load().kvr_prefill_rope(ctypes.byref(desc), _rope(rope, desc), q, k, v, int(L), o, kc, vc,
                                   _stream(stream)), "kvr_prefill_rope")


def kvr_workspace_bytes_rope(desc, L_prefix, total_S, n=1):
    return load().kvr_workspace_bytes_rope(ctypes.byref(desc), int(L_prefix), int(total_S), int(n))


def workspace_for_rope(desc, L_prefix, total_S, n=1, device="cuda"):
    """Allocate (with torch) the workspace of a RoPE continuation."""
    nb = kvr_workspace_bytes_rope(desc, L_prefix, total_S, n)
    if nb == ctypes.c_size_t(-1).value:
        raise ValueError("invalid layer descriptor")
    return torch.empty(max(nb, 1), dtype=torch.uint8, device=device)


def kvr_continue_rope(desc, rope, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out, ws, append=False, stream=None):
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    q = _check(Qs, "Qs", desc, (S, Hq, d))
    k = _check(Ks, "Ks", desc, (S, Hkv, d))
    v = _check(Vs, "Vs", desc, (S, Hkv, d))
    o = _check(out, "out", desc, (S, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, L_prefix > 0 or append)
    wp, wn = _workspace(ws)
    _raise(load().kvr_continue_rope(ctypes.byref(desc), _rope(rope, desc), q, k, v, kc, vc, int(L_prefix), int(S),
                                    1 if append else 0, o, wp, wn, _stream(stream)), "kvr_continue_rope")


def kvr_continue_batched_rope(desc, rope, Qs, Ks, Vs, cu_seqlens, kcache, vcache, L_prefix, out, ws,
                              stream=None):
    Hq, Hkv, d = desc.n_q_heads, desc.n_kv_heads, desc.head_dim
    cu = [int(x) for x in (cu_seqlens.tolist() if isinstance(cu_seqlens, torch.Tensor) else cu_seqlens)]
    n = len(cu) - 1
    if n < 0:
        raise ValueError("cu_seqlens needs at least one entry")
    total = cu[-1]
    q = _check(Qs, "Qs", desc, (total, Hq, d))
    k = _check(Ks, "Ks", desc, (total, Hkv, d))
    v = _check(Vs, "Vs", desc, (total, Hkv, d))
    o = _check(out, "out", desc, (total, Hq, d))
    kc, vc = _cache_ptrs(desc, kcache, vcache, L_prefix > 0)
    arr = (ctypes.c_int32 * len(cu))(*cu)
    wp, wn = _workspace(ws)
    _raise(load().kvr_continue_batched_rope(ctypes.byref(desc), _rope(rope, desc), q, k, v, arr, n, kc, vc,
                                            int(L_prefix), o, wp, wn, _stream(stream)),
           "kvr_continue_batched_rope")

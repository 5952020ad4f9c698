"""Python binding of libkvr_model (include/kvr_model.h): argument marshalling
only, plus holders for random weights, caches and workspaces of a
Qwen3-4B-shaped model (torch allocates the memory; every step runs in the
libraries' kernels and hipBLASLt).
"""
import ctypes
import os

import torch

from . import kvr

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvr_model.so")
EXPORTS = ("kvr_blas_create", "kvr_blas_destroy", "kvr_linear", "kvr_rmsnorm", "kvr_layer_workspace_bytes",
           "kvr_layer_forward", "kvr_model_abi_version")
BLAS_WORKSPACE_BYTES = 32 << 20

# Qwen3-4B's published configuration
QWEN3_4B = dict(hidden=2560, intermediate=9728, n_q_heads=32, n_kv_heads=8, head_dim=128, eps=1e-6,
                layers=36, vocab=151936, base=1.0e6)


class kvr_layer_shape(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("intermediate", ctypes.c_int32), ("eps", ctypes.c_float),
                ("reserved", ctypes.c_int32)]


class kvr_layer_weights(ctypes.Structure):
    _fields_ = [(nm, ctypes.c_void_p) for nm in ("ln1", "wqkv", "q_norm", "k_norm", "wo", "ln2", "wgu", "wd")]


_lib = None


def load():
    global _lib
    if _lib is not None:
        return _lib
    kvr.load()
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libkvr_model.so is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    D = ctypes.POINTER(kvr.kvr_desc)
    S = ctypes.POINTER(kvr_layer_shape)
    lib.kvr_blas_create.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.kvr_blas_destroy.argtypes = [P]
    lib.kvr_linear.argtypes = [P, I32, P, P, I64, I32, I32, ctypes.c_float, P, P, SZ, P]
    lib.kvr_rmsnorm.argtypes = [I32, P, P, I64, I32, ctypes.c_float, P, P]
    lib.kvr_layer_workspace_bytes.argtypes = [D, S, I64, I64]
    lib.kvr_layer_workspace_bytes.restype = SZ
    lib.kvr_layer_forward.argtypes = [D, S, ctypes.POINTER(kvr_layer_weights), ctypes.POINTER(kvr.kvr_rope), P, P,
                                      I64, I64, P, P, P, SZ, P]
    for f in (lib.kvr_blas_create, lib.kvr_blas_destroy, lib.kvr_linear, lib.kvr_rmsnorm, lib.kvr_layer_forward,
              lib.kvr_model_abi_version):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def _raise(st, where):
    if st != kvr.KVR_OK:
        raise kvr.KvrError(st, where)


def _ptr(t, name, dtype, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError("%s must be a contiguous GPU tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return t.data_ptr()


def _dt(dtype):
    return {torch.bfloat16: kvr.KVR_BF16, torch.float16: kvr.KVR_F16}[dtype]


class Blas:
    """A matrix-product context (kvr_blas_create); destroyed with the object."""

    def __init__(self):
        h = ctypes.c_void_p()
        _raise(load().kvr_blas_create(ctypes.byref(h)), "kvr_blas_create")
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.kvr_blas_destroy(self.handle)
            self.handle = None


def kvr_rmsnorm(x, w, eps, y, stream=None):
    rows, n = x.shape
    dt = x.dtype
    _raise(load().kvr_rmsnorm(_dt(dt), _ptr(x, "x", dt), _ptr(w, "w", dt, (n,)), rows, n, float(eps),
                              _ptr(y, "y", dt, (rows, n)), kvr._stream(stream)), "kvr_rmsnorm")


def kvr_linear(blas, x, w, y, beta=0.0, ws=None, stream=None):
    rows, n_in = x.shape
    n_out = w.shape[0]
    dt = x.dtype
    if ws is None:
        ws = torch.empty(BLAS_WORKSPACE_BYTES, dtype=torch.uint8, device=x.device)
    _raise(load().kvr_linear(blas.handle, _dt(dt), _ptr(x, "x", dt), _ptr(w, "w", dt, (n_out, n_in)), rows, n_in,
                             n_out, float(beta), _ptr(y, "y", dt, (rows, n_out)), ws.data_ptr(),
                             ws.numel(), kvr._stream(stream)), "kvr_linear")


def layer_shape(cfg):
    return kvr_layer_shape(int(cfg["hidden"]), int(cfg["intermediate"]), float(cfg["eps"]), 0)


def random_layer(cfg, dtype, generator, device="cuda"):
    """Seeded random weights of one layer: projections ~ N(0, 1/n_in), norm
    weights 1 + N(0, 0.1^2)."""
    H, I = cfg["hidden"], cfg["intermediate"]
    Hq, Hkv, d = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"]

    def mat(o, i):
        return (torch.randn((o, i), generator=generator, device=device) / i ** 0.5).to(dtype)

    def vec(n):
        return (1 + 0.1 * torch.randn((n,), generator=generator, device=device)).to(dtype)

    return {"ln1": vec(H), "wqkv": mat((Hq + 2 * Hkv) * d, H), "q_norm": vec(d), "k_norm": vec(d),
            "wo": mat(H, Hq * d), "ln2": vec(H), "wgu": mat(2 * I, H), "wd": mat(H, I)}


def _weights_struct(W, cfg, dtype):
    H, I = cfg["hidden"], cfg["intermediate"]
    Hq, Hkv, d = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    shapes = {"ln1": (H,), "wqkv": ((Hq + 2 * Hkv) * d, H), "q_norm": (d,), "k_norm": (d,), "wo": (H, Hq * d),
              "ln2": (H,), "wgu": (2 * I, H), "wd": (H, I)}
    return kvr_layer_weights(*[_ptr(W[nm], nm, dtype, shapes[nm]) for nm, _ in kvr_layer_weights._fields_])


def kvr_layer_workspace_bytes(desc, cfg, T, L_prefix_max):
    nb = load().kvr_layer_workspace_bytes(ctypes.byref(desc), ctypes.byref(layer_shape(cfg)), int(T),
                                          int(L_prefix_max))
    if nb == ctypes.c_size_t(-1).value:
        raise ValueError("invalid layer arguments")
    return nb


def kvr_layer_forward(desc, cfg, W, rope, blas, h, T, L_prefix, kcache, vcache, ws, stream=None):
    dt = h.dtype
    kc, vc = kvr._cache_ptrs(desc, kcache, vcache, True)
    _raise(load().kvr_layer_forward(ctypes.byref(desc), ctypes.byref(layer_shape(cfg)),
                                    ctypes.byref(_weights_struct(W, cfg, dt)), kvr._rope(rope, desc), blas.handle,
                                    _ptr(h, "h", dt, (T, cfg["hidden"])), int(T), int(L_prefix), kc, vc,
                                    _ptr(ws, "ws", torch.uint8), ws.numel(), kvr._stream(stream)),
           "kvr_layer_forward")


class Model:
    """A stack of random-weight layers with resident caches: prefill(h) runs
    the stack over the context, step(h) continues it by the next tokens, and
    logits(h) applies the final norm and the (tied) output projection to the
    last row.  Token positions continue from the cache's length."""

    def __init__(self, cfg, n_layers, capacity, dtype=torch.bfloat16, seed=0, vocab=None, max_tokens=None,
                 device="cuda"):
        self.cfg, self.dtype, self.device = dict(cfg), dtype, device
        self.n_layers = n_layers
        g = torch.Generator(device=device)
        g.manual_seed(seed)
        self.layers = [random_layer(cfg, dtype, g, device) for _ in range(n_layers)]
        self.vocab = vocab if vocab is not None else cfg.get("vocab", 0)
        H = cfg["hidden"]
        self.norm = (1 + 0.1 * torch.randn((H,), generator=g, device=device)).to(dtype)
        self.embed = (torch.randn((self.vocab, H), generator=g, device=device) / H ** 0.5).to(dtype) \
            if self.vocab else None
        self.desc = kvr.make_desc(cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"], dtype, capacity)
        shape = (cfg["n_kv_heads"], capacity, cfg["head_dim"])
        self.caches = [(torch.zeros(shape, dtype=dtype, device=device), torch.zeros(shape, dtype=dtype, device=device))
                       for _ in range(n_layers)]
        self.rope = kvr.RopeTable(cfg["head_dim"], capacity, cfg["base"], device=device)
        self.blas = Blas()
        self.max_tokens = max_tokens or capacity
        self.ws = torch.empty(kvr_layer_workspace_bytes(self.desc, cfg, self.max_tokens, capacity),
                              dtype=torch.uint8, device=device)
        self.xn = torch.empty((1, H), dtype=dtype, device=device)
        self.logit_buf = torch.empty((1, self.vocab), dtype=dtype, device=device) if self.vocab else None
        self.length = 0

    def forward(self, h, L_prefix):
        """Run the stack over h [T, hidden] (in place) at positions L_prefix.."""
        T = h.shape[0]
        if T > self.max_tokens:
            raise ValueError("more tokens than the workspace was sized for")
        for W, (kc, vc) in zip(self.layers, self.caches):
            kvr_layer_forward(self.desc, self.cfg, W, self.rope, self.blas, h, T, L_prefix, kc, vc, self.ws)
        return h

    def logits(self, h):
        """Final norm of the last row, then its logits against the tied embedding."""
        kvr_rmsnorm(h[-1:].contiguous() if h.shape[0] > 1 else h, self.norm, self.cfg["eps"], self.xn)
        kvr_linear(self.blas, self.xn, self.embed, self.logit_buf, ws=self.ws[-BLAS_WORKSPACE_BYTES:])
        return self.logit_buf

    def prefill(self, h):
        self.forward(h, 0)
        self.length = h.shape[0]
        return h

    def step(self, h):
        self.forward(h, self.length)
        self.length += h.shape[0]
        return h

"""Python front end of the fp64 CPU oracle (``kvr_ref.c``).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this module.  The GPU product path
never imports it and must not fall back to it.

Inputs are converted to fp64 exactly (bf16 and fp32 widen without rounding),
so the oracle sees the very values the GPU received.  Every function follows
the paper's method as restated in ``kvr_ref.c``:

* :func:`prefill`   -- Alg. 1's forward pass, attention part (causal, L tokens).
* :func:`continue_` -- Alg. 2's forward call over a cached prefix: positions
  L_prefix.., mask spanning the whole prefix plus the new tokens.
* :func:`cache_append` -- the cache update of Alg. 2 (exact copy).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvr_ref.c")
_LIB = os.path.join(_HERE, "libkvr_ref.so")
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I64P = ctypes.POINTER(ctypes.c_int64)


def build(force=False):
    """Compile the oracle with gcc (-O2, fp64, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        lib.kvr_ref_prefill.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                        _D, _D, _D, ctypes.c_int64, _I64P, ctypes.c_int64,
                                        _D, _D, ctypes.c_int]
        lib.kvr_ref_continue.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                         _D, _D, _D, ctypes.c_int64,
                                         _D, _D, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                         _I64P, ctypes.c_int64, _D, _D, ctypes.c_int]
        lib.kvr_ref_cache_append.argtypes = [ctypes.c_int, ctypes.c_int, _D, _D, ctypes.c_int64,
                                             _D, _D, ctypes.c_int64, ctypes.c_int64]
        for f in (lib.kvr_ref_prefill, lib.kvr_ref_continue, lib.kvr_ref_cache_append):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(a):
    """Any torch tensor / numpy array -> C-contiguous fp64 numpy array (exact widening)."""
    if hasattr(a, "detach"):
        a = a.detach().to("cpu")
        import torch
        a = a.to(torch.float64).numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return a.ctypes.data_as(_D)


def _rows(rows, n_all):
    if rows is None:
        return None, n_all, None
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    if r.size and (r.min() < 0 or r.max() >= n_all):
        raise ValueError("row index out of range")
    return r, int(r.size), r.ctypes.data_as(_I64P)


def default_threads():
    return max(1, os.cpu_count() or 1)


def prefill(Q, K, V, scale=None, rows=None, nthreads=None):
    """Causal prefill attention.  Q [L,Hq,d], K/V [L,Hkv,d] -> (out [n,Hq,d], lse [n,Hq])."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    L, Hq, D = Q.shape
    Hkv = K.shape[1]
    if K.shape != (L, Hkv, D) or V.shape != K.shape:
        raise ValueError("shape mismatch")
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    r, n, rp = _rows(rows, L)
    out = np.zeros((n, Hq, D))
    lse = np.zeros((n, Hq))
    rc = _load().kvr_ref_prefill(Hq, Hkv, D, float(scale), _ptr(Q), _ptr(K), _ptr(V), L,
                                 rp, n, _ptr(out), _ptr(lse), nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle rejected the arguments (%d)" % rc)
    return out, lse


def continue_(Qs, Ks, Vs, kcache, vcache, L_prefix, scale=None, rows=None, k_range=None,
              nthreads=None):
    """Continuation over cached rows [0, L_prefix) of kcache/vcache [Hkv,cap,d].

    Qs [S,Hq,d] sit at positions L_prefix..L_prefix+S-1; Ks/Vs [S,Hkv,d] are
    their own keys.  ``k_range=(lo, hi)`` restricts the key sequence.
    """
    Qs, Ks, Vs = _f64(Qs), _f64(Ks), _f64(Vs)
    kc, vc = _f64(kcache), _f64(vcache)
    S, Hq, D = Qs.shape
    Hkv, cap, _ = kc.shape
    if Ks.shape != (S, Hkv, D) or Vs.shape != Ks.shape or vc.shape != kc.shape:
        raise ValueError("shape mismatch")
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    lo, hi = (0, L_prefix + S) if k_range is None else k_range
    r, n, rp = _rows(rows, S)
    out = np.zeros((n, Hq, D))
    lse = np.zeros((n, Hq))
    rc = _load().kvr_ref_continue(Hq, Hkv, D, float(scale), _ptr(Qs), _ptr(Ks), _ptr(Vs), S,
                                  _ptr(kc), _ptr(vc), cap, int(L_prefix), int(lo), int(hi),
                                  rp, n, _ptr(out), _ptr(lse), nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle rejected the arguments (%d)" % rc)
    return out, lse


def cache_append(kcache, vcache, Ks, Vs, L_cur):
    """Return copies of the caches with rows [L_cur, L_cur+S) replaced by Ks/Vs (fp64)."""
    kc, vc = _f64(kcache).copy(), _f64(vcache).copy()
    Ks, Vs = _f64(Ks), _f64(Vs)
    Hkv, cap, D = kc.shape
    S = Ks.shape[0]
    rc = _load().kvr_ref_cache_append(Hkv, D, _ptr(Ks), _ptr(Vs), S, _ptr(kc), _ptr(vc), cap,
                                      int(L_cur))
    if rc != 0:
        raise ValueError("oracle rejected the arguments (%d)" % rc)
    return kc, vc

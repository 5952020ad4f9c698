"""Oracle of the quantized KV artifact (the paper's Section "Quantizing the
artifact: size vs. exactness": the context KV stored at per-tensor symmetric
int8, halving its size at the cost of token-exactness).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this module.  The GPU product path
never imports it and must not fall back to it.

The paper names the scheme (per-tensor, symmetric, int8) and nothing more.
The reading used here:

* one scale per tensor: s = max|x| / 127 over every element of the tensor (all
  kv heads, cached rows [0, L)); s = 1 for an all-zero tensor;
* code q = clamp(round-half-even(x / s), -127, 127);
* dequantized value q * s.

The codes are integers decided by floating point, so they are computed in the
precision the GPU uses: the scale and the quotient x / s in IEEE fp32
(correctly rounded division), the rounding to an integer exact.  The attention
over the dequantized cache is the plain fp64 oracle of ``ref.continue_``.
"""
import numpy as np

from oracle import ref

QMAX = 127


def _f32(a):
    if hasattr(a, "detach"):
        import torch
        a = a.detach().to("cpu").to(torch.float32).numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def scale_of(x):
    """Per-tensor symmetric scale, fp32: max|x| / 127, or 1 for an all-zero tensor."""
    a = _f32(x)
    m = np.float32(np.max(np.abs(a))) if a.size else np.float32(0.0)
    if m == 0:
        return np.float32(1.0)
    return np.float32(m / np.float32(QMAX))


def quantize(x):
    """(codes int8 same shape, scale fp32) of one tensor."""
    a = _f32(x)
    s = scale_of(a)
    q = np.rint(a / s)                     # fp32 quotient, round half to even
    q = np.clip(q, -QMAX, QMAX)
    return q.astype(np.int8), s


def dequantize(codes, s):
    """codes * s in fp64 (exact: an int8 times an fp32 fits in fp64)."""
    return np.asarray(codes, dtype=np.float64) * np.float64(s)


def quantize_cache(kcache, vcache, L):
    """Quantize rows [0, L) of a [Hkv, cap, d] cache pair; K and V each have one scale."""
    kc = _f32(kcache)[:, :L, :]
    vc = _f32(vcache)[:, :L, :]
    kq, sk = quantize(kc)
    vq, sv = quantize(vc)
    return kq, vq, sk, sv


def continue_q8(Qs, Ks, Vs, kq, vq, sk, sv, L_prefix, scale=None, rows=None, nthreads=None):
    """Continuation over the dequantized cached rows [0, L_prefix) of the artifact
    (codes [Hkv, L, d]); the new tokens' own keys and values are not quantized."""
    kd = dequantize(kq, sk)
    vd = dequantize(vq, sv)
    return ref.continue_(Qs, Ks, Vs, kd, vd, L_prefix, scale=scale, rows=rows, nthreads=nthreads)

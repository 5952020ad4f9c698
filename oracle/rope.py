"""Oracle of rotary position embedding with a position offset (the paper's
Section "Consuming an artifact": the continuation's tokens take position ids
L, L+1, ... so that positional encodings such as RoPE agree with a pass from
scratch; Alg. 2 derives those positions from the artifact's length).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this module.  The GPU product path
never imports it and must not fall back to it.

The paper names RoPE as the positional encoding of its models and gives no
formula.  The reading used here is rotary embedding as defined by Su et al.
(RoFormer), in the half-split pairing of the Qwen family the paper evaluates:

* head dimension d, pair i in [0, d/2) is (x[i], x[i + d/2]);
* frequency theta_i = base ** (-2 i / d);
* at position p the pair turns by the angle p * theta_i:
      y[i]       = x[i] cos(p theta_i) - x[i + d/2] sin(p theta_i)
      y[i + d/2] = x[i + d/2] cos(p theta_i) + x[i] sin(p theta_i)

Queries and keys are rotated, values are not; the cache holds rotated keys.
The rotation is fp64 on the exact (widened) input values.  A model holds the
rotated rows in its own element format: the rotated keys are what its cache
stores, and the rotated queries are the operands of its score product.  So
with ``fmt`` given (bf16, fp16 or fp32) the rotated rows are rounded once to
that format, round to nearest with ties to even (:func:`round_to`), before the
fp64 attention of ``ref``.
"""
import numpy as np

from oracle import ref

QWEN3_BASE = 1.0e6   # rope base of the Qwen3 models


# significand bits (with the leading one) and the smallest normal exponent of
# the element formats
_FORMATS = {"bf16": (8, -126), "fp16": (11, -14), "fp32": (24, -126)}


def _fmt_name(fmt):
    if fmt is None or isinstance(fmt, str):
        return fmt
    import torch
    return {torch.bfloat16: "bf16", torch.float16: "fp16", torch.float32: "fp32"}[fmt]


def round_to(x, fmt):
    """Round fp64 values to the nearest value of the format, ties to even.

    A value is written m * 2^e with m in [0.5, 1); with p significand bits its
    quantum is 2^(e - p), or the subnormal quantum 2^(emin - p + 1) below the
    normal range.  Overflow does not occur for the magnitudes used here.
    """
    name = _fmt_name(fmt)
    if name is None:
        return np.asarray(x, dtype=np.float64)
    p, emin = _FORMATS[name]
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.ldexp(1.0, np.maximum(e, emin + 1) - p)          # quantum of each value
    return np.rint(x / q) * q


def thetas(d, base):
    """theta_i = base ** (-2 i / d), i in [0, d/2)."""
    if d % 2:
        raise ValueError("head_dim must be even")
    i = np.arange(d // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * i / d)


def table(d, base, n_pos):
    """cos and sin of p * theta_i: array [n_pos, d/2, 2] (cos, sin), fp64."""
    ang = np.arange(n_pos, dtype=np.float64)[:, None] * thetas(d, base)[None, :]
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1)


def rotate(x, positions, base):
    """Rotate rows x [T, H, d] (any float type, widened exactly) at positions [T]."""
    x = ref._f64(x)
    T, H, d = x.shape
    pos = np.asarray(positions, dtype=np.float64).reshape(T)
    ang = pos[:, None] * thetas(d, base)[None, :]          # [T, d/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    lo, hi = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def prefill(Q, K, V, base, scale=None, rows=None, nthreads=None, fmt=None):
    """Prefill with RoPE at positions 0..L-1.

    Returns (out, lse, k_rot): k_rot [L, Hkv, d] are the rotated keys the
    cache holds (rounded to ``fmt`` when given).
    """
    L = Q.shape[0]
    pos = np.arange(L)
    qr, kr = round_to(rotate(Q, pos, base), fmt), round_to(rotate(K, pos, base), fmt)
    out, lse = ref.prefill(qr, kr, V, scale=scale, rows=rows, nthreads=nthreads)
    return out, lse, kr


def continue_(Qs, Ks, Vs, kcache, vcache, L_prefix, base, scale=None, rows=None, nthreads=None,
              pos0=None, fmt=None):
    """Continuation with RoPE: Qs/Ks rotated at positions pos0..pos0+S-1 (pos0 =
    L_prefix, Alg. 2) over the cached, already rotated keys of kcache.

    ``pos0`` other than L_prefix reproduces the paper's shifted failure mode.
    Returns (out, lse, k_rot) with k_rot the rotated new keys (rounded to
    ``fmt`` when given).
    """
    S = Qs.shape[0]
    p0 = L_prefix if pos0 is None else pos0
    pos = p0 + np.arange(S)
    qr, kr = round_to(rotate(Qs, pos, base), fmt), round_to(rotate(Ks, pos, base), fmt)
    out, lse = ref.continue_(qr, kr, Vs, kcache, vcache, L_prefix, scale=scale, rows=rows,
                             nthreads=nthreads)
    return out, lse, kr

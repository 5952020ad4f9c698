"""Oracle of a Qwen3-style decoder layer around the attention (the model whose
prefill and continuation costs the paper compares in Table 1: Qwen3-4B, 36
layers, 8 KV heads of width 128).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this module.  The GPU product path
never imports it and must not fall back to it.

The paper gives the model's name, layer count and KV geometry, not its
layer.  The reading used here is the published Qwen3 decoder layer (pre-norm,
residual):

    x  = rmsnorm(h) * ln1
    q, k, v = x Wq^T, x Wk^T, x Wv^T          (one fused weight, rows q | k | v)
    q_h = rope(rmsnorm(q_h) * q_norm), k_h = rope(rmsnorm(k_h) * k_norm)   per head
    h  = h + attention(q, k, v) Wo^T           (causal GQA over the cache + own rows)
    x  = rmsnorm(h) * ln2
    h  = h + (silu(x Wg^T) * (x Wu^T)) Wd^T    (fused weight, rows gate | up)

with rmsnorm(x) = x / sqrt(mean(x^2) + eps) and silu(x) = x / (1 + e^-x).
Token t of a call sits at position L_prefix + t (Alg. 2's positions from the
artifact's length); the cache receives the rotated keys and the values.

Arithmetic is fp64.  With ``fmt`` given, every tensor the model holds between
operations is rounded once to the element format, as a model running in that
format holds it: the normalized rows, the projections, the rotated q/k rows,
the attention output, the residual stream after each add, the gate/up
products and the activation.
"""
import numpy as np

from oracle import ref
from oracle import rope

# Qwen3-4B's published configuration (head geometry as the paper states it)
QWEN3_4B = dict(hidden=2560, intermediate=9728, n_q_heads=32, n_kv_heads=8, head_dim=128,
                eps=1e-6, layers=36, vocab=151936, base=1.0e6)


def rmsnorm(x, w, eps):
    """x / sqrt(mean(x^2) + eps) * w over the last axis (fp64)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(w, dtype=np.float64)


def silu(x):
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def _f64(a):
    return ref._f64(a)


def layer(h, W, shape, kcache, vcache, L_prefix, fmt=None):
    """One decoder layer over T tokens at positions L_prefix..L_prefix+T-1.

    h [T, hidden]; W: dict of ln1, wqkv [(Hq+2Hkv) d, hidden], q_norm [d],
    k_norm [d], wo [hidden, Hq d], ln2, wgu [2 inter, hidden], wd [hidden, inter];
    kcache/vcache [Hkv, cap, d] hold rows [0, L_prefix) (rotated keys).
    Returns (h_out [T, hidden], k_rows [T, Hkv, d], v_rows [T, Hkv, d]): the
    new cache rows the layer writes at L_prefix.. .
    """
    r = lambda x: rope.round_to(x, fmt)        # noqa: E731
    Hq, Hkv, d = shape["n_q_heads"], shape["n_kv_heads"], shape["head_dim"]
    eps = shape["eps"]
    h = _f64(h)
    T = h.shape[0]
    Wd = {k: _f64(v) for k, v in W.items()}
    x = r(rmsnorm(h, Wd["ln1"], eps))
    qkv = r(x @ Wd["wqkv"].T)
    q = qkv[:, : Hq * d].reshape(T, Hq, d)
    k = qkv[:, Hq * d: (Hq + Hkv) * d].reshape(T, Hkv, d)
    v = qkv[:, (Hq + Hkv) * d:].reshape(T, Hkv, d)
    pos = L_prefix + np.arange(T)
    q = r(rope.rotate(rmsnorm(q, Wd["q_norm"], eps), pos, shape["base"]))
    k = r(rope.rotate(rmsnorm(k, Wd["k_norm"], eps), pos, shape["base"]))
    if L_prefix == 0:
        att, _ = ref.prefill(q, k, v)
    else:
        att, _ = ref.continue_(q, k, v, kcache, vcache, L_prefix)
    att = r(att).reshape(T, Hq * d)
    h = r(h + att @ Wd["wo"].T)
    x = r(rmsnorm(h, Wd["ln2"], eps))
    gu = r(x @ Wd["wgu"].T)
    inter = gu.shape[1] // 2
    act = r(silu(gu[:, :inter]) * gu[:, inter:])
    h = r(h + act @ Wd["wd"].T)
    return h, k, v


def model(h, layers_W, shape, L_prefix=0, caches=None, fmt=None):
    """The layer stack over T tokens at positions L_prefix..; caches is a list of
    (kcache, vcache) per layer holding rows [0, L_prefix) (fp64, [Hkv, cap, d]),
    extended in place with the new rows.  Returns the final residual stream."""
    Hkv, d = shape["n_kv_heads"], shape["head_dim"]
    T = _f64(h).shape[0]
    if caches is None:
        caches = [(np.zeros((Hkv, T, d)), np.zeros((Hkv, T, d))) for _ in layers_W]
    for W, (kc, vc) in zip(layers_W, caches):
        h, k, v = layer(h, W, shape, kc, vc, L_prefix, fmt)
        kc[:, L_prefix:L_prefix + T] = np.transpose(k, (1, 0, 2))
        vc[:, L_prefix:L_prefix + T] = np.transpose(v, (1, 0, 2))
    return h


def logits(h_last, norm_w, w_lm, eps, fmt=None):
    """Next-token logits of the last row: rmsnorm(h) * norm_w, times w_lm^T [vocab, hidden]."""
    r = lambda x: rope.round_to(x, fmt)        # noqa: E731
    x = r(rmsnorm(_f64(h_last), _f64(norm_w), eps))
    return r(x @ _f64(w_lm).T)

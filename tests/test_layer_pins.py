"""Pins of the decoder-layer oracle (``oracle/layer.py``) against facts fixed
outside it.

* RMSNorm and SiLU against hand closed forms and an identity
  (silu(x) - silu(-x) = x);
* the residual structure: with zero output projections the layer is the
  identity on the residual stream, and the cache still receives the rotated,
  normalized keys;
* attention inside the layer: with zero query and key weights every score is
  0, so the attention output is the running mean of the value rows (written
  with a cumulative sum) and the layer's output is h + mean(V) Wo^T;
* the paper's Claim 1 for the whole stack: a continuation of the last tokens
  over the cached layers equals the matching rows of one prefill, exactly in
  fp64 and also with every activation rounded to bf16 (each row's arithmetic
  is the same in both); restarting the continuation's positions at 0 breaks it.
"""
import numpy as np
import pytest

from oracle import layer as LO
from oracle import ref
from oracle import rope

SH = dict(hidden=64, intermediate=96, n_q_heads=4, n_kv_heads=2, head_dim=16, eps=1e-6, base=1e4)


def weights(seed, sh=SH, zero=()):
    g = np.random.default_rng(seed)
    H, I, Hq, Hkv, d = sh["hidden"], sh["intermediate"], sh["n_q_heads"], sh["n_kv_heads"], sh["head_dim"]
    W = {
        "ln1": 1 + 0.1 * g.standard_normal(H), "ln2": 1 + 0.1 * g.standard_normal(H),
        "q_norm": 1 + 0.1 * g.standard_normal(d), "k_norm": 1 + 0.1 * g.standard_normal(d),
        "wqkv": g.standard_normal(((Hq + 2 * Hkv) * d, H)) / np.sqrt(H),
        "wo": g.standard_normal((H, Hq * d)) / np.sqrt(Hq * d),
        "wgu": g.standard_normal((2 * I, H)) / np.sqrt(H),
        "wd": g.standard_normal((H, I)) / np.sqrt(I),
    }
    for z in zero:
        if z == "wqk":
            W["wqkv"][: (Hq + Hkv) * d] = 0.0
        else:
            W[z] = np.zeros_like(W[z])
    return W


def test_rmsnorm_closed_form():
    y = LO.rmsnorm(np.array([[3.0, 4.0]]), np.array([1.0, 2.0]), 0.0)
    r = np.sqrt(12.5)
    np.testing.assert_allclose(y, [[3 / r, 8 / r]], rtol=1e-15)
    np.testing.assert_array_equal(LO.rmsnorm(np.zeros((1, 5)), np.ones(5), 1e-6), np.zeros((1, 5)))
    c = LO.rmsnorm(np.full((1, 8), -2.5), np.arange(8.0), 0.0)          # constant row -> -w
    np.testing.assert_allclose(c, [-np.arange(8.0)], rtol=1e-15)
    e = LO.rmsnorm(np.array([[1.0, 1.0]]), np.ones(2), 3.0)             # eps inside the root
    np.testing.assert_allclose(e, [[0.5, 0.5]], rtol=1e-15)


def test_silu_closed_form():
    assert LO.silu(0.0) == 0.0
    np.testing.assert_allclose(LO.silu(np.log(3.0)), np.log(3.0) * 0.75, rtol=1e-15)   # sigma(ln 3) = 3/4
    x = np.linspace(-20, 20, 81)
    np.testing.assert_allclose(LO.silu(x) - LO.silu(-x), x, atol=1e-13)
    assert abs(LO.silu(40.0) - 40.0) < 1e-12 and abs(LO.silu(-40.0)) < 1e-15


def test_zero_projections_are_the_identity():
    W = weights(1, zero=("wo", "wd"))
    g = np.random.default_rng(2)
    h = g.standard_normal((7, SH["hidden"]))
    out, k, v = LO.layer(h, W, SH, None, None, 0)
    np.testing.assert_array_equal(out, h)
    # the cache rows: rotated, normalized keys and the raw values
    x = LO.rmsnorm(h, W["ln1"], SH["eps"])
    Hq, Hkv, d = SH["n_q_heads"], SH["n_kv_heads"], SH["head_dim"]
    kk = (x @ W["wqkv"][Hq * d:(Hq + Hkv) * d].T).reshape(7, Hkv, d)
    want_k = rope.rotate(LO.rmsnorm(kk, W["k_norm"], SH["eps"]), np.arange(7), SH["base"])
    np.testing.assert_allclose(k, want_k, atol=1e-13)
    np.testing.assert_allclose(v, (x @ W["wqkv"][(Hq + Hkv) * d:].T).reshape(7, Hkv, d), atol=1e-13)


def test_zero_scores_give_the_running_mean():
    W = weights(3, zero=("wqk", "wd"))
    g = np.random.default_rng(4)
    T = 9
    h = g.standard_normal((T, SH["hidden"]))
    out, _, _ = LO.layer(h, W, SH, None, None, 0)
    Hq, Hkv, d = SH["n_q_heads"], SH["n_kv_heads"], SH["head_dim"]
    x = LO.rmsnorm(h, W["ln1"], SH["eps"])
    v = (x @ W["wqkv"][(Hq + Hkv) * d:].T).reshape(T, Hkv, d)
    mean_v = np.cumsum(v, axis=0) / np.arange(1, T + 1)[:, None, None]       # causal mean per kv head
    att = np.repeat(mean_v, Hq // Hkv, axis=1).reshape(T, Hq * d)             # head h reads kv head h // G
    np.testing.assert_allclose(out, h + att @ W["wo"].T, atol=1e-12)


@pytest.mark.parametrize("fmt", [None, "bf16"])
def test_claim1_for_the_stack(fmt):
    n_layers, Lp, S = 3, 11, 5
    n = Lp + S
    Ws = [weights(10 + i) for i in range(n_layers)]
    h = np.random.default_rng(5).standard_normal((n, SH["hidden"]))
    if fmt:
        h = rope.round_to(h, fmt)
    full = LO.model(h, Ws, SH, fmt=fmt)
    Hkv, d = SH["n_kv_heads"], SH["head_dim"]
    caches = [(np.zeros((Hkv, n, d)), np.zeros((Hkv, n, d))) for _ in Ws]
    LO.model(h[:Lp], Ws, SH, 0, caches, fmt)
    cont = LO.model(h[Lp:], Ws, SH, Lp, caches, fmt)
    if fmt:
        np.testing.assert_array_equal(cont, full[Lp:])
    else:
        np.testing.assert_allclose(cont, full[Lp:], rtol=0, atol=1e-12)
    # the shifted failure: the same continuation with its rows rotated at
    # positions 0.. while the mask still spans the cache (fp64, fmt ignored)
    caches2 = [(np.zeros((Hkv, n, d)), np.zeros((Hkv, n, d))) for _ in Ws]
    LO.model(h[:Lp], Ws, SH, 0, caches2)
    Hq, eps, base = SH["n_q_heads"], SH["eps"], SH["base"]
    h2 = h[Lp:]
    for W, (kc, vc) in zip(Ws, caches2):
        x = LO.rmsnorm(h2, W["ln1"], eps)
        qkv = x @ W["wqkv"].T
        q = rope.rotate(LO.rmsnorm(qkv[:, :Hq * d].reshape(S, Hq, d), W["q_norm"], eps), np.arange(S), base)
        k = rope.rotate(LO.rmsnorm(qkv[:, Hq * d:(Hq + Hkv) * d].reshape(S, Hkv, d), W["k_norm"], eps),
                        np.arange(S), base)
        v = qkv[:, (Hq + Hkv) * d:].reshape(S, Hkv, d)
        att, _ = ref.continue_(q, k, v, kc, vc, Lp)
        h2 = h2 + att.reshape(S, Hq * d) @ W["wo"].T
        x = LO.rmsnorm(h2, W["ln2"], eps)
        gu = x @ W["wgu"].T
        inter = gu.shape[1] // 2
        h2 = h2 + (LO.silu(gu[:, :inter]) * gu[:, inter:]) @ W["wd"].T
    assert np.max(np.abs(h2 - full[Lp:])) > 1e-2


def test_logits_tied_head():
    g = np.random.default_rng(6)
    E = g.standard_normal((50, SH["hidden"]))
    h = g.standard_normal(SH["hidden"])
    w = 1 + 0.1 * g.standard_normal(SH["hidden"])
    lg = LO.logits(h, w, E, 1e-6)
    x = h / np.sqrt(np.mean(h * h) + 1e-6) * w
    np.testing.assert_allclose(lg, [float(np.dot(x, E[i])) for i in range(50)], rtol=1e-12)


def _mlp_only(seed, gate_sign):
    """A layer whose attention adds nothing (zero output projection) and whose
    MLP input is positive: h > 0 and ln2 > 0 give x = rmsnorm(h) * ln2 > 0, so
    gate rows with entries of one sign make every gate value x.Wg of that sign
    and far from 0."""
    W = weights(seed, zero=("wo",))
    g = np.random.default_rng(seed + 100)
    H, I = SH["hidden"], SH["intermediate"]
    W["ln2"] = 0.5 + g.random(H)                                  # positive, not 1
    W["wgu"][:I] = gate_sign * (2.0 + g.random((I, H)))           # gate rows: |x.Wg| >> 1
    h = 0.2 + g.random((6, H))
    return W, h


def test_mlp_with_open_gate_is_the_product():
    """silu(g) = g for g >> 0, so the MLP term is (x Wg^T * x Wu^T) Wd^T with
    x = rmsnorm(h) * ln2 and the fused weight's rows gate | up, written out by
    hand here.  Swapping gate and up (silu on the up half), dropping ln2, or
    adding to anything but the residual stream all fail it."""
    W, h = _mlp_only(7, +1.0)
    I = SH["intermediate"]
    out, _, _ = LO.layer(h, W, SH, None, None, 0)
    x = h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + SH["eps"]) * W["ln2"]
    gate = x @ W["wgu"][:I].T
    up = x @ W["wgu"][I:].T
    assert gate.min() > 40.0                                      # silu(gate) = gate to 1e-16
    assert (up < 0).any() and (up > 0).any()                      # up is not one-signed
    want = h + (gate * up) @ W["wd"].T
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-10)
    # the swapped reading (silu applied to the up half) is far from it
    swapped = h + (LO.silu(up) * gate) @ W["wd"].T
    assert np.max(np.abs(swapped - want)) > 1.0


def test_mlp_with_closed_gate_vanishes():
    """silu(g) = 0 for g << 0: the layer returns its input (attention adds
    nothing either), whatever the up and down weights are."""
    W, h = _mlp_only(8, -1.0)
    out, _, _ = LO.layer(h, W, SH, None, None, 0)
    np.testing.assert_allclose(out, h, rtol=0, atol=1e-12)

"""Pins of the fp64 oracle against facts fixed outside it.

Nothing here compares the oracle with itself: each test checks it against a
closed form, an invariant of the mathematics, the paper's own claim (Claim 1
and its argument), a pure-Python brute force, or numbers printed in the paper.
Each check is chosen so that a plausible slip (wrong scale, exp base, sign,
mask off by one, wrong kv-head map, transposed operand, wrong cache stride)
fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import brute, ref


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def cache_from(Kfull, Vfull, L_prefix, capacity):
    """Cache [Hkv, cap, d] holding the first L_prefix rows of K/V [n, Hkv, d]."""
    Hkv, D = Kfull.shape[1], Kfull.shape[2]
    kc = np.full((Hkv, capacity, D), np.nan)
    vc = np.full((Hkv, capacity, D), np.nan)
    return ref.cache_append(kc, vc, Kfull[:L_prefix], Vfull[:L_prefix], 0)


# ------------------------------------------------------------------ P1 brute force
TINY_SHAPES = [  # (L, Hq, Hkv, d)
    (1, 1, 1, 1), (2, 1, 1, 2), (5, 2, 1, 3), (7, 4, 2, 8), (13, 6, 3, 5),
    (23, 4, 1, 8), (40, 4, 4, 8), (17, 8, 2, 4),
]


@pytest.mark.parametrize("L,Hq,Hkv,D", TINY_SHAPES)
def test_brute_force_prefill(L, Hq, Hkv, D):
    Q, K, V = rnd((L, Hq, D), 1), rnd((L, Hkv, D), 2), rnd((L, Hkv, D), 3)
    scale = 1.0 / math.sqrt(D)
    out, lse = ref.prefill(Q, K, V, scale, nthreads=3)
    bo, bl = brute.attend(Q.tolist(), K.tolist(), V.tolist(), Hq, Hkv, scale, 0)
    assert np.max(np.abs(out - np.array(bo))) <= 1e-12
    assert np.max(np.abs(lse - np.array(bl))) <= 1e-12


@pytest.mark.parametrize("L,Hq,Hkv,D", TINY_SHAPES)
def test_brute_force_continue(L, Hq, Hkv, D):
    n = L + 5
    Q, K, V = rnd((n, Hq, D), 4), rnd((n, Hkv, D), 5), rnd((n, Hkv, D), 6)
    scale = 0.37
    kc, vc = cache_from(K, V, L, L + 9)
    out, lse = ref.continue_(Q[L:], K[L:], V[L:], kc, vc, L, scale)
    # brute force sees the plain concatenated key sequence and positions L..L+4
    bo, bl = brute.attend(Q[L:].tolist(), K.tolist(), V.tolist(), Hq, Hkv, scale, L)
    assert np.max(np.abs(out - np.array(bo))) <= 1e-12
    assert np.max(np.abs(lse - np.array(bl))) <= 1e-12


def test_brute_force_tiny_workload():
    """The 144-token fp32 workload (2 q heads, 1 kv head, d 64, seed 0)."""
    Q, K, V = W.qkv(W.TINY_L + W.TINY_S, W.TINY, seed=0)
    Qd, Kd, Vd = (x.double().numpy() for x in (Q, K, V))
    out, lse = ref.prefill(Q, K, V)
    bo, bl = brute.attend(Qd.tolist(), Kd.tolist(), Vd.tolist(), 2, 1, 1.0 / 8.0, 0)
    assert np.max(np.abs(out - np.array(bo))) <= 1e-12
    assert np.max(np.abs(lse - np.array(bl))) <= 1e-12


# ------------------------------------------------------------ closed forms
def test_two_key_closed_form():
    """d = 4, scale 1/2: scores (0, 1) give weights (1 - s, s) with s = e / (1 + e)."""
    D = 4
    Q = np.zeros((2, 1, D)); Q[:, 0, 0] = 2.0
    K = np.zeros((2, 1, D)); K[1, 0, 0] = 1.0
    V = np.zeros((2, 1, D)); V[0, 0, 0] = 1.0; V[1, 0, 1] = 1.0
    out, lse = ref.prefill(Q, K, V)                    # default scale 1/sqrt(4)
    s = math.e / (1.0 + math.e)
    assert np.allclose(out[1, 0], [1.0 - s, s, 0.0, 0.0], atol=1e-15, rtol=0)
    assert abs(lse[1, 0] - math.log(1.0 + math.e)) <= 1e-15
    assert np.array_equal(out[0, 0], V[0, 0])          # row 0 sees only key 0
    assert lse[0, 0] == 0.0


def test_three_key_negative_scores():
    """Scores (-1, 0.5, -2.5) at position 2 reproduce a hand-written softmax."""
    D = 1
    Q = np.array([[[1.0]], [[1.0]], [[1.0]]])
    K = np.array([[[-1.0]], [[0.5]], [[-2.5]]])
    V = np.array([[[3.0]], [[-1.0]], [[7.0]]])
    out, lse = ref.prefill(Q, K, V, scale=1.0)
    e = [math.exp(-1.0), math.exp(0.5), math.exp(-2.5)]
    want = (3.0 * e[0] - 1.0 * e[1] + 7.0 * e[2]) / sum(e)
    assert abs(out[2, 0, 0] - want) <= 1e-15
    assert abs(lse[2, 0] - math.log(sum(e))) <= 1e-15
    want1 = (3.0 * e[0] - 1.0 * e[1]) / (e[0] + e[1])
    assert abs(out[1, 0, 0] - want1) <= 1e-15


def test_huge_scores_no_overflow():
    """A score gap of 1000 would overflow exp without the max shift: result is V of the winner."""
    Q = np.array([[[1.0]], [[1.0]]])
    K = np.array([[[0.0]], [[1000.0]]])
    V = np.array([[[5.0]], [[-2.0]]])
    out, lse = ref.prefill(Q, K, V, scale=1.0)
    assert out[1, 0, 0] == -2.0 and lse[1, 0] == 1000.0


# ------------------------------------------------------------- P2 normalisation
def test_rows_sum_to_one():
    """V = 1 everywhere gives an output of exactly one up to rounding (weights sum to 1)."""
    L, Hq, Hkv, D = 37, 4, 2, 16
    Q, K = rnd((L, Hq, D), 7) * 3, rnd((L, Hkv, D), 8)
    out, _ = ref.prefill(Q, K, np.ones((L, Hkv, D)))
    assert np.max(np.abs(out - 1.0)) <= 1e-15


def test_convex_hull():
    """Every output component lies between the min and max of the visible values."""
    L, Hq, Hkv, D = 29, 2, 1, 8
    Q, K, V = rnd((L, Hq, D), 9), rnd((L, Hkv, D), 10), rnd((L, Hkv, D), 11)
    out, _ = ref.prefill(Q, K, V)
    for i in range(L):
        lo, hi = V[: i + 1, 0].min(axis=0), V[: i + 1, 0].max(axis=0)
        assert np.all(out[i] >= lo - 1e-15) and np.all(out[i] <= hi + 1e-15)


# ---------------------------------------------------------------- P3 single key
def test_single_key_returns_value():
    L, Hq, Hkv, D = 9, 4, 2, 8
    Q, K, V = rnd((L, Hq, D), 12), rnd((L, Hkv, D), 13), rnd((L, Hkv, D), 14)
    out, lse = ref.prefill(Q, K, V)
    for h in range(Hq):
        assert np.array_equal(out[0, h], V[0, h // 2])
    out1, _ = ref.prefill(Q[:1], K[:1], V[:1])
    assert np.array_equal(out1[0], V[0][[0, 0, 1, 1]])


# ---------------------------------------------------------- P4 equal scores
def test_equal_scores_give_running_mean():
    """Q = 0 makes every visible score equal: the output is the causal running mean of V."""
    L, Hq, Hkv, D = 31, 6, 3, 5
    K, V = rnd((L, Hkv, D), 15), rnd((L, Hkv, D), 16)
    out, lse = ref.prefill(np.zeros((L, Hq, D)), K, V)
    mean = np.cumsum(V, axis=0) / np.arange(1, L + 1)[:, None, None]
    for h in range(Hq):
        assert np.max(np.abs(out[:, h] - mean[:, h // 2])) <= 1e-13
    assert np.max(np.abs(lse[:, 0] - np.log(np.arange(1, L + 1)))) <= 1e-13

    # continuation row i sits at position L_prefix + i: mean over L_prefix + i + 1 keys
    Lp, S = 20, 11
    kc, vc = cache_from(K, V, Lp, 40)
    outc, _ = ref.continue_(np.zeros((S, Hq, D)), K[Lp:], V[Lp:], kc, vc, Lp)
    for h in range(Hq):
        assert np.max(np.abs(outc[:, h] - mean[Lp:, h // 2])) <= 1e-13


# ------------------------------------------------------- P5 Claim 1, oracle side
@pytest.mark.parametrize("Lp,S", [(0, 7), (1, 1), (16, 16), (50, 13), (128, 16)])
def test_claim1_continuation_equals_prefill_rows(Lp, S):
    """Continuing over a cached prefix reproduces the matching rows of a full prefill."""
    Hq, Hkv, D = 4, 2, 16
    n = Lp + S
    Q, K, V = rnd((n, Hq, D), 17), rnd((n, Hkv, D), 18), rnd((n, Hkv, D), 19)
    full, lse_full = ref.prefill(Q, K, V)
    kc, vc = cache_from(K, V, Lp, n + 3)
    cont, lse_c = ref.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp)
    assert np.max(np.abs(cont - full[Lp:])) <= 1e-12
    assert np.max(np.abs(lse_c - lse_full[Lp:])) <= 1e-12


# ---------------------------------------------------------------- P8 negatives
def test_shifted_failure_mode_is_detectable():
    """Hiding the prefix (the mask does not span it) changes the outputs far beyond tolerance."""
    Hq, Hkv, D, Lp, S = 4, 2, 16, 40, 8
    n = Lp + S
    Q, K, V = rnd((n, Hq, D), 20), rnd((n, Hkv, D), 21), rnd((n, Hkv, D), 22)
    kc, vc = cache_from(K, V, Lp, n)
    good, _ = ref.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp)
    hidden, _ = ref.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp, k_range=(Lp, n))
    fresh, _ = ref.prefill(Q[Lp:], K[Lp:], V[Lp:])   # positions restarted at 0
    assert np.max(np.abs(good - hidden)) > 0.1
    assert np.max(np.abs(good - fresh)) > 0.1


# ---------------------------------------------------------------- P9 causality
def test_causality_future_rows_do_not_matter():
    Hq, Hkv, D, L, t = 4, 1, 8, 30, 17
    Q, K, V = rnd((L, Hq, D), 23), rnd((L, Hkv, D), 24), rnd((L, Hkv, D), 25)
    a, la = ref.prefill(Q, K, V)
    K2, V2 = K.copy(), V.copy()
    K2[t:] = rnd((L - t, Hkv, D), 26) * 5
    V2[t:] = rnd((L - t, Hkv, D), 27) * 5
    b, lb = ref.prefill(Q, K2, V2)
    assert np.array_equal(a[:t], b[:t]) and np.array_equal(la[:t], lb[:t])
    assert np.max(np.abs(a[t:] - b[t:])) > 0.1


# -------------------------------------------------------------- P10 LSE merge
def test_lse_merge_of_key_splits():
    """Attention over disjoint key ranges, merged by log-sum-exp weights, equals the unsplit result."""
    Hq, Hkv, D, Lp, S = 4, 2, 16, 90, 6
    n = Lp + S
    Q, K, V = rnd((n, Hq, D), 28), rnd((n, Hkv, D), 29), rnd((n, Hkv, D), 30)
    kc, vc = cache_from(K, V, Lp, n)
    full, lse = ref.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp)
    cuts = [0, 13, 64, Lp, n]
    parts = [ref.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp, k_range=(a, b))
             for a, b in zip(cuts[:-1], cuts[1:])]
    lses = np.stack([p[1] for p in parts])            # [P, S, Hq]
    outs = np.stack([p[0] for p in parts])
    M = lses.max(axis=0)
    wts = np.exp(lses - M)
    merged_lse = M + np.log(wts.sum(axis=0))
    merged = (outs * np.exp(lses - merged_lse)[..., None]).sum(axis=0)
    assert np.max(np.abs(merged - full)) <= 1e-13
    assert np.max(np.abs(merged_lse - lse)) <= 1e-13


# ----------------------------------------------------------------- P11 GQA map
@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (32, 8), (6, 3), (4, 4)])
def test_gqa_head_map(Hq, Hkv):
    """V[:, g, :] = g makes out[:, h, :] = h // (Hq / Hkv) exactly."""
    L, D = 12, 8
    Q, K = rnd((L, Hq, D), 31), rnd((L, Hkv, D), 32)
    V = np.broadcast_to(np.arange(Hkv, dtype=np.float64)[None, :, None], (L, Hkv, D)).copy()
    out, _ = ref.prefill(Q, K, V)
    G = Hq // Hkv
    for h in range(Hq):
        assert np.max(np.abs(out[:, h] - h // G)) <= 1e-14


def test_cache_append_is_exact_copy():
    """Rows [L_cur, L_cur + S) become the new rows; every other row is untouched."""
    Hkv, cap, D, S, Lc = 3, 20, 4, 5, 7
    kc, vc = rnd((Hkv, cap, D), 33), rnd((Hkv, cap, D), 34)
    Ks, Vs = rnd((S, Hkv, D), 35), rnd((S, Hkv, D), 36)
    k2, v2 = ref.cache_append(kc, vc, Ks, Vs, Lc)
    for g in range(Hkv):
        assert np.array_equal(k2[g, Lc:Lc + S], Ks[:, g]) and np.array_equal(v2[g, Lc:Lc + S], Vs[:, g])
    mask = np.ones(cap, bool); mask[Lc:Lc + S] = False
    assert np.array_equal(k2[:, mask], kc[:, mask]) and np.array_equal(v2[:, mask], vc[:, mask])
    with pytest.raises(ValueError):
        ref.cache_append(kc, vc, Ks, Vs, cap - S + 1)


def test_bf16_inputs_widen_exactly():
    """The oracle reads bf16 inputs as their exact values (no second rounding)."""
    q, k, v = W.qkv(5, W.Shape(2, 1, 8, torch.bfloat16), seed=3)
    out, _ = ref.prefill(q, k, v)
    assert np.array_equal(out[0, 0], v[0, 0].double().numpy())

"""Pins of the RoPE oracle (``oracle/rope.py``) against facts fixed outside it.

* the complex-number form of rotary embedding: pair i is the complex number
  x[i] + 1j x[i + d/2], multiplied by exp(1j p theta_i) (a sign slip, a wrong
  pairing or a swapped cos/sin fails it);
* the two-dimensional case, a plane rotation by p radians (theta_0 = 1);
* the geometric frequencies theta_i = base ** (-2 i / d);
* invariants: identity at p = 0, norms kept, R_a R_b = R_(a+b), and scores that
  depend only on the distance between positions;
* the paper's exactness argument with positions (Section "Consuming an
  artifact"): a continuation at positions L.. over the rotated cache equals the
  matching rows of a prefill; positions that restart at 0 (the shifted failure
  mode the paper warns about) do not.
"""
import numpy as np
import pytest

from oracle import ref
from oracle import rope


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("d,base", [(128, 1e6), (64, 1e4), (8, 10.0), (2, 1e6)])
def test_complex_form(d, base):
    x = rnd((5, 3, d), d)
    pos = np.array([0, 1, 7, 1000, 40000])
    z = x[..., : d // 2] + 1j * x[..., d // 2:]
    th = base ** (-2.0 * np.arange(d // 2) / d)
    zr = z * np.exp(1j * pos[:, None, None] * th[None, None, :])
    want = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(rope.rotate(x, pos, base), want, rtol=0, atol=1e-12)


def test_plane_rotation():
    """d = 2: theta_0 = 1 for any base, so position p turns the plane by p radians."""
    x = np.array([[[1.0, 0.0]], [[0.0, 1.0]], [[3.0, 4.0]]])
    for p in (0, 1, 2, 5):
        y = rope.rotate(x, [p, p, p], base=12345.0)
        c, s = np.cos(p), np.sin(p)
        np.testing.assert_allclose(y[0, 0], [c, s], atol=1e-15)
        np.testing.assert_allclose(y[1, 0], [-s, c], atol=1e-15)
        np.testing.assert_allclose(y[2, 0], [3 * c - 4 * s, 4 * c + 3 * s], atol=1e-14)


def test_frequencies():
    th = rope.thetas(128, 1e6)
    assert th[0] == 1.0
    assert abs(th[32] - 1e6 ** -0.5) < 1e-18                     # i = d/4: base^(-1/2)
    np.testing.assert_allclose(th[1:] / th[:-1], 1e6 ** (-2.0 / 128), rtol=1e-13)
    tab = rope.table(128, 1e6, 5)
    assert tab.shape == (5, 64, 2)
    np.testing.assert_array_equal(tab[0, :, 0], 1.0)
    np.testing.assert_array_equal(tab[0, :, 1], 0.0)
    np.testing.assert_allclose(tab[3, 0], [np.cos(3.0), np.sin(3.0)], atol=1e-15)


def test_identity_norm_and_group():
    x = rnd((6, 4, 64), 2)
    np.testing.assert_array_equal(rope.rotate(x, np.zeros(6), 1e4), x)
    y = rope.rotate(x, np.arange(6) * 977, 1e4)
    pn = lambda a: a[..., :32] ** 2 + a[..., 32:] ** 2          # noqa: E731  squared norm of each pair
    np.testing.assert_allclose(pn(y), pn(x), rtol=1e-12)
    a, b = np.arange(6) * 31, np.arange(6) * 5 + 900
    np.testing.assert_allclose(rope.rotate(rope.rotate(x, a, 1e4), b, 1e4), rope.rotate(x, a + b, 1e4),
                               atol=1e-10)


def test_scores_depend_on_distance_only():
    q = rnd((1, 1, 128), 3)
    k = rnd((1, 1, 128), 4)
    s = lambda m, n: float(np.sum(rope.rotate(q, [m], 1e6) * rope.rotate(k, [n], 1e6)))  # noqa: E731
    for m, n, c in ((10, 3, 1000), (500, 0, 3774), (7, 7, 12345)):
        assert abs(s(m, n) - s(m + c, n + c)) < 1e-9
    assert abs(s(10, 3) - s(10, 4)) > 1e-3                    # the distance does matter


@pytest.mark.parametrize("Lp,S,Hq,Hkv", [(40, 9, 4, 2), (130, 17, 8, 2), (1, 5, 2, 1)])
def test_claim1_with_positions(Lp, S, Hq, Hkv):
    """Continuation at positions Lp.. over the rotated cache == prefill rows Lp..;
    a continuation that restarts its positions at 0 misses them."""
    d, base = 64, 1e4
    n = Lp + S
    g = np.random.default_rng(Lp + S)
    Q, K, V = g.standard_normal((n, Hq, d)), g.standard_normal((n, Hkv, d)), g.standard_normal((n, Hkv, d))
    full, _, k_rot = rope.prefill(Q, K, V, base)
    kc = np.transpose(k_rot[:Lp], (1, 0, 2)).copy()
    vc = np.transpose(V[:Lp], (1, 0, 2)).copy()
    got, _, kr_new = rope.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp, base)
    np.testing.assert_allclose(got, full[Lp:], rtol=0, atol=1e-12)
    np.testing.assert_allclose(kr_new, k_rot[Lp:], rtol=0, atol=1e-12)
    shifted, _, _ = rope.continue_(Q[Lp:], K[Lp:], V[Lp:], kc, vc, Lp, base, pos0=0)
    assert np.max(np.abs(shifted - full[Lp:])) > 1e-2
    # without RoPE on either side the positions would not matter: the rotation is what needs them
    plain, _ = ref.continue_(Q[Lp:], K[Lp:], V[Lp:], np.transpose(K[:Lp], (1, 0, 2)).copy(), vc, Lp)
    want, _ = ref.prefill(Q, K, V, rows=list(range(Lp, n)))
    np.testing.assert_allclose(plain, want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("fmt", ["bf16", "fp16", "fp32"])
def test_round_to_matches_torch(fmt):
    """Rounding to the element format against torch's own conversion of fp32
    values (a single correct rounding), including ties, subnormals of fp16 and
    values just around rounding boundaries."""
    import torch
    tdt = {"bf16": torch.bfloat16, "fp16": torch.float16, "fp32": torch.float32}[fmt]
    g = np.random.default_rng(11)
    x = np.concatenate([g.standard_normal(20000), g.standard_normal(2000) * 1e-6,
                        np.ldexp(g.integers(1, 4096, 2000).astype(np.float64), -30),
                        [0.0, -0.0, 1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -11,
                         65504.0, 2.0 ** -24, 3 * 2.0 ** -25]]).astype(np.float32)
    want = torch.from_numpy(x).to(tdt).to(torch.float64).numpy()
    np.testing.assert_array_equal(rope.round_to(x.astype(np.float64), fmt), want)
    assert rope.round_to(np.array([1.0 + 2.0 ** -8]), "bf16")[0] == 1.0        # tie to even
    assert rope.round_to(np.array([1.0 + 3 * 2.0 ** -8]), "bf16")[0] == 1.0 + 2.0 ** -6

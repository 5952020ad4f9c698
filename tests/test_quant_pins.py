"""Pins of the quantized-artifact oracle (oracle/quant.py) against closed forms,
invariants and the sizes the paper prints (Section "Quantizing the artifact:
size vs. exactness": a 692-token context, fp16 102.1 MB -> int8 51.1 MB, 2.0x).
"""
import numpy as np
import pytest

from harness import accounting as A
from oracle import quant as Q
from oracle import ref


def test_exact_scale_round_half_even_and_symmetry():
    """max|x| = 127 gives s = 1 exactly: codes are the round-half-even of x."""
    x = np.array([127.0, 0.5, 1.5, 2.5, -2.5, -127.0, 3.49, -0.5, 126.5], dtype=np.float32)
    q, s = Q.quantize(x)
    assert s == np.float32(1.0)
    assert q.tolist() == [127, 0, 2, 2, -2, -127, 3, 0, 126]
    q2, s2 = Q.quantize(-x)
    assert s2 == s and (q2 == -q).all()


def test_power_of_two_scale():
    """max|x| = 63.5 gives s = 0.5 exactly: x / s is exact, ties to even."""
    x = np.array([63.5, 0.25, 0.75, -0.25, -63.5, 1.25], dtype=np.float32)
    q, s = Q.quantize(x)
    assert s == np.float32(0.5)
    assert q.tolist() == [127, 0, 2, 0, -127, 2]


def test_zero_tensor():
    q, s = Q.quantize(np.zeros((3, 4), dtype=np.float32))
    assert s == np.float32(1.0) and (q == 0).all()


def test_codes_bounds_and_error_bound():
    """Random bf16-like data: the largest magnitude maps to +-127, every code is in
    [-127, 127], the dequantization error is at most s/2 (to fp32 rounding of x/s),
    and the map is monotonic."""
    rng = np.random.default_rng(7)
    for scale in (1e-3, 1.0, 37.0):
        x = (rng.standard_normal(5000) * scale).astype(np.float32)
        q, s = Q.quantize(x)
        assert q.dtype == np.int8
        assert q.min() >= -127 and q.max() <= 127
        i = int(np.argmax(np.abs(x)))
        assert abs(int(q[i])) == 127 and np.sign(q[i]) == np.sign(x[i])
        err = np.abs(Q.dequantize(q, s) - x.astype(np.float64))
        assert err.max() <= 0.5 * float(s) * (1 + 1e-6)
        order = np.argsort(x, kind="stable")
        assert (np.diff(q[order].astype(np.int32)) >= 0).all()


def test_scale_is_fp32_division():
    """s is the fp32 quotient max|x| / 127 (not an fp64 value)."""
    x = np.array([1.0, -3.0, 2.0], dtype=np.float32)
    _, s = Q.quantize(x)
    assert s == np.float32(np.float32(3.0) / np.float32(127.0))
    assert float(s) != 3.0 / 127.0


def test_per_tensor_cache_quantization():
    """One scale for all heads and rows [0, L) of K, one for V; rows past L ignored."""
    rng = np.random.default_rng(3)
    kc = rng.standard_normal((2, 10, 8)).astype(np.float32)
    vc = rng.standard_normal((2, 10, 8)).astype(np.float32)
    kc[1, 9, 0] = 1000.0          # past L = 9: must not set the scale
    kq, vq, sk, sv = Q.quantize_cache(kc, vc, 9)
    assert kq.shape == (2, 9, 8) and vq.shape == (2, 9, 8)
    assert sk == np.float32(np.max(np.abs(kc[:, :9])) / np.float32(127))
    assert sv == np.float32(np.max(np.abs(vc[:, :9])) / np.float32(127))


def test_continue_over_exact_codes_is_the_plain_oracle():
    """When the cache holds integers times a power of two the quantization is exact,
    and continue_q8 equals the bf16-cache oracle bit for bit."""
    rng = np.random.default_rng(11)
    Hq, Hkv, D, L, S = 4, 2, 8, 12, 3
    kc = (rng.integers(-127, 128, (Hkv, L, D)) * 0.25).astype(np.float32)
    vc = (rng.integers(-127, 128, (Hkv, L, D)) * 0.5).astype(np.float32)
    kc[0, 0, 0] = 127 * 0.25
    vc[0, 0, 0] = 127 * 0.5
    qs = rng.standard_normal((S, Hq, D)).astype(np.float32)
    ks = rng.standard_normal((S, Hkv, D)).astype(np.float32)
    vs = rng.standard_normal((S, Hkv, D)).astype(np.float32)
    kq, vq, sk, sv = Q.quantize_cache(kc, vc, L)
    assert sk == np.float32(0.25) and sv == np.float32(0.5)
    a, la = Q.continue_q8(qs, ks, vs, kq, vq, sk, sv, L)
    b, lb = ref.continue_(qs, ks, vs, kc, vc, L)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_quantized_continuation_differs_but_stays_close():
    """Quantization is lossy (the paper: exactness is broken), yet on N(0,1) data the
    attention output moves by far less than the spread of V."""
    rng = np.random.default_rng(5)
    Hq, Hkv, D, L, S = 4, 2, 16, 64, 4
    kc = rng.standard_normal((Hkv, L, D)).astype(np.float32)
    vc = rng.standard_normal((Hkv, L, D)).astype(np.float32)
    qs = rng.standard_normal((S, Hq, D)).astype(np.float32)
    ks = rng.standard_normal((S, Hkv, D)).astype(np.float32)
    vs = rng.standard_normal((S, Hkv, D)).astype(np.float32)
    kq, vq, sk, sv = Q.quantize_cache(kc, vc, L)
    a, _ = Q.continue_q8(qs, ks, vs, kq, vq, sk, sv, L)
    b, _ = ref.continue_(qs, ks, vs, kc, vc, L)
    d = np.abs(a - b).max()
    assert 0 < d < 0.05


def test_artifact_sizes_match_the_paper():
    """692 tokens, 36 layers x 8 kv heads x 128: fp16 102.1 MB, int8 51.1 MB, 2.0x.
    The printed sizes include a file format this model does not have; allow 0.1 MB."""
    fp16 = A.kv_bytes_per_token(8, 128, 2, layers=36) * 692
    q8 = A.q8_artifact_bytes(692, 8, 128, layers=36)
    assert abs(fp16 / 1e6 - 102.1) < 0.1
    assert abs(q8 / 1e6 - 51.1) < 0.1
    assert round(fp16 / q8, 1) == 2.0

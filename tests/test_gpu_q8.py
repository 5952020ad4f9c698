"""GPU parity of the int8 KV artifact (kvr_quantize_cache, kvr_continue_q8)
against the oracle of oracle/quant.py.

Bars: the int8 codes and the two scales are bit-exact (they are integers and
fp32 values decided in the same fp32 arithmetic on both sides); the
continuation over the artifact matches the fp64 oracle over the dequantized
cache within the bf16 tolerance 1e-2.  Codes are compared in their natural
[kv head][row][head dim] order after undoing the artifact's documented byte
order (include/kvr.h).
"""
import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import quant as QO
from oracle import ref
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu

TOL = 1e-2
DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def pos_k(d):
    return 64 * ((d >> 3) & 1) + 8 * (d >> 4) + (d & 7)


def pos_v(k):
    return 16 * ((k >> 2) & 1) + 8 * (k >> 4) + 4 * ((k >> 3) & 1) + (k & 3)


def natural_codes(desc, kq, vq, L):
    """Undo the artifact byte order: (K codes [Hkv, L, 128], V codes [Hkv, L, 128], padding rows)."""
    Hkv, D = desc.n_kv_heads, desc.head_dim
    P = (desc.capacity + 31) // 32 * 32
    kq = kq.cpu().numpy().reshape(Hkv, P, D)
    vq = vq.cpu().numpy().reshape(Hkv, P // 32, D, 32)
    k_nat = kq[:, :, pos_k(np.arange(D))]                          # [Hkv, P, D]
    v_blk = vq[:, :, :, pos_v(np.arange(32))]                      # [Hkv, P/32, D, key]
    v_nat = v_blk.transpose(0, 1, 3, 2).reshape(Hkv, P, D)
    Lp = (L + 31) // 32 * 32
    return k_nat[:, :L], v_nat[:, :L], (k_nat[:, L:Lp], v_nat[:, L:Lp])


def make_cache(Hkv, cap, L, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    kc = (torch.randn((Hkv, cap, 128), generator=g) * scale).to(torch.bfloat16)
    vc = (torch.randn((Hkv, cap, 128), generator=g) * scale).to(torch.bfloat16)
    return kc, vc


def gpu_quantize(desc, kc, vc, L):
    kq, vq, sc = kvr.q8_artifact(desc)
    kq.fill_(77)           # the padding rows must come out as zero codes
    vq.fill_(77)
    kvr.kvr_quantize_cache(desc, kc.to(DEV), vc.to(DEV), L, kq, vq, sc)
    torch.cuda.synchronize()
    return kq, vq, sc


@pytest.mark.parametrize("cap,L,scale,seed", [
    (64, 1, 1.0, 0), (160, 100, 1.0, 1), (4096, 3774, 1.0, 2), (300, 257, 37.0, 3), (128, 128, 1e-3, 4),
])
def test_quantize_bit_exact(cap, L, scale, seed):
    say("quantize: cap %d L %d scale %g" % (cap, L, scale))
    Hkv = 8
    desc = kvr.make_desc(32, Hkv, 128, kvr.KVR_BF16, cap)
    kc, vc = make_cache(Hkv, cap, L, seed, scale)
    kq, vq, sc = gpu_quantize(desc, kc, vc, L)
    want_k, want_v, sk, sv = QO.quantize_cache(kc, vc, L)
    got = sc.cpu().numpy()
    assert got[0] == sk and got[1] == sv, (got, sk, sv)
    k_nat, v_nat, (k_pad, v_pad) = natural_codes(desc, kq, vq, L)
    assert np.array_equal(k_nat, want_k)
    assert np.array_equal(v_nat, want_v)
    assert (k_pad == 0).all() and (v_pad == 0).all()


def test_quantize_zero_tensor():
    say("quantize: all-zero cache")
    desc = kvr.make_desc(32, 8, 128, kvr.KVR_BF16, 64)
    kc = torch.zeros((8, 64, 128), dtype=torch.bfloat16)
    kq, vq, sc = gpu_quantize(desc, kc, kc.clone(), 40)
    assert sc.cpu().tolist() == [1.0, 1.0]
    k_nat, v_nat, _ = natural_codes(desc, kq, vq, 40)
    assert (k_nat == 0).all() and (v_nat == 0).all()


def run_q8(desc, L_art, Lp, S, seed, rows=None):
    """Quantize an artifact of L_art rows, continue S tokens over its first Lp rows."""
    Hq, Hkv = desc.n_q_heads, desc.n_kv_heads
    cap = desc.capacity
    kc, vc = make_cache(Hkv, cap, L_art, seed)
    kq, vq, sc = gpu_quantize(desc, kc, vc, L_art)
    sh = W.Shape(Hq, Hkv, 128, torch.bfloat16)
    qs, ks, vs = W.qkv(S, sh, seed=seed + 100)
    out = torch.empty((S, Hq, 128), dtype=torch.bfloat16, device=DEV)
    ws = kvr.workspace_for(desc, Lp, S)
    kvr.kvr_continue_q8(desc, qs.to(DEV), ks.to(DEV), vs.to(DEV), kq, vq, sc, Lp, S, out, ws)
    torch.cuda.synchronize()
    k_codes, v_codes, sk, sv = QO.quantize_cache(kc, vc, L_art)
    want, _ = QO.continue_q8(qs, ks, vs, k_codes, v_codes, sk, sv, Lp, rows=rows)
    got = out.float().cpu().numpy().astype(np.float64)
    if rows is not None:
        got = got[rows]
    return got, want, (kc, vc, qs, ks, vs, out, kq, vq, sc)


@pytest.mark.parametrize("Lp,S,extra", [
    (1, 1, 0), (100, 24, 0), (1000, 1, 7), (3774, 24, 0), (3774, 3, 40), (5000, 17, 0), (257, 24, 1),
    (32768 + 5, 1, 0), (32768 + 2, 24, 9),      # prefixes just past a round length (last split takes the extra keys)
    (1, 24, 0), (40, 24, 0), (65, 9, 3), (64, 24, 0),   # one or two cached stages
])
def test_continue_q8_matches_oracle(Lp, S, extra):
    say("continue_q8: Lp %d S %d artifact %d" % (Lp, S, Lp + extra))
    desc = kvr.make_desc(32, 8, 128, kvr.KVR_BF16, Lp + extra + 8)
    got, want, _ = run_q8(desc, Lp + extra, Lp, S, seed=Lp + S)
    err = np.abs(got - want).max()
    assert err <= TOL, err


def test_continue_q8_other_group_sizes():
    """G = 1 (96 rows = 3 column tiles at S = 96), G = 8, G = 2 (40 and 64 rows, up to 32
    new tokens) and two kv heads."""
    for Hq, Hkv, S in ((8, 8, 96), (64, 8, 12), (16, 8, 20), (16, 8, 32), (16, 2, 5)):
        say("continue_q8: Hq %d Hkv %d S %d" % (Hq, Hkv, S))
        desc = kvr.make_desc(Hq, Hkv, 128, kvr.KVR_BF16, 2048)
        got, want, _ = run_q8(desc, 2000, 2000, S, seed=Hq)
        assert np.abs(got - want).max() <= TOL


def test_continue_q8_without_prefix_is_plain_continuation():
    """L_prefix = 0: nothing is quantized; the result equals kvr_continue bit for bit."""
    say("continue_q8: no prefix")
    desc = kvr.make_desc(32, 8, 128, kvr.KVR_BF16, 64)
    qs, ks, vs = (x.to(DEV) for x in W.qkv(24, W.QWEN, seed=5))
    kq, vq, sc = kvr.q8_artifact(desc)
    a = torch.empty((24, 32, 128), dtype=torch.bfloat16, device=DEV)
    b = torch.empty_like(a)
    kvr.kvr_continue_q8(desc, qs, ks, vs, kq, vq, sc, 0, 24, a)
    kvr.kvr_continue(desc, qs, ks, vs, None, None, 0, 24, b)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_continue_q8_full_size_sampled_and_deterministic():
    """The 32k-token decode-chain layer: S = 1 and S = 24 over a 32768-row artifact,
    sampled rows from the oracle; a second run is bit-identical."""
    for S in (1, 24):
        say("continue_q8: 32768 prefix, S %d" % S)
        desc = kvr.make_desc(32, 8, 128, kvr.KVR_BF16, 32768 + 24)
        rows = sorted({0, S - 1, S // 2})
        got, want, t = run_q8(desc, 32768, 32768, S, seed=11 + S, rows=rows)
        assert np.abs(got - want).max() <= TOL
        kc, vc, qs, ks, vs, out, kq, vq, sc = t
        again = torch.empty_like(out)
        kvr.kvr_continue_q8(desc, qs.to(DEV), ks.to(DEV), vs.to(DEV), kq, vq, sc, 32768, S, again,
                            kvr.workspace_for(desc, 32768, S))
        torch.cuda.synchronize()
        assert torch.equal(out, again)


def test_q8_is_lossy_but_close_to_the_bf16_cache():
    """The paper's finding: int8 is not exact.  Against the unquantized bf16 cache the
    outputs move, by far less than the spread of V on N(0,1) data."""
    say("continue_q8 vs bf16 cache")
    Lp, S = 3774, 24
    desc = kvr.make_desc(32, 8, 128, kvr.KVR_BF16, Lp + 8)
    got, _, t = run_q8(desc, Lp, Lp, S, seed=9)
    kc, vc, qs, ks, vs, *_ = t
    exact, _ = ref.continue_(qs, ks, vs, kc, vc, Lp)
    d = np.abs(got - exact).max()
    say("  max |int8 - bf16-cache oracle| = %.4g" % d)
    assert 0 < d < 0.05

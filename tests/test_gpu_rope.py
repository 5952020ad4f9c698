"""GPU parity of RoPE with the position offset against the fp64 oracle
(``oracle/rope.py``), through the C ABI.

Bars.  The table's cos/sin are fp64 values rounded once to fp32: within
2^-24 of the oracle's.  A rotated row is computed in fp32 and rounded once to
the element format; the oracle rounds its fp64 rotation to the same format, so
the two agree but for rare rows near a rounding boundary, which differ by one
unit in the last place: 2^-7 |y| (bf16), 2^-10 |y| (fp16), a few ulps (fp32).
Attention outputs keep the bars of the plain paths (1e-2 bf16, 5e-3 fp16, 1e-5
fp32 against the oracle, which attends over the rounded rotated rows).  Between a
GPU continuation and the matching rows of a GPU prefill (Claim 1 with
positions): 2e-3 plus one output ulp, since both rotate every row to the same
bits.  Cache rows written by different calls at the same position are
bit-identical.
"""
import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import rope as ORope
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu

DEV = "cuda"
BASE = ORope.QWEN3_BASE
TOL = {torch.bfloat16: 1e-2, torch.float16: 5e-3, torch.float32: 1e-5}
ULP = {torch.bfloat16: 2.0 ** -7, torch.float16: 2.0 ** -10, torch.float32: 2.0 ** -21}
CLAIM1 = {torch.bfloat16: (2e-3, 2.0 ** -7), torch.float16: (2e-3, 2.0 ** -10), torch.float32: (1e-5, 0.0)}


def say(msg):
    print(msg, flush=True)


def dev(*ts):
    return [t.to(DEV).contiguous() for t in ts]


def maxabs(gpu, want):
    return float(np.max(np.abs(gpu.double().cpu().numpy() - want))) if want.size else 0.0


def claim1(a, b, dt):
    tol, ulp = CLAIM1[dt]
    a, b = a.double().cpu(), b.double().cpu()
    worst = float(((a - b).abs() - (tol + ulp * b.abs())).max())
    assert worst <= 0.0, worst


def within_ulp(gpu, want, dt):
    g = gpu.double().cpu().numpy()
    bound = ULP[dt] * np.abs(want) + 1e-6
    worst = float(np.max(np.abs(g - want) - bound))
    assert worst <= 0.0, worst


def to_cache(rows, cap):
    """[n, H, d] rows -> [H, cap, d] (zeros past n), as the oracle expects a cache."""
    if isinstance(rows, torch.Tensor):
        rows = rows.double().numpy()
    n, H, d = rows.shape
    out = np.zeros((H, cap, d))
    out[:, :n] = np.transpose(np.asarray(rows, dtype=np.float64), (1, 0, 2))
    return out


def prefill_rope(sh, tab, q, k, v, cap=None):
    L = q.shape[0]
    cap = cap if cap is not None else L
    d = kvr.make_desc(sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.dtype, cap)
    qd, kd, vd = dev(q, k, v)
    out = torch.empty_like(qd)
    kc = torch.zeros((sh.n_kv_heads, cap, sh.head_dim), dtype=sh.dtype, device=DEV)
    vc = torch.zeros_like(kc)
    kvr.kvr_prefill_rope(d, tab, qd, kd, vd, L, out, kc, vc)
    return out, kc, vc, d


@pytest.mark.parametrize("D,base,n", [(128, 1e6, 40000), (64, 1e4, 3000)])
def test_table(D, base, n):
    say("rope table d=%d base=%g n=%d" % (D, base, n))
    tab = kvr.RopeTable(D, n, base)
    torch.cuda.synchronize()
    want = ORope.table(D, base, n)
    got = tab.cos_sin.double().cpu().numpy()
    assert float(np.max(np.abs(got - want))) <= 2.0 ** -24 + 1e-12


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float16, torch.float32])
@pytest.mark.parametrize("D", [128, 64])
def test_apply(dt, D):
    say("rope apply %s d=%d" % (dt, D))
    tab = kvr.RopeTable(D, 4000, BASE)
    d = kvr.make_desc(8, 8, D, dt, 0)
    x = torch.randn((50, 8, D), generator=W.gen(D)).to(dt)
    xd = dev(x)[0]
    y = kvr.kvr_rope_apply(d, tab, xd, 3000, torch.empty_like(xd))
    torch.cuda.synchronize()
    want = ORope.rotate(x, 3000 + np.arange(50), BASE)
    within_ulp(y, want, dt)
    kvr.kvr_rope_apply(d, tab, xd, 3000)          # in place: the same bits
    torch.cuda.synchronize()
    assert torch.equal(xd, y)


CASES_PREFILL = [(32, 8, 128, 1, torch.bfloat16), (32, 8, 128, 70, torch.bfloat16),
                 (32, 8, 128, 1100, torch.bfloat16), (8, 2, 64, 130, torch.bfloat16),
                 (32, 8, 128, 300, torch.float16), (4, 2, 64, 100, torch.float32),
                 (4, 4, 128, 90, torch.float32)]


@pytest.mark.parametrize("Hq,Hkv,D,L,dt", CASES_PREFILL)
def test_prefill_rope(Hq, Hkv, D, L, dt):
    say("prefill rope %d/%d/%d L=%d %s" % (Hq, Hkv, D, L, dt))
    sh = W.Shape(Hq, Hkv, D, dt)
    tab = kvr.RopeTable(D, L + 8, BASE)
    q, k, v = W.qkv(L, sh, seed=L + D + 1)
    out, kc, vc, d = prefill_rope(sh, tab, q, k, v, cap=L + 8)
    torch.cuda.synchronize()
    want, _, k_rot = ORope.prefill(q, k, v, BASE, fmt=dt)
    assert maxabs(out, want) <= TOL[dt]
    # cache: rotated keys within an ulp of the oracle's, bit-identical to the
    # standalone rotation; values copied bit for bit; rows past L untouched
    within_ulp(kc[:, :L], np.transpose(k_rot, (1, 0, 2)), dt)
    kd = dev(k)[0]
    kr = kvr.kvr_rope_apply(d, tab, kd, 0, torch.empty_like(kd))
    torch.cuda.synchronize()
    assert torch.equal(kc[:, :L].cpu(), kr.transpose(0, 1).cpu())
    assert torch.equal(vc[:, :L].cpu(), v.transpose(0, 1))
    assert not torch.any(kc[:, L:]) and not torch.any(vc[:, L:])


# (Lp, S): the row-split kernel (1000 + 24), the keys-split kernel (decode, long
# ranges), the register-staged kernel (more than 96 rows), no prefix at all
@pytest.mark.parametrize("Lp,S,dt", [(1000, 24, torch.bfloat16), (3774, 24, torch.bfloat16),
                                     (900, 1, torch.bfloat16), (20000, 24, torch.bfloat16),
                                     (300, 40, torch.bfloat16), (0, 7, torch.bfloat16),
                                     (1000, 24, torch.float16), (200, 9, torch.float32),
                                     (32768 + 6, 1, torch.bfloat16), (32768 + 2, 12, torch.float16)])
def test_continue_rope(Lp, S, dt):
    say("continue rope Lp=%d S=%d %s" % (Lp, S, dt))
    Hq, Hkv, D = (32, 8, 128) if dt != torch.float32 else (4, 2, 64)
    sh = W.Shape(Hq, Hkv, D, dt)
    n = Lp + S
    tab = kvr.RopeTable(D, n, BASE)
    q, k, v = W.qkv(n, sh, seed=5 + Lp + S)
    if Lp:
        _, kc, vc, d = prefill_rope(sh, tab, q[:Lp], k[:Lp], v[:Lp], cap=n)
    else:
        d = kvr.make_desc(Hq, Hkv, D, dt, n)
        kc = torch.zeros((Hkv, n, D), dtype=dt, device=DEV)
        vc = torch.zeros_like(kc)
    qs, ks, vs = dev(q[Lp:], k[Lp:], v[Lp:])
    out = torch.empty_like(qs)
    ws = kvr.workspace_for_rope(d, Lp, S)
    kvr.kvr_continue_rope(d, tab, qs, ks, vs, kc, vc, Lp, S, out, ws)
    torch.cuda.synchronize()
    assert not torch.any(kc[:, Lp:])                  # append off: the cache is read only
    k_rot_prefix = ORope.round_to(ORope.rotate(k[:Lp], np.arange(Lp), BASE), dt)
    want, _, _ = ORope.continue_(q[Lp:], k[Lp:], v[Lp:], to_cache(k_rot_prefix, n), to_cache(v[:Lp], n), Lp, BASE,
                                 fmt=dt)
    assert maxabs(out, want) <= TOL[dt]
    # append: the same output, and cache rows identical to a prefill's
    out2 = torch.empty_like(qs)
    kvr.kvr_continue_rope(d, tab, qs, ks, vs, kc, vc, Lp, S, out2, ws, append=True)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    if n <= 4000:
        full, kcf, vcf, _ = prefill_rope(sh, tab, q, k, v, cap=n)
        torch.cuda.synchronize()
        claim1(out, full[Lp:], dt)
        assert torch.equal(kc, kcf) and torch.equal(vc, vcf)


def test_shifted_positions_diverge():
    """The paper's shifted failure mode on the GPU: the same continuation with
    its rows rotated at positions 0.. instead of L.. (plain kvr_continue over
    rows rotated by kvr_rope_apply) misses the prefill rows that the RoPE
    continuation reproduces."""
    say("shifted positions")
    sh = W.Shape(32, 8, 128, torch.bfloat16)
    Lp, S = 1000, 24
    n = Lp + S
    tab = kvr.RopeTable(128, n, BASE)
    q, k, v = W.qkv(n, sh, seed=99)
    full, _, _, _ = prefill_rope(sh, tab, q, k, v)
    _, kc, vc, d = prefill_rope(sh, tab, q[:Lp], k[:Lp], v[:Lp], cap=n)
    qs, ks, vs = dev(q[Lp:], k[Lp:], v[Lp:])
    good = torch.empty_like(qs)
    kvr.kvr_continue_rope(d, tab, qs, ks, vs, kc, vc, Lp, S, good, kvr.workspace_for_rope(d, Lp, S))
    for pos0, expect_match in ((Lp, True), (0, False)):
        qr = kvr.kvr_rope_apply(d, tab, qs, pos0, torch.empty_like(qs))
        kr = kvr.kvr_rope_apply(d, tab, ks, pos0, torch.empty_like(ks))
        out = torch.empty_like(qs)
        kvr.kvr_continue(d, qr, kr, vs, kc, vc, Lp, S, out, kvr.workspace_for(d, Lp, S))
        torch.cuda.synchronize()
        err = float((out.double() - full[Lp:].double()).abs().max())
        say("  rows rotated at %d..: max |diff| vs prefill %.3g" % (pos0, err))
        if expect_match:
            claim1(out, full[Lp:], torch.bfloat16)
            assert torch.equal(out, good)
        else:
            assert err > 0.1
    claim1(good, full[Lp:], torch.bfloat16)


@pytest.mark.parametrize("Hq,Hkv,D,dt", [(32, 8, 128, torch.bfloat16), (8, 2, 64, torch.bfloat16),
                                         (32, 8, 128, torch.float16), (4, 2, 64, torch.float32)])
def test_readers_rope(Hq, Hkv, D, dt):
    say("readers rope %d/%d/%d %s" % (Hq, Hkv, D, dt))
    sh = W.Shape(Hq, Hkv, D, dt)
    Lp = 700
    lens = [24, 0, 77, 256, 5]
    cu = W.cu_seqlens(lens)
    tab = kvr.RopeTable(D, Lp + max(lens), BASE)
    g = W.gen(7 + D)
    qp, kp, vp = W.qkv(Lp, sh, generator=g)
    qs, ks, vs = W.qkv(cu[-1], sh, generator=g)
    _, kc, vc, d = prefill_rope(sh, tab, qp, kp, vp, cap=Lp)
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.empty_like(qd)
    ws = kvr.workspace_for_rope(d, Lp, cu[-1], len(lens))
    kvr.kvr_continue_batched_rope(d, tab, qd, kd, vd, cu, kc, vc, Lp, out, ws)
    torch.cuda.synchronize()
    assert torch.equal(kd.cpu(), ks)                  # inputs untouched
    kc_o = to_cache(ORope.round_to(ORope.rotate(kp, np.arange(Lp), BASE), dt), Lp)
    vc_o = to_cache(vp, Lp)
    for r in range(len(lens)):
        a, b = cu[r], cu[r + 1]
        if a == b:
            continue
        want, _, _ = ORope.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp, BASE, fmt=dt)
        assert maxabs(out[a:b], want) <= TOL[dt], r


def test_decode_chain_rope():
    """Decode steps as single calls: continue_rope(S = 1, append) at positions
    L, L+1, ...; the rows equal a prefill of the whole sequence."""
    say("decode chain rope")
    sh = W.Shape(32, 8, 128, torch.bfloat16)
    Lp, T = 777, 6
    n = Lp + T
    tab = kvr.RopeTable(128, n, BASE)
    q, k, v = W.qkv(n, sh, seed=123)
    _, kc, vc, d = prefill_rope(sh, tab, q[:Lp], k[:Lp], v[:Lp], cap=n)
    ws = kvr.workspace_for_rope(d, n, 1)
    outs = []
    for t in range(T):
        qs, ks, vs = dev(q[Lp + t:Lp + t + 1], k[Lp + t:Lp + t + 1], v[Lp + t:Lp + t + 1])
        o = torch.empty_like(qs)
        kvr.kvr_continue_rope(d, tab, qs, ks, vs, kc, vc, Lp + t, 1, o, ws, append=True)
        outs.append(o)
    full, kcf, vcf, _ = prefill_rope(sh, tab, q, k, v)
    torch.cuda.synchronize()
    got = torch.cat(outs)
    claim1(got, full[Lp:], torch.bfloat16)
    assert torch.equal(kc, kcf) and torch.equal(vc, vcf)
    want, _, _ = ORope.prefill(q, k, v, BASE, rows=list(range(Lp, n)), fmt=torch.bfloat16)
    assert maxabs(got, want) <= TOL[torch.bfloat16]

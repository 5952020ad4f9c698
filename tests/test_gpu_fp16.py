"""GPU parity of the fp16 path (the paper's precision) against the fp64 oracle.

fp16 uses the same kernels as bf16 with fp16 MFMA operands.  Bars, derived
from the arithmetic: fp16 rounds to 11 significant bits, so the output's own
rounding moves it by at most |x|·2^-11, the weights P carry 2^-11 relative
rounding into the second product, and the accumulation is fp32.  On N(0,1)
workloads (|x| up to about 3) that is below 2e-3; the oracle bar is 5e-3.
Between a GPU continuation and the matching GPU prefill rows: 2e-3 plus one
output ulp (|x|·2^-10), as for bf16.  Cache rows are bit-exact copies.
"""
import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import ref
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu

TOL = 5e-3
CLAIM1_TOL = 2e-3
DEV = "cuda"
F16 = torch.float16


def say(msg):
    print(msg, flush=True)


def dev(*ts):
    return [t.to(DEV).contiguous() for t in ts]


def maxabs(gpu, want):
    return float(np.max(np.abs(gpu.float().cpu().numpy().astype(np.float64) - want))) if want.size else 0.0


def claim1(a, b):
    a = a.double().cpu()
    b = b.double().cpu()
    worst = float(((a - b).abs() - (CLAIM1_TOL + 2.0 ** -10 * b.abs())).max())
    assert worst <= 0.0, worst


def prefill(sh, q, k, v, cap=None, kc=None, vc=None):
    L = q.shape[0]
    cap = cap if cap is not None else L
    d = kvr.make_desc(sh.n_q_heads, sh.n_kv_heads, sh.head_dim, F16, cap)
    qd, kd, vd = dev(q, k, v)
    out = torch.empty_like(qd)
    if kc is None:
        kc = torch.zeros((sh.n_kv_heads, cap, sh.head_dim), dtype=F16, device=DEV)
        vc = torch.zeros_like(kc)
    kvr.kvr_prefill(d, qd, kd, vd, L, out, kc, vc)
    return out, kc, vc, d


def cont(d, qs, ks, vs, kc, vc, Lp):
    S = qs.shape[0]
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.empty_like(qd)
    kvr.kvr_continue(d, qd, kd, vd, kc, vc, Lp, S, out, kvr.workspace_for(d, Lp, S))
    return out


@pytest.mark.parametrize("Hq,Hkv,D,L", [(32, 8, 128, 1), (32, 8, 128, 70), (32, 8, 128, 1100), (8, 2, 64, 130),
                                        (4, 4, 128, 300)])
def test_prefill_f16_vs_oracle(Hq, Hkv, D, L):
    say("prefill fp16 %d/%d/%d L=%d" % (Hq, Hkv, D, L))
    sh = W.Shape(Hq, Hkv, D, F16)
    q, k, v = W.qkv(L, sh, seed=L + D)
    out, kc, vc, _ = prefill(sh, q, k, v)
    torch.cuda.synchronize()
    want, _ = ref.prefill(q, k, v)
    assert maxabs(out, want) <= TOL
    # the cache holds the K/V rows bit for bit
    assert torch.equal(kc.cpu(), k.transpose(0, 1).contiguous())
    assert torch.equal(vc.cpu(), v.transpose(0, 1).contiguous())


@pytest.mark.parametrize("Lp,S", [(1000, 24), (3774, 24), (900, 1), (20000, 24), (300, 40), (0, 7)])
def test_continue_f16_vs_oracle_and_prefill(Lp, S):
    """Every continuation kernel: waves split the rows (24 tokens, short ranges),
    the keys (decode, long ranges) or neither (more than 96 rows)."""
    say("continue fp16 32/8/128 Lp=%d S=%d" % (Lp, S))
    sh = W.Shape(32, 8, 128, F16)
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=3 + Lp + S)
    if Lp:
        _, kc, vc, d = prefill(sh, q[:Lp], k[:Lp], v[:Lp], cap=n + 2)
    else:
        kc = vc = None
        d = kvr.make_desc(32, 8, 128, F16, 0)
    out = cont(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    kc_o = k[:Lp].transpose(0, 1).contiguous()
    vc_o = v[:Lp].transpose(0, 1).contiguous()
    want, _ = ref.continue_(q[Lp:], k[Lp:], v[Lp:], kc_o, vc_o, Lp)
    assert maxabs(out, want) <= TOL
    if n <= 4000:
        full, _, _, _ = prefill(sh, q, k, v)
        torch.cuda.synchronize()
        claim1(out, full[Lp:])


def test_readers_and_decode_f16():
    """Many readers in one call, then a short decode chain with appends."""
    say("readers + decode fp16")
    sh = W.Shape(32, 8, 128, F16)
    Lp = 900
    lens = [24, 0, 77, 256, 5]
    cu = W.cu_seqlens(lens)
    g = W.gen(31)
    qp, kp, vp = W.qkv(Lp, sh, generator=g)
    qs, ks, vs = W.qkv(cu[-1], sh, generator=g)
    _, kc, vc, d = prefill(sh, qp, kp, vp, cap=Lp + 8)
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.empty_like(qd)
    kvr.kvr_continue_batched(d, qd, kd, vd, cu, kc, vc, Lp, out, kvr.workspace_for(d, Lp, cu[-1], len(lens)))
    torch.cuda.synchronize()
    kc_o, vc_o = kp.transpose(0, 1).contiguous(), vp.transpose(0, 1).contiguous()
    for r in range(len(lens)):
        a, b = cu[r], cu[r + 1]
        if a == b:
            continue
        want, _ = ref.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp)
        assert maxabs(out[a:b], want) <= TOL, r
    # decode: 4 steps of continue(S = 1) + append reproduce the oracle's rows
    q2, k2, v2 = W.qkv(4, sh, seed=41)
    outs = []
    for t in range(4):
        p = Lp + t
        outs.append(cont(d, q2[t:t + 1], k2[t:t + 1], v2[t:t + 1], kc, vc, p))
        kd1, vd1 = dev(k2[t:t + 1], v2[t:t + 1])
        kvr.kvr_cache_append(d, kd1, vd1, 1, kc, vc, p)
    torch.cuda.synchronize()
    qa = torch.cat([qp, q2])
    ka = torch.cat([kp, k2])
    va = torch.cat([vp, v2])
    want, _ = ref.prefill(qa, ka, va, rows=list(range(Lp, Lp + 4)))
    assert maxabs(torch.cat(outs), want) <= TOL


def test_f16_is_closer_than_bf16():
    """The same N(0,1) inputs through both 16-bit formats: fp16's three extra
    significand bits show in the error against the fp64 oracle."""
    say("fp16 vs bf16 error")
    errs = {}
    for dt in (torch.bfloat16, F16):
        sh = W.Shape(32, 8, 128, dt)
        q, k, v = W.qkv(600, W.Shape(32, 8, 128, torch.float32), seed=77)
        q, k, v = q.to(dt), k.to(dt), v.to(dt)
        d = kvr.make_desc(32, 8, 128, dt, 600)
        qd, kd, vd = dev(q, k, v)
        out = torch.empty_like(qd)
        kc = torch.zeros((8, 600, 128), dtype=dt, device=DEV)
        vc = torch.zeros_like(kc)
        kvr.kvr_prefill(d, qd, kd, vd, 600, out, kc, vc)
        torch.cuda.synchronize()
        want, _ = ref.prefill(q, k, v)
        errs[dt] = maxabs(out, want)
    say("  max err bf16 %.3g, fp16 %.3g" % (errs[torch.bfloat16], errs[F16]))
    assert errs[F16] < errs[torch.bfloat16] / 2


@pytest.mark.parametrize("Hq,Hkv,Lp,S", [(8, 2, 3000, 5), (16, 2, 2500, 3)])
def test_continue_f16_head_dim_64_split(Hq, Hkv, Lp, S):
    """head_dim 64 continuations with several key splits (the merge's
    4-rows-per-workgroup geometry) in fp16: oracle and Claim 1."""
    say("continue fp16 %d/%d/64 Lp=%d S=%d" % (Hq, Hkv, Lp, S))
    sh = W.Shape(Hq, Hkv, 64, F16)
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=43 + Lp)
    full, _, _, _ = prefill(sh, q, k, v)
    _, kc, vc, d = prefill(sh, q[:Lp], k[:Lp], v[:Lp], cap=n)
    assert kvr.kvr_workspace_bytes(d, Lp, S) > 0      # the plan splits the prefix
    out = cont(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    claim1(out, full[Lp:])
    want, _ = ref.continue_(q[Lp:], k[Lp:], v[Lp:], k[:Lp].transpose(0, 1).contiguous(),
                            v[:Lp].transpose(0, 1).contiguous(), Lp)
    assert maxabs(out, want) <= TOL

"""kvr_continue_append (a continuation and its tokens' cache update in one
call) on every continuation path: the output is the very output of
kvr_continue (same kernels, same arithmetic), the cache rows L_prefix.. hold
the new K/V rows bit for bit, every other row is untouched, and a decode chain
of such steps reproduces the prefill rows (Claim 1 bar)."""
import pytest
import torch

from harness import workloads as W
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def dev(*ts):
    return [t.to(DEV).contiguous() for t in ts]


# the row-split and keys-split kernels store the rows themselves; d = 64, more
# than 96 rows and fp32 take the separate update
@pytest.mark.parametrize("Hq,Hkv,D,Lp,S,dt", [
    (32, 8, 128, 1000, 24, torch.bfloat16), (32, 8, 128, 3774, 24, torch.bfloat16),
    (32, 8, 128, 900, 1, torch.bfloat16), (32, 8, 128, 20000, 24, torch.bfloat16),
    (32, 8, 128, 0, 7, torch.bfloat16), (32, 8, 128, 1000, 24, torch.float16),
    (32, 8, 128, 300, 40, torch.bfloat16), (8, 2, 64, 500, 9, torch.bfloat16),
    (4, 2, 64, 200, 9, torch.float32), (8, 8, 128, 5000, 12, torch.bfloat16)])
def test_continue_append_equals_continue_then_append(Hq, Hkv, D, Lp, S, dt):
    say("continue_append %d/%d/%d Lp=%d S=%d %s" % (Hq, Hkv, D, Lp, S, dt))
    sh = W.Shape(Hq, Hkv, D, dt)
    cap = Lp + S + 5
    q, k, v = W.qkv(Lp + S, sh, seed=Lp + 3 * S)
    d = kvr.make_desc(Hq, Hkv, D, dt, cap)
    kc = torch.randn((Hkv, cap, D), generator=W.gen(1)).to(dt).to(DEV)    # canary rows everywhere
    vc = torch.randn((Hkv, cap, D), generator=W.gen(2)).to(dt).to(DEV)
    if Lp:
        kvr.kvr_cache_append(d, *dev(k[:Lp], v[:Lp]), Lp, kc, vc, 0)
    before_k, before_v = kc.clone(), vc.clone()
    qs, ks, vs = dev(q[Lp:], k[Lp:], v[Lp:])
    ws = kvr.workspace_for(d, Lp, S)
    ref_out = torch.empty_like(qs)
    kvr.kvr_continue(d, qs, ks, vs, kc, vc, Lp, S, ref_out, ws)
    out = torch.empty_like(qs)
    kvr.kvr_continue_append(d, qs, ks, vs, kc, vc, Lp, S, out, ws)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out)
    assert torch.equal(kc[:, Lp:Lp + S].cpu(), k[Lp:].transpose(0, 1))
    assert torch.equal(vc[:, Lp:Lp + S].cpu(), v[Lp:].transpose(0, 1))
    for a, b in ((kc, before_k), (vc, before_v)):
        assert torch.equal(a[:, :Lp], b[:, :Lp]) and torch.equal(a[:, Lp + S:], b[:, Lp + S:])


def test_decode_chain_with_fused_update():
    say("decode chain, fused update")
    sh = W.QWEN
    Lp, T = 1500, 8
    n = Lp + T
    q, k, v = W.qkv(n, sh, seed=17)
    d = kvr.make_desc(32, 8, 128, torch.bfloat16, n)
    qd, kd, vd = dev(q, k, v)
    full = torch.empty_like(qd)
    kc = torch.zeros((8, n, 128), dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    kvr.kvr_prefill(d, qd, kd, vd, n, full, kc, vc)
    kc2 = torch.zeros_like(kc)
    vc2 = torch.zeros_like(kc)
    kvr.kvr_prefill(d, *dev(q[:Lp], k[:Lp], v[:Lp]), Lp, torch.empty_like(qd[:Lp]), kc2, vc2)
    ws = kvr.workspace_for(d, n, 1)
    outs = []
    for t in range(Lp, n):
        o = torch.empty_like(qd[t:t + 1])
        kvr.kvr_continue_append(d, qd[t:t + 1], kd[t:t + 1], vd[t:t + 1], kc2, vc2, t, 1, o, ws)
        outs.append(o)
    torch.cuda.synchronize()
    got = torch.cat(outs).double()
    want = full[Lp:].double()
    assert float(((got - want).abs() - (2e-3 + 2.0 ** -7 * want.abs())).max()) <= 0.0
    assert torch.equal(kc, kc2) and torch.equal(vc, vc2)

"""The continuation entry point that allocates nothing (kvr_continue_noalloc)
against the one with a caller workspace (kvr_continue), through the C ABI:
bit-identical outputs on two calls in a row, the second with a smaller input
(the fixed buffer keeps the first call's partials; the second must not read
them), plus the oracle on the continuation rows."""
import pytest
import torch

from harness import workloads as W
from oracle import ref
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def case(Lp, S, seed):
    sh = W.QWEN
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=seed)
    d = kvr.make_desc(32, 8, 128, torch.bfloat16, n)
    kc = torch.zeros((8, n, 128), dtype=torch.bfloat16)
    vc = torch.zeros_like(kc)
    kc[:, :Lp] = k[:Lp].transpose(0, 1)
    vc[:, :Lp] = v[:Lp].transpose(0, 1)
    kc, vc = kc.to(DEV), vc.to(DEV)
    qs, ks, vs = (t[Lp:].contiguous().to(DEV) for t in (q, k, v))
    return q, k, v, d, kc, vc, qs, ks, vs


def test_noalloc_matches_workspace_entry_point():
    for Lp, S, seed in ((20000, 24, 1), (3000, 5, 2)):
        say("noalloc vs workspace continuation Lp=%d S=%d" % (Lp, S))
        q, k, v, d, kc, vc, qs, ks, vs = case(Lp, S, seed)
        assert kvr.kvr_workspace_bytes(d, Lp, S) > 0        # the plan uses split partials
        out_ws = torch.empty_like(qs)
        kvr.kvr_continue(d, qs, ks, vs, kc, vc, Lp, S, out_ws, kvr.workspace_for(d, Lp, S))
        out_na = torch.full_like(qs, float("nan"))
        kvr.kvr_continue_noalloc(d, qs, ks, vs, kc, vc, Lp, S, out_na)
        torch.cuda.synchronize()
        assert torch.equal(out_na, out_ws)
        want, _ = ref.prefill(q, k, v, rows=list(range(Lp, Lp + S)))
        err = float((out_na.double().cpu() - torch.from_numpy(want)).abs().max())
        assert err <= 1e-2, err


def test_noalloc_too_large_launches_nothing():
    d = kvr.make_desc(32, 8, 128, torch.bfloat16, 1 << 16)
    qs = torch.zeros((256, 32, 128), dtype=torch.bfloat16, device=DEV)
    ks = torch.zeros((256, 8, 128), dtype=torch.bfloat16, device=DEV)
    kc = torch.zeros((8, 1 << 16, 128), dtype=torch.bfloat16, device=DEV)
    out = torch.full_like(qs, 3.0)
    with pytest.raises(kvr.KvrError):
        kvr.kvr_continue_noalloc(d, qs, ks, ks, kc, kc, 20000, 256, out)
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())

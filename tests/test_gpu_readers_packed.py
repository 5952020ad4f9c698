"""Many readers on the two-group kernel: rows packed across readers, and the
last partial round of row tiles split over the keys and merged.

Every row of every reader against the fp64 oracle (1e-2 for 16-bit inputs),
on shapes that put reader boundaries inside row tiles (a row of a later
reader must not see the earlier readers' rows in its tile), readers of one
token, empty readers, no cached prefix, group sizes 1, 2, 3, 4 and 8 (3: rows
of a token straddle tiles, no key split), fp16, RoPE (bf16 and fp16), 128
readers in one launch and 129 in two, prefixes just at and below the split
threshold, and batches small enough that every tile is split.  Each case also checks that the call was planned
the way it names (split or not, from the workspace it asks for), that every
output row was written, and that two calls give the same bits.
"""
import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import ref
from oracle import rope as ORope
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu

DEV = "cuda"
TOL = 1e-2
F16 = torch.float16
BF16 = torch.bfloat16


def say(msg):
    print(msg, flush=True)


def dev(*ts):
    return [t.to(DEV).contiguous() for t in ts]


def maxabs(gpu, want):
    return float(np.max(np.abs(gpu.double().cpu().numpy() - want))) if want.size else 0.0


def lengths(kind, seed):
    g = torch.Generator()
    g.manual_seed(seed)
    if kind == "three":
        return [24, 200, 77]
    if kind == "tiny":            # 60 readers of 1-3 tokens: many boundaries per tile
        return [1 + int(x) for x in torch.randint(0, 3, (60,), generator=g)]
    if kind == "mixed":           # empty and one-token readers among longer ones
        return [5, 1, 60, 0, 130, 1, 0, 33]
    if kind == "flat93":          # 64 readers of 93 tokens: 93 tiles, 29 in the last round
        return [93] * 64
    if kind == "r128":            # the most readers one launch holds, 1-40 tokens each
        return [1 + int(x) for x in torch.randint(0, 40, (128,), generator=g)]
    if kind == "r129":            # one reader past a launch: packed per launch, never split
        return [1 + int(x) for x in torch.randint(0, 40, (129,), generator=g)]
    if kind.startswith("u"):      # "u<n>": n readers, S ~ U[24, 256]
        return [int(x) for x in torch.randint(24, 257, (int(kind[1:]),), generator=g)]
    raise ValueError(kind)


# (name, Hq, Hkv, dtype, L_prefix, lengths, split expected)
CASES = [
    ("3 readers over 3774, every tile split", 32, 8, BF16, 3774, "three", True),
    ("tiny readers over 1100, split", 32, 8, BF16, 1100, "tiny", True),
    ("mixed readers, no prefix", 32, 8, BF16, 0, "mixed", False),
    ("mixed readers over 200 (too few keys to split)", 32, 8, BF16, 200, "mixed", False),
    ("G = 1, 16 kv heads", 16, 16, BF16, 1500, "u40", True),
    ("G = 8", 64, 8, BF16, 1024, "u6", True),
    ("G = 3 (no split)", 24, 8, BF16, 700, "u40", False),
    ("fp16", 32, 8, F16, 2000, "u16", True),
    ("40 readers, a 23-tile last round kept whole", 32, 8, BF16, 2000, "u40", False),
    ("64 x 93 tokens, last round too full to split", 32, 8, BF16, 1500, "flat93", False),
    ("4 kv heads", 32, 4, BF16, 2100, "mixed", True),
    ("128 readers, one launch", 32, 8, BF16, 1000, "r128", True),
    ("129 readers, two launches", 32, 8, BF16, 1000, "r129", False),
    ("G = 2, 4 kv heads", 8, 4, BF16, 900, "u6", True),
    ("512 cached keys: two splits at most", 32, 8, BF16, 512, "three", True),
    ("511 cached keys: too few to split", 32, 8, BF16, 511, "three", False),
]


def run_case(Hq, Hkv, dt, Lp, lens, seed):
    sh = W.Shape(Hq, Hkv, 128, dt)
    cu = W.cu_seqlens(lens)
    total, n = cu[-1], len(lens)
    g = W.gen(seed)
    qp, kp, vp = W.qkv(max(Lp, 1), sh, generator=g)
    qs, ks, vs = W.qkv(total, sh, generator=g)
    d = kvr.make_desc(Hq, Hkv, 128, dt, max(Lp, 1))
    kc = torch.zeros((Hkv, max(Lp, 1), 128), dtype=dt, device=DEV)
    vc = torch.zeros_like(kc)
    if Lp > 0:
        qd, kd, vd = dev(qp[:Lp], kp[:Lp], vp[:Lp])
        kvr.kvr_prefill(d, qd, kd, vd, Lp, torch.empty_like(qd), kc, vc)
    qd, kd, vd = dev(qs, ks, vs)
    ws = kvr.workspace_for(d, Lp, total, n)
    outs = []
    for _ in range(2):
        out = torch.full_like(qd, float("nan"))
        kvr.kvr_continue_batched(d, qd, kd, vd, cu, kc, vc, Lp, out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    return cu, (qs, ks, vs), (kp[:Lp], vp[:Lp]), outs, ws, (d, kc, vc)


@pytest.mark.parametrize("name,Hq,Hkv,dt,Lp,kind,split", CASES, ids=[c[0] for c in CASES])
def test_packed_readers_vs_oracle(name, Hq, Hkv, dt, Lp, kind, split):
    say("packed readers: %s" % name)
    lens = lengths(kind, seed=Hq + Lp)
    cu, (qs, ks, vs), (kp, vp), (out, out2), ws, _ = run_case(Hq, Hkv, dt, Lp, lens, seed=Lp + 7)
    assert (ws is not None) == split, "workspace %s" % (None if ws is None else ws.numel())
    assert not torch.isnan(out).any()                     # every row written
    assert torch.equal(out, out2)                         # same bits on a second call
    kc_o, vc_o = kp.transpose(0, 1).contiguous(), vp.transpose(0, 1).contiguous()
    worst = 0.0
    for r in range(len(lens)):
        a, b = cu[r], cu[r + 1]
        if a == b:
            continue
        want, _ = ref.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp)
        err = maxabs(out[a:b], want)
        worst = max(worst, err)
        assert err <= TOL, (r, err)
    say("  max |gpu - oracle| = %.5f" % worst)


@pytest.mark.parametrize("dt", [BF16, F16], ids=["bf16", "fp16"])
def test_packed_readers_rope_split(dt):
    """RoPE: each reader's rows rotated at L_prefix + (token within the reader),
    not at their place in the packed tile; three readers, every tile split."""
    say("packed readers with RoPE, split, %s" % dt)
    sh = W.Shape(32, 8, 128, dt)
    Lp = 2000
    lens = [24, 100, 31]
    cu = W.cu_seqlens(lens)
    n = len(lens)
    tab = kvr.RopeTable(128, Lp + max(lens))
    g = W.gen(91)
    qp, kp, vp = W.qkv(Lp, sh, generator=g)
    qs, ks, vs = W.qkv(cu[-1], sh, generator=g)
    d = kvr.make_desc(32, 8, 128, dt, Lp)
    qd, kd, vd = dev(qp, kp, vp)
    kc = torch.zeros((8, Lp, 128), dtype=dt, device=DEV)
    vc = torch.zeros_like(kc)
    kvr.kvr_prefill_rope(d, tab, qd, kd, vd, Lp, torch.empty_like(qd), kc, vc)
    assert kvr.kvr_workspace_bytes(d, Lp, cu[-1], n) > 0      # the split plan
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.full_like(qd, float("nan"))
    kvr.kvr_continue_batched_rope(d, tab, qd, kd, vd, cu, kc, vc, Lp, out,
                                  kvr.workspace_for_rope(d, Lp, cu[-1], n))
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()
    fmt = "fp16" if dt == F16 else "bf16"
    k_rot = ORope.round_to(ORope.rotate(kp, np.arange(Lp), ORope.QWEN3_BASE), fmt)
    kc_o = np.transpose(k_rot, (1, 0, 2)).copy()
    vc_o = vp.transpose(0, 1).contiguous()
    for r in range(n):
        a, b = cu[r], cu[r + 1]
        want, _, _ = ORope.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp, ORope.QWEN3_BASE, fmt=fmt)
        assert maxabs(out[a:b], want) <= TOL, r


def test_split_tail_matches_unsplit_rows():
    """The split tail against the same rows computed whole: the readers of a
    batch small enough to split every tile, and the same readers as single
    continuations (kvr_continue, its own split plan): equal up to rounding."""
    say("split tail vs single continuations")
    Hq, Hkv, Lp = 32, 8, 3774
    lens = [24, 200, 77]
    cu, (qs, ks, vs), _, (out, _), ws, (d, kc, vc) = run_case(Hq, Hkv, BF16, Lp, lens, seed=5)
    assert ws is not None
    for r in range(len(lens)):
        a, b = cu[r], cu[r + 1]
        S = b - a
        q1, k1, v1 = dev(qs[a:b], ks[a:b], vs[a:b])
        o1 = torch.empty_like(q1)
        kvr.kvr_continue(d, q1, k1, v1, kc, vc, Lp, S, o1, kvr.workspace_for(d, Lp, S))
        torch.cuda.synchronize()
        diff = (o1.float() - out[a:b].float()).abs()
        bar = 2e-3 + out[a:b].float().abs() * 2.0 ** -7
        assert bool((diff <= bar).all()), (r, float(diff.max()))

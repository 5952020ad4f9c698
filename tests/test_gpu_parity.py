"""GPU parity: libkvr (through its C ABI) against the fp64 oracle.

Bars: max-abs error <= 1e-2 for bf16 inputs (fp32 accumulation), <= 1e-5 for
fp32 inputs; a GPU continuation agrees with the matching rows of a GPU
prefill within 2e-3 (Claim 1 of the paper); cache writes are bit-exact.
Small cases are checked on every element; the full-size workloads on sampled
rows the oracle can compute one by one.
"""
import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import ref
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu

TOL = {torch.bfloat16: 1e-2, torch.float32: 1e-5}
CLAIM1_TOL = 2e-3
DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def dev(*ts):
    return [t.to(DEV).contiguous() for t in ts]


def gpu_prefill(shape, q, k, v, capacity=None, kc=None, vc=None):
    L = q.shape[0]
    cap = capacity if capacity is not None else L
    d = kvr.make_desc(shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.dtype, cap)
    qd, kd, vd = dev(q, k, v)
    out = torch.empty_like(qd)
    if kc is None:
        kc = torch.zeros((shape.n_kv_heads, cap, shape.head_dim), dtype=shape.dtype, device=DEV)
        vc = torch.zeros_like(kc)
    kvr.kvr_prefill(d, qd, kd, vd, L, out, kc, vc)
    return out, kc, vc, d


def gpu_continue(d, qs, ks, vs, kc, vc, Lp):
    S = qs.shape[0]
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.empty_like(qd)
    ws = kvr.workspace_for(d, Lp, S)
    kvr.kvr_continue(d, qd, kd, vd, kc, vc, Lp, S, out, ws)
    return out


def claim1(a, b, dtype=torch.bfloat16):
    """Continuation rows vs prefill rows, both from the GPU.

    2e-3 on the workloads' scale; each bf16 result is also rounded to the
    output format on its own, so two different summation orders may land on
    neighbouring bf16 values: one output ulp (|x| * 2^-7) is allowed on top
    (it matters only where outputs exceed ~0.25, i.e. short contexts).
    """
    a = a.double().cpu()
    b = b.double().cpu()
    rel = 2.0 ** -7 if dtype == torch.bfloat16 else 0.0
    worst = float(((a - b).abs() - (CLAIM1_TOL + rel * b.abs())).max())
    assert worst <= 0.0, worst


def maxabs(gpu, want):
    return float(np.max(np.abs(gpu.float().cpu().numpy().astype(np.float64) - want))) if want.size else 0.0


# ------------------------------------------------------------ tiny fp32 workload
def test_tiny_fp32_workload():
    """2 q heads, 1 kv head, d 64, fp32: prefill 144, continue 16 over cached 128."""
    say("tiny fp32: prefill 144, continue 16 over 128")
    sh, Lp, S = W.TINY, W.TINY_L, W.TINY_S
    q, k, v = W.qkv(Lp + S, sh, seed=0)
    want, _ = ref.prefill(q, k, v)
    full, kc_full, _, _ = gpu_prefill(sh, q, k, v)
    torch.cuda.synchronize()
    assert maxabs(full, want) <= TOL[torch.float32]
    # cache of the prefix only, then continue
    _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=Lp + S)
    cont = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    assert maxabs(cont, want[Lp:]) <= TOL[torch.float32]
    assert float((cont - full[Lp:]).abs().max()) <= CLAIM1_TOL


# --------------------------------------------------------- prefill vs oracle
PREFILL_CASES = [  # (Hq, Hkv, d, L)
    (32, 8, 128, 1), (32, 8, 128, 2), (32, 8, 128, 31), (32, 8, 128, 33), (32, 8, 128, 63),
    (32, 8, 128, 64), (32, 8, 128, 65), (32, 8, 128, 129), (32, 8, 128, 517),
    (8, 8, 128, 100), (8, 1, 128, 300), (16, 2, 64, 200), (12, 3, 128, 150), (4, 2, 64, 77),
]


@pytest.mark.parametrize("Hq,Hkv,D,L", PREFILL_CASES)
def test_prefill_bf16_vs_oracle(Hq, Hkv, D, L):
    say("prefill bf16 Hq=%d Hkv=%d d=%d L=%d" % (Hq, Hkv, D, L))
    sh = W.Shape(Hq, Hkv, D, torch.bfloat16)
    q, k, v = W.qkv(L, sh, seed=L)
    out, kc, vc, _ = gpu_prefill(sh, q, k, v, capacity=L + 5)
    torch.cuda.synchronize()
    want, _ = ref.prefill(q, k, v)
    assert maxabs(out, want) <= TOL[torch.bfloat16]
    assert torch.equal(kc[:, :L].cpu(), k.transpose(0, 1)) and torch.equal(vc[:, :L].cpu(), v.transpose(0, 1))


@pytest.mark.parametrize("Hq,Hkv,D,L", [(32, 8, 128, 100), (8, 2, 64, 130), (4, 4, 128, 70)])
def test_prefill_fp32_vs_oracle(Hq, Hkv, D, L):
    say("prefill fp32 Hq=%d Hkv=%d d=%d L=%d" % (Hq, Hkv, D, L))
    sh = W.Shape(Hq, Hkv, D, torch.float32)
    q, k, v = W.qkv(L, sh, seed=L + 1)
    out, _, _, _ = gpu_prefill(sh, q, k, v)
    torch.cuda.synchronize()
    want, _ = ref.prefill(q, k, v)
    assert maxabs(out, want) <= TOL[torch.float32]


# ------------------------------------------------ continuation vs oracle and prefill
CONT_CASES = [  # (Lp, S)
    (0, 24), (1, 1), (5, 3), (64, 24), (100, 1), (1000, 24), (3774, 24), (4096, 1), (2500, 17),
    (777, 256), (300, 40),
]


@pytest.mark.parametrize("Lp,S", CONT_CASES)
def test_continue_bf16_vs_oracle_and_prefill(Lp, S):
    """Claim 1 on the GPU: continuation rows equal full-prefill rows L_prefix.. (and the oracle)."""
    say("continue bf16 32/8/128 Lp=%d S=%d" % (Lp, S))
    sh = W.QWEN
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=7 + Lp)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=n + 3) if Lp > 0 else (None, None, None, None)
    if d is None:
        d = kvr.make_desc(32, 8, 128, torch.bfloat16, 0)
    cont = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    claim1(cont, full[Lp:])
    kc_o = k[:Lp].transpose(0, 1).contiguous() if Lp else torch.zeros((8, 0, 128), dtype=torch.bfloat16)
    vc_o = v[:Lp].transpose(0, 1).contiguous() if Lp else torch.zeros((8, 0, 128), dtype=torch.bfloat16)
    want, _ = ref.continue_(q[Lp:], k[Lp:], v[Lp:], kc_o, vc_o, Lp)
    assert maxabs(cont, want) <= TOL[torch.bfloat16]


@pytest.mark.parametrize("Hq,Hkv,Lp,S", [
    (8, 8, 900, 50), (16, 8, 2000, 40), (64, 8, 1500, 9), (32, 8, 513, 10), (32, 8, 4159, 12), (8, 8, 70, 96),
])
def test_continue_group_sizes(Hq, Hkv, Lp, S):
    """Other GQA groups and row counts (33..96 rows per kv head, one or several
    column tiles per wave group, ragged prefixes): oracle and Claim 1."""
    say("continue bf16 %d/%d/128 Lp=%d S=%d" % (Hq, Hkv, Lp, S))
    sh = W.Shape(Hq, Hkv, 128, torch.bfloat16)
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=5 + Hq + Lp)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=n + 1)
    cont = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    claim1(cont, full[Lp:])
    want, _ = ref.continue_(q[Lp:], k[Lp:], v[Lp:], k[:Lp].transpose(0, 1).contiguous(),
                            v[:Lp].transpose(0, 1).contiguous(), Lp)
    assert maxabs(cont, want) <= TOL[torch.bfloat16]


@pytest.mark.parametrize("Lp,S", [(0, 5), (129, 16), (600, 33)])
def test_continue_fp32_vs_oracle(Lp, S):
    say("continue fp32 8/2/64 Lp=%d S=%d" % (Lp, S))
    sh = W.Shape(8, 2, 64, torch.float32)
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=11)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    if Lp:
        _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=n)
    else:
        kc = vc = None
        d = kvr.make_desc(8, 2, 64, torch.float32, 0)
    cont = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    want, _ = ref.prefill(q, k, v, rows=list(range(Lp, n)))
    assert maxabs(cont, want) <= TOL[torch.float32]
    assert float((cont - full[Lp:]).abs().max()) <= CLAIM1_TOL


# ------------------------------------------------------------ stress inputs
@pytest.mark.parametrize("kind", ["scaled", "sink", "tile_end", "rising"])
def test_stress_softmax(kind):
    """Peaky rows that force the online softmax to rescale, prefill and split continuation."""
    say("stress %s" % kind)
    sh = W.QWEN
    Lp, S = 1500, 24
    n = Lp + S
    q, k, v = W.stress(kind, n, sh, seed=3)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=n)
    cont = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    rows = list(range(0, 70)) + list(range(700, 760)) + list(range(Lp - 3, n))
    want, _ = ref.prefill(q, k, v, rows=rows)
    # Peaky rows have outputs of magnitude up to ~8, where rounding the output
    # to bf16 alone moves it by up to |x| * 2^-8: the absolute bars get that
    # allowance on top (and one bf16 ulp, |x| * 2^-7, between two GPU results).
    excess(full[rows], want, TOL[torch.bfloat16], 2.0 ** -8)
    excess(cont, want[-S:], TOL[torch.bfloat16], 2.0 ** -8)
    # Claim 1 between two GPU results at the plain bar (2e-3 and one output
    # ulp): a tile that holds a significant share of a row's weight and a new
    # maximum moves the reference to that maximum exactly, so a dominant key's
    # weight is 1 and never rounded in P.
    claim1(cont, full[Lp:])


def excess(gpu, want, tol, rel):
    """Assert |gpu - want| <= tol + rel * |want| elementwise."""
    got = gpu.float().cpu().numpy().astype(np.float64)
    bound = tol + rel * np.abs(want)
    worst = float(np.max(np.abs(got - want) - bound))
    assert worst <= 0.0, worst


# ------------------------------------------------------------- invariants
def test_cache_exact_and_canaries():
    """prefill(L) + append(S) leaves the same cache bits as prefill(L+S); other rows untouched."""
    say("cache exactness")
    sh = W.QWEN
    L, S, cap = 300, 37, 400
    q, k, v = W.qkv(L + S, sh, seed=5)
    canary = torch.full((8, cap, 128), -7.25, dtype=torch.bfloat16, device=DEV)
    kc1, vc1 = canary.clone(), canary.clone()
    gpu_prefill(sh, q, k, v, capacity=cap, kc=kc1, vc=vc1)
    kc2, vc2 = canary.clone(), canary.clone()
    _, _, _, d = gpu_prefill(sh, q[:L], k[:L], v[:L], capacity=cap, kc=kc2, vc=vc2)
    ks, vs = dev(k[L:], v[L:])
    kvr.kvr_cache_append(d, ks, vs, S, kc2, vc2, L)
    torch.cuda.synchronize()
    assert torch.equal(kc1, kc2) and torch.equal(vc1, vc2)
    assert torch.equal(kc1[:, :L + S].cpu(), k.transpose(0, 1))
    assert bool((kc1[:, L + S:] == -7.25).all()) and bool((vc1[:, L + S:] == -7.25).all())


def test_decode_chain():
    """T steps of continue(S=1) + append reproduce prefill rows L..L+T-1."""
    say("decode chain")
    sh = W.QWEN
    L, T = 700, 10
    q, k, v = W.qkv(L + T, sh, seed=9)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:L], k[:L], v[:L], capacity=L + T)
    outs = []
    for t in range(T):
        p = L + t
        o = gpu_continue(d, q[p:p + 1], k[p:p + 1], v[p:p + 1], kc, vc, p)
        ks, vs = dev(k[p:p + 1], v[p:p + 1])
        kvr.kvr_cache_append(d, ks, vs, 1, kc, vc, p)
        outs.append(o)
    torch.cuda.synchronize()
    chain = torch.cat(outs)
    claim1(chain, full[L:])
    want, _ = ref.prefill(q, k, v, rows=list(range(L, L + T)))
    assert maxabs(chain, want) <= TOL[torch.bfloat16]


def test_many_readers_batched():
    """64 readers of one cached 3774-token prefix, suffixes U[24, 256] (the
    many-readers workload at full size), in one call: every row of every reader
    against the oracle."""
    say("many readers: 64 over a cached 3774-token prefix")
    sh = W.QWEN
    Lp = W.READERS_L
    lens = W.reader_lengths(n=W.READERS_N, seed=0)
    cu = W.cu_seqlens(lens)
    total = cu[-1]
    g = W.gen(21)
    qp, kp, vp = W.qkv(Lp, sh, generator=g)
    qs, ks, vs = W.qkv(total, sh, generator=g)
    _, kc, vc, d = gpu_prefill(sh, qp, kp, vp, capacity=Lp)
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.empty_like(qd)
    kvr.kvr_continue_batched(d, qd, kd, vd, cu, kc, vc, Lp, out, kvr.workspace_for(d, Lp, total, len(lens)))
    torch.cuda.synchronize()
    got = out.cpu()
    kc_o, vc_o = kp.transpose(0, 1).contiguous(), vp.transpose(0, 1).contiguous()
    worst = 0.0
    for r in range(W.READERS_N):
        a, b = cu[r], cu[r + 1]
        want, _ = ref.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp)
        err = maxabs(got[a:b], want)
        worst = max(worst, err)
        assert err <= TOL[torch.bfloat16], (r, err)
    say("  readers max |gpu - oracle| = %.5f" % worst)
    # each reader equals its own single continuation (rounding only)
    for r in (0, 17, 63):
        a, b = cu[r], cu[r + 1]
        single = gpu_continue(d, qs[a:b], ks[a:b], vs[a:b], kc, vc, Lp)
        torch.cuda.synchronize()
        claim1(single, out[a:b])


def test_shifted_failure_mode():
    """Dropping the prefix (positions restarted) is far outside tolerance: the mask is live."""
    say("shifted negative")
    sh = W.QWEN
    Lp, S = 500, 24
    q, k, v = W.qkv(Lp + S, sh, seed=13)
    _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=Lp + S)
    good = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    shifted = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, 0)
    torch.cuda.synchronize()
    assert float((good - shifted).abs().max()) > 0.05


def test_causality_and_determinism():
    say("causality / determinism")
    sh = W.QWEN
    L, t = 400, 150
    q, k, v = W.qkv(L, sh, seed=17)
    a, _, _, _ = gpu_prefill(sh, q, k, v)
    a2, _, _, _ = gpu_prefill(sh, q, k, v)
    k2, v2 = k.clone(), v.clone()
    k2[t:] = -k2[t:] * 3
    v2[t:] = v2[t:] + 5
    b, _, _, _ = gpu_prefill(sh, q, k2, v2)
    torch.cuda.synchronize()
    assert torch.equal(a, a2)
    assert torch.equal(a[:t], b[:t])
    assert float((a[t:] - b[t:]).abs().max()) > 0.1
    # continuation with a key split is reproducible bit for bit
    _, kc, vc, d = gpu_prefill(sh, q[:300], k[:300], v[:300], capacity=L)
    c1 = gpu_continue(d, q[300:], k[300:], v[300:], kc, vc, 300)
    c2 = gpu_continue(d, q[300:], k[300:], v[300:], kc, vc, 300)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)


def test_closed_forms_on_gpu():
    """V = 1 gives 1; V[:, g] = g gives the kv-head index; Q = 0 gives the causal running mean."""
    say("closed forms")
    for dtype in (torch.bfloat16, torch.float32):
        sh = W.Shape(32, 8, 128, dtype)
        L = 260
        q, k, v = W.qkv(L, sh, seed=19)
        ones = torch.ones_like(v)
        o1, _, _, _ = gpu_prefill(sh, q, k, ones)
        gidx = torch.arange(8, dtype=torch.float32).view(1, 8, 1).expand(L, 8, 128).to(dtype).contiguous()
        o2, _, _, _ = gpu_prefill(sh, q, k, gidx)
        o3, _, _, _ = gpu_prefill(sh, torch.zeros_like(q), k, v)
        torch.cuda.synchronize()
        tol = TOL[dtype]
        assert float((o1.float() - 1).abs().max()) <= tol
        heads = (torch.arange(32) // 4).view(1, 32, 1).float().to(DEV)
        assert float((o2.float() - heads).abs().max()) <= tol * 4   # values up to 7
        mean = torch.cumsum(v.double(), 0) / torch.arange(1, L + 1, dtype=torch.float64).view(L, 1, 1)
        mean = mean.repeat_interleave(4, dim=1)
        assert float((o3.double().cpu() - mean).abs().max()) <= tol


# ------------------------------------------------- full-size workloads, sampled
def sampled_prefill_rows(n, seed):
    """Rows of an n-token prefill checked against the oracle at full size: the
    first and last 128, every 64-token tile boundary +-1 (the prefill's row
    tiles hold 64 tokens of a kv group, its key tiles 64 keys), and 256 drawn
    at random; the last 128 include the ragged last tile."""
    rows = set(range(min(128, n))) | set(range(max(0, n - 128), n))
    for b in range(64, n, 64):
        rows |= {b - 1, b, b + 1}
    rows |= set(np.random.default_rng(seed).integers(0, n, 256).tolist())
    return sorted(r for r in rows if 0 <= r < n)


@pytest.mark.parametrize("L", [3774, 16384, 32768])
def test_full_size_sampled(L):
    """The layer workloads at full size: continuation rows all checked, prefill
    rows sampled (first/last 128, every tile boundary +-1, 256 random)."""
    S = 24
    n = L + S
    say("full size L=%d S=%d" % (L, S))
    sh = W.QWEN
    q, k, v = W.qkv(n, sh, seed=0)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:L], k[:L], v[:L], capacity=n)
    cont = gpu_continue(d, q[L:], k[L:], v[L:], kc, vc, L)
    torch.cuda.synchronize()
    assert float((cont - full[L:]).abs().max()) <= CLAIM1_TOL
    rows = sampled_prefill_rows(n, L)
    say("  %d prefill rows against the oracle" % len(rows))
    want, _ = ref.prefill(q, k, v, rows=rows)
    assert maxabs(full[rows], want) <= TOL[torch.bfloat16]
    want_c, _ = ref.prefill(q, k, v, rows=list(range(L, n)))
    assert maxabs(cont, want_c) <= TOL[torch.bfloat16]


@pytest.mark.parametrize("Hq,Hkv,Lp,S", [(8, 2, 3000, 5), (16, 2, 2500, 3), (8, 2, 4100, 24)])
def test_continue_head_dim_64_split(Hq, Hkv, Lp, S):
    """head_dim 64 continuations whose split plan has several key splits (the
    merge's 4-rows-per-workgroup geometry): oracle and Claim 1."""
    say("continue bf16 %d/%d/64 Lp=%d S=%d" % (Hq, Hkv, Lp, S))
    sh = W.Shape(Hq, Hkv, 64, torch.bfloat16)
    n = Lp + S
    q, k, v = W.qkv(n, sh, seed=31 + Lp)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:Lp], k[:Lp], v[:Lp], capacity=n)
    assert kvr.kvr_workspace_bytes(d, Lp, S) > 0     # the plan splits the prefix
    cont = gpu_continue(d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp)
    torch.cuda.synchronize()
    claim1(cont, full[Lp:])
    want, _ = ref.continue_(q[Lp:], k[Lp:], v[Lp:], k[:Lp].transpose(0, 1).contiguous(),
                            v[:Lp].transpose(0, 1).contiguous(), Lp)
    assert maxabs(cont, want) <= TOL[torch.bfloat16]


# ------------------------------------- prefixes just past a round length (split plan)
@pytest.mark.parametrize("L,S", [(32768 + 5, 1), (32768 + 30, 1), (32768 + 5, 24), (32768 + 3, 12), (16384 + 3, 24),
                                 (16384 + 7, 1)])
def test_prefix_just_past_round_length(L, S):
    """Prefixes a few keys past a multiple of the split count x 128 keys: the last split
    takes the extra prefix keys with the new rows (the plan a decode chain hits on every
    step after the first).  Continuation and continuation + cache update against the
    oracle and against the GPU prefill rows; the updated cache rows are exact copies."""
    n = L + S
    say("prefix just past a round length L=%d S=%d" % (L, S))
    sh = W.QWEN
    q, k, v = W.qkv(n, sh, seed=L + S)
    full, _, _, _ = gpu_prefill(sh, q, k, v)
    _, kc, vc, d = gpu_prefill(sh, q[:L], k[:L], v[:L], capacity=n)
    cont = gpu_continue(d, q[L:], k[L:], v[L:], kc, vc, L)
    qs, ks, vs = dev(q[L:], k[L:], v[L:])
    out2 = torch.empty_like(qs)
    kvr.kvr_continue_append(d, qs, ks, vs, kc, vc, L, S, out2, kvr.workspace_for(d, L, S))
    torch.cuda.synchronize()
    assert torch.equal(cont, out2)
    assert torch.equal(kc[:, L:n].cpu(), k[L:].transpose(0, 1)) and torch.equal(vc[:, L:n].cpu(), v[L:].transpose(0, 1))
    assert float((cont - full[L:]).abs().max()) <= CLAIM1_TOL
    want, _ = ref.prefill(q, k, v, rows=list(range(L, n)))
    assert maxabs(cont, want) <= TOL[torch.bfloat16]

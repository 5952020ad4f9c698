"""The library under HIP-graph capture and on concurrent streams.

Every entry point enqueues kernels only (no allocation, no host sync, no
memset), so a captured sequence replays the very work of the eager calls.
The replays run several times with other eager work and synchronizations in
between, and each replay is compared with the eager result bit for bit.
"""
import pytest
import torch

from harness import workloads as W
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def test_graph_replay_matches_eager():
    say("graph replay: prefill + continuation + decode steps with the cache update")
    sh = W.QWEN
    Lp, S, T = 700, 24, 3
    n = Lp + S + T
    q, k, v = (x.to(DEV) for x in W.qkv(n, sh, seed=51))
    d = kvr.make_desc(32, 8, 128, torch.bfloat16, n)
    kc = torch.zeros((8, n, 128), dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    outp = torch.empty_like(q[:Lp])
    outc = torch.empty_like(q[Lp:Lp + S])
    outd = torch.empty_like(q[:T])
    ws = kvr.workspace_for(d, n, S)

    def work():
        kvr.kvr_prefill(d, q[:Lp], k[:Lp], v[:Lp], Lp, outp, kc, vc)
        kvr.kvr_continue_append(d, q[Lp:Lp + S], k[Lp:Lp + S], v[Lp:Lp + S], kc, vc, Lp, S, outc, ws)
        for t in range(T):
            p = Lp + S + t
            kvr.kvr_continue_append(d, q[p:p + 1], k[p:p + 1], v[p:p + 1], kc, vc, p, 1, outd[t:t + 1], ws)

    work()
    torch.cuda.synchronize()
    want = [x.clone() for x in (outp, outc, outd, kc, vc)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        work()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    for rep in range(3):
        for x in (outp, outc, outd, kc, vc):     # eager work between replays
            x.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, w in zip((outp, outc, outd, kc, vc), want):
            assert torch.equal(got, w), rep


def test_concurrent_streams():
    say("two streams at once")
    sh = W.QWEN
    jobs = []
    for seed, (Lp, S) in ((61, (2000, 24)), (62, (900, 1))):
        q, k, v = (x.to(DEV) for x in W.qkv(Lp + S, sh, seed=seed))
        d = kvr.make_desc(32, 8, 128, torch.bfloat16, Lp + S)
        kc = torch.zeros((8, Lp + S, 128), dtype=torch.bfloat16, device=DEV)
        vc = torch.zeros_like(kc)
        kvr.kvr_prefill(d, q[:Lp], k[:Lp], v[:Lp], Lp, torch.empty_like(q[:Lp]), kc, vc)
        out = torch.empty_like(q[Lp:])
        ws = kvr.workspace_for(d, Lp, S)
        jobs.append((d, q[Lp:], k[Lp:], v[Lp:], kc, vc, Lp, S, out, ws))
    torch.cuda.synchronize()
    serial = []
    for j in jobs:
        kvr.kvr_continue(*j)
        torch.cuda.synchronize()
        serial.append(j[8].clone())
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(5):
        for j in jobs:
            j[8].zero_()
        torch.cuda.synchronize()
        for s, j in zip(streams, jobs):
            s.wait_stream(torch.cuda.current_stream())
            for _ in range(3):
                kvr.kvr_continue(*j, stream=s)
        torch.cuda.synchronize()
        for j, w in zip(jobs, serial):
            assert torch.equal(j[8], w), rep

#!/usr/bin/env python3
"""Benchmark of the prefill / prefix-reuse attention path on one MI355X.

One step = one pass of the whole hot path over a Qwen3-4B-shaped attention
layer (32 query heads, 8 kv heads, head_dim 128, bf16, synthetic N(0,1)) at
the long context the targets are stated for:
  1. kvr_prefill           32792 tokens (attention + cache fill)      <- `value`
  2. kvr_continue          24 tokens over a cached 32768-token prefix
  3. kvr_continue          24 tokens over a cached 16384-token prefix
  4. kvr_cache_append      the 24 new K/V rows after the 32768-token prefix
  5. kvr_continue_batched  64 readers (S ~ U[24, 256]) of one cached
                           3774-token prefix
  6. decode step           kvr_continue_append(S=1) over 32768 cached rows
Every call is timed with HIP events on the stream it runs on.  The
continuations read caches from pools of >= 1 GiB (each step reads a cache
last touched several steps earlier), so the 256 MB last-level cache cannot
serve them.

After the timed steps, the length sweep (prefix 1024 / 4096 / 16384 / 32768,
S = 24, continuations graph-replayed over rotated caches), the 36-layer
decode chain (32768-token caches, 24 steps of S=1), 2..64 readers of the
3774-token prefix in one call against the same continuations one by one,
and a CPU-oracle baseline on a bounded sample of the 32792-token prefill are
measured.

Prints ONE JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefill attn TFLOP/s (%MFMA peak); continue GB/s (%HBM peak); reuse speedup"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E
ELT = 2


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-decode36", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-artifact", action="store_true")
    ap.add_argument("--no-rope", action="store_true")
    ap.add_argument("--no-readers-sweep", action="store_true")
    ap.add_argument("--readers-sweep-only", action="store_true",
                    help="only the 2..64-reader sweep (one JSON object)")
    ap.add_argument("--decode36-only", action="store_true",
                    help="only the 36-layer decode chain (one JSON object)")
    ap.add_argument("--no-model", action="store_true",
                    help="skip the random-weight 36-layer model (Table 1's prefill vs continuation step)")
    ap.add_argument("--model-only", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU-oracle sample time")
    ap.add_argument("--sweep-lengths", type=str, default=None,
                    help="comma-separated prefix lengths for the sweep (default: all four)")
    ap.add_argument("--sweep-suffix", type=int, default=None,
                    help="suffix length S of the sweep continuations (default 24)")
    ap.add_argument("--sweep-only", action="store_true",
                    help="skip the layer step (for profiling one sweep length)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run one plain 1 GiB device copy (reference for HBM byte counters)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from harness import accounting as A
    from harness import workloads as W
    from paper_2606_13361_amd import kvr

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    kvr.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    sh = W.QWEN
    Hq, Hkv, D = sh.n_q_heads, sh.n_kv_heads, sh.head_dim

    if args.copy_calibration:
        # a plain copy of known size: reads 1 GiB, writes 1 GiB
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # ---------------------------------------------------------------- inputs
    L32, L16, S = W.SWEEP_L[3], W.SWEEP_L[2], W.SWEEP_S
    n32, n16 = L32 + S, L16 + S
    q, k, v = W.qkv_device(n32, sh, seed=L32, device=dev)
    desc32 = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, n32 + 1)
    desc16 = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, n16 + 1)
    out_full = torch.empty_like(q)
    qs, ks, vs = q[L32:].contiguous(), k[L32:].contiguous(), v[L32:].contiguous()
    out_c32, out_c16 = torch.empty_like(qs), torch.empty_like(qs)
    ws32, ws16 = kvr.workspace_for(desc32, L32, S), kvr.workspace_for(desc16, L16, S)
    # cache pools of >= 1 GiB each: the prefill of step i fills pool32[i % R32];
    # the continuations of step i read caches last written R32 / 2 (R16) steps before
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)

    def pool(n_rows):
        cache_bytes = 2 * Hkv * n_rows * D * ELT
        R = max(2, -(-(1 << 30) // cache_bytes))
        pl = torch.empty((R, 2, Hkv, n_rows, D), dtype=torch.bfloat16, device=dev)
        for i in range(R):
            pl[i].copy_(torch.randn((2, Hkv, n_rows, D), generator=gen, device=dev))
        return pl, R
    pool32, R32 = pool(n32 + 1)
    pool16, R16 = pool(n16 + 1)
    # many readers of one 3774-token prefix
    Lr = W.READERS_L
    desc_r = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, Lr)
    kc_r = torch.randn((Hkv, Lr, D), generator=gen, device=dev).to(torch.bfloat16)
    vc_r = torch.randn((Hkv, Lr, D), generator=gen, device=dev).to(torch.bfloat16)
    lens = W.reader_lengths()
    cu = W.cu_seqlens(lens)
    rq, rk, rv = W.qkv_device(cu[-1], sh, seed=1, device=dev)
    rout = torch.empty_like(rq)
    ws_rd = kvr.workspace_for(desc_r, Lr, cu[-1], len(cu) - 1)
    dq, dk, dv = W.qkv_device(1, sh, seed=2, device=dev)
    dout = torch.empty_like(dq)
    ws_dec = kvr.workspace_for(desc32, L32, 1)

    names = ["prefill", "continue32k", "continue16k", "append", "readers", "decode_step"]

    def step(i, ev=None):
        def rec(j):
            if ev is not None:
                ev[j].record(stream)
        c_new = pool32[i % R32]
        c_old = pool32[(i + R32 // 2) % R32]
        c16 = pool16[i % R16]
        rec(0)
        kvr.kvr_prefill(desc32, q, k, v, n32, out_full, c_new[0], c_new[1])
        rec(1)
        kvr.kvr_continue(desc32, qs, ks, vs, c_old[0], c_old[1], L32, S, out_c32, ws32)
        rec(2)
        kvr.kvr_continue(desc16, qs, ks, vs, c16[0], c16[1], L16, S, out_c16, ws16)
        rec(3)
        kvr.kvr_cache_append(desc32, ks, vs, S, c_new[0], c_new[1], L32)
        rec(4)
        kvr.kvr_continue_batched(desc_r, rq, rk, rv, cu, kc_r, vc_r, Lr, rout, ws_rd)
        rec(5)
        kvr.kvr_continue_append(desc32, dq, dk, dv, c_old[0], c_old[1], L32, 1, dout, ws_dec)
        rec(6)

    if args.model_only:
        print(json.dumps({"model": model_table1(torch, A, W, dev)}), flush=True)
        return

    if args.decode36_only:
        print(json.dumps({"decode36": decode36(torch, kvr, A, W, dev, stream)}), flush=True)
        return

    if args.readers_sweep_only:
        print(json.dumps({"readers_sweep": readers_sweep(torch, kvr, A, W, dev, stream)}), flush=True)
        return

    if args.sweep_only:
        res = {"sweep": sweep(torch, kvr, A, W, dev, stream,
                              [int(x) for x in args.sweep_lengths.split(",")] if args.sweep_lengths
                              else list(W.SWEEP_L), args.sweep_suffix)}
        print(json.dumps(res), flush=True)
        return

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {nm: [] for nm in names}
    for ev in events:
        for j, nm in enumerate(names):
            per[nm].append(ev[j].elapsed_time(ev[j + 1]) * 1e-3)   # seconds
    avg = {nm: sum(v_) / len(v_) for nm, v_ in per.items()}
    med = {nm: sorted(v_)[len(v_) // 2] for nm, v_ in per.items()}

    pf_flops = A.prefill_flops(n32, Hq, D)
    pf_tflops = pf_flops / avg["prefill"] / 1e12
    c32_bytes = A.continue_bytes(L32, S, Hq, Hkv, D, ELT)
    c16_bytes = A.continue_bytes(L16, S, Hq, Hkv, D, ELT)
    c32_gbps = c32_bytes / avg["continue32k"] / 1e9
    c16_gbps = c16_bytes / avg["continue16k"] / 1e9
    rd_flops = A.batched_flops(Lr, lens, Hq, D)
    rd_tflops = rd_flops / avg["readers"] / 1e12
    dec_bytes = A.continue_bytes(L32, 1, Hq, Hkv, D, ELT) + A.append_bytes(1, Hkv, D, ELT)

    # parity spot check of this very run (Claim 1): the continuation over the
    # cache the last prefill wrote, against that prefill's rows
    last = pool32[(args.warmup + args.steps - 1) % R32]
    kvr.kvr_continue(desc32, qs, ks, vs, last[0], last[1], L32, S, out_c32, ws32)
    torch.cuda.synchronize()
    claim1 = float((out_c32 - out_full[L32:]).abs().max())

    result = {
        "metric": METRIC,
        "value": round(pf_tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: Q/K/V ~ N(0,1), seeded (no document text or weights)",
        "config": {
            "workload": "Qwen3-4B-shaped attention layer, 32 q heads / 8 kv heads / head_dim 128, bf16, "
                        "batch 1: prefill 32792 tokens (value); continue 24 tokens over cached 32768- and "
                        "16384-token prefixes; 64 readers (S ~ U[24,256]) of a cached 3774-token prefix; "
                        "one decode step over 32768",
            "prefill_tokens": n32, "prefix_tokens": [L32, L16], "suffix_tokens": S,
            "readers": len(lens), "reader_prefix": Lr, "reader_tokens": cu[-1],
            "global_batch": 1, "seq_len": n32,
        },
        "prefill_ms": round(avg["prefill"] * 1e3, 4),
        "prefill_tflops": round(pf_tflops, 2),
        "prefill_mfma_frac": round(pf_tflops / PEAK_BF16_TFLOPS, 4),
        "continue32k_us": round(avg["continue32k"] * 1e6, 2),
        "continue32k_GBps": round(c32_gbps, 1),
        "continue32k_hbm_frac": round(c32_gbps / PEAK_HBM_GBPS, 4),
        "continue16k_us": round(avg["continue16k"] * 1e6, 2),
        "continue16k_GBps": round(c16_gbps, 1),
        "continue16k_hbm_frac": round(c16_gbps / PEAK_HBM_GBPS, 4),
        "continue_caches": "pools of %d x 32768- and %d x 16384-token caches (>= 1 GiB each), read "
                           "several steps after they were last written" % (R32, R16),
        "reuse_speedup_32k": round(avg["prefill"] / avg["continue32k"], 2),
        "break_even_N_32k": round(A.break_even(avg["prefill"], avg["continue32k"]), 4),
        "append24_us": round(avg["append"] * 1e6, 2),
        "readers_ms": round(avg["readers"] * 1e3, 4),
        "readers_tflops": round(rd_tflops, 2),
        "readers_mfma_frac": round(rd_tflops / PEAK_BF16_TFLOPS, 4),
        "decode_step_us": round(avg["decode_step"] * 1e6, 2),
        "decode_step_GBps": round(dec_bytes / avg["decode_step"] / 1e9, 1),
        "decode_step_hbm_frac": round(dec_bytes / avg["decode_step"] / 1e9 / PEAK_HBM_GBPS, 4),
        "median_ms": {nm: round(med[nm] * 1e3, 4) for nm in names},
        "claim1_maxabs": claim1,
        "paper_context": "paper Table 1: full-model reuse 8.6-49.7x cheaper (Qwen3-4B fp16, Apple M1 Pro "
                         "MPS, one continuation step); not comparable hardware or scope",
    }
    # rooflines of the step's calls; `roofline` is the one that takes the most time
    digest = kernel_source_digest()
    traffic = measured_traffic(digest)

    def roof(call, kernel, bound, achieved, work, t):
        peak = PEAK_BF16_TFLOPS if bound == "mfma" else PEAK_HBM_GBPS
        return {"call": call, "kernel": kernel, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s" if bound == "mfma" else "GB/s", "frac": round(achieved / peak, 4),
                "work_per_launch": work, "avg_launch_ms": round(t * 1e3, 4), "traffic": traffic.get(call)}
    roofs = {
        "prefill": roof("prefill", "attn_pp_kernel<prefill>", "mfma", pf_tflops, pf_flops, avg["prefill"]),
        "continue32k": roof("continue32k", "attn_cont_kernel<3> + merge_bf16_kernel<128>", "hbm", c32_gbps,
                            c32_bytes, avg["continue32k"]),
        "continue16k": roof("continue16k", "attn_rows_kernel + merge_bf16_kernel<128>", "hbm", c16_gbps,
                            c16_bytes, avg["continue16k"]),
        "readers": roof("readers", "attn_pp_kernel<readers> + merge_bf16_kernel<128>", "mfma", rd_tflops, rd_flops,
                        avg["readers"]),
        "decode_step": roof("decode_step", "attn_cont_kernel<1> + merge_bf16_kernel<128>", "hbm",
                            dec_bytes / avg["decode_step"] / 1e9, dec_bytes, avg["decode_step"]),
    }
    dominant = max(roofs, key=lambda c: roofs[c]["avg_launch_ms"])
    result["roofline"] = roofs[dominant]
    result["rooflines"] = roofs
    result["kernel_source_digest"] = digest
    del pool32, pool16, q, k, v, out_full
    torch.cuda.empty_cache()

    if not args.no_sweep:
        lens_ = [int(x) for x in args.sweep_lengths.split(",")] if args.sweep_lengths else list(W.SWEEP_L)
        result["sweep"] = sweep(torch, kvr, A, W, dev, stream, lens_, args.sweep_suffix)
    if not args.no_decode36:
        result["decode36"] = decode36(torch, kvr, A, W, dev, stream)
    if not args.no_artifact:
        result["artifact"] = artifact(torch, kvr, W, dev, stream)
    if not args.no_rope:
        result["rope"] = rope_calls(torch, kvr, A, W, dev, stream)
    if not args.no_readers_sweep:
        result["readers_sweep"] = readers_sweep(torch, kvr, A, W, dev, stream)
    if not args.no_model:
        result["model"] = model_table1(torch, A, W, dev)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(W, A, args.cpu_seconds)
    print(json.dumps(result), flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_per_launch.md")


def kernel_source_digest():
    """Digest of every kernel source file: counter figures taken for other sources are stale."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2606_13361_amd", "csrc")
    h = hashlib.sha256()
    for fn in sorted(os.listdir(csrc)):
        if fn.endswith((".hip", ".hpp")):
            h.update(fn.encode())
            with open(os.path.join(csrc, fn), "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(digest):
    """HBM bytes per launch (FETCH + WRITE, calibrated) from the committed rocprofv3
    summary, keyed by kernel; empty when that summary was taken for other sources."""
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return {}
    if not any(ln.strip() == "source digest: " + digest for ln in lines):
        return {}
    out = {}
    for ln in lines:
        cells = [c.strip() for c in ln.strip().strip("|").split("|")]
        if len(cells) >= 5 and cells[0].startswith("`") and cells[-1].replace(".", "").isdigit():
            out[cells[0].strip("`")] = int(float(cells[-1]))
    return out


def graph_time(torch, stream, issue, n_calls, replays=5):
    """Seconds per call of `issue()` (which issues n_calls calls) captured in a HIP graph and replayed."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        issue()                       # warm up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        issue()
    g.replay()
    torch.cuda.synchronize()
    cur = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(cur)
    for _ in range(replays):
        g.replay()
    b.record(cur)
    torch.cuda.synchronize()
    del g
    return a.elapsed_time(b) * 1e-3 / (replays * n_calls)


def timed(torch, stream, fn, iters):
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(iters + 1)]
    ev[0].record(stream)
    for i in range(iters):
        fn(i)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) * 1e-3 for i in range(iters)]


def sweep(torch, kvr, A, W, dev, stream, lengths, suffix=None):
    """Prefill of L+24 vs continuation of 24 over L, L in {1024, 4096, 16384, 32768}, over
    the bf16 cache and over its int8 artifact; and one token (a decode step's attention)
    over both."""
    sh = W.QWEN
    Hq, Hkv, D = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    S = suffix or W.SWEEP_S
    rows = []
    for L in lengths:
        n = L + S
        q, k, v = W.qkv_device(n, sh, seed=L, device=dev)
        desc = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, n)
        out = torch.empty_like(q)
        kc = torch.empty((Hkv, n, D), dtype=torch.bfloat16, device=dev)
        vc = torch.empty_like(kc)
        reps = 5 if L >= 16384 else 20
        # warm up for at least 0.2 s of back-to-back calls: the engine clock
        # ramps over milliseconds under a sustained MFMA load, and a 2-8 ms
        # kernel timed right after two calls would be measured mid-ramp
        t_w = time.perf_counter()
        while True:
            kvr.kvr_prefill(desc, q, k, v, n, out, kc, vc)
            torch.cuda.synchronize()
            if time.perf_counter() - t_w >= 0.2:
                break
        tp = timed(torch, stream, lambda i: kvr.kvr_prefill(desc, q, k, v, n, out, kc, vc), reps)
        # continuation over R distinct caches (>= 1 GiB in total)
        cache_bytes = 2 * Hkv * n * D * 2
        R = max(2, -(-(1 << 30) // cache_bytes))
        pool = torch.randn((R, 2, Hkv, n, D), device=dev).to(torch.bfloat16)
        qs, ks, vs = q[L:].contiguous(), k[L:].contiguous(), v[L:].contiguous()
        oc = torch.empty_like(qs)
        ws = kvr.workspace_for(desc, L, S)
        iters = max(2 * R, 40)

        def cont(i):
            c = pool[i % R]
            kvr.kvr_continue(desc, qs, ks, vs, c[0], c[1], L, S, oc, ws)
        for i in range(R):
            cont(i)
        tc_eager = timed(torch, stream, cont, iters)
        # GPU time without host launch overhead: the R calls captured in one HIP
        # graph, replayed; the last replay's output must equal the eager one bit for bit
        cont(R - 1)
        torch.cuda.synchronize()
        ref_out = oc.clone()
        tc = graph_time(torch, stream, lambda: [cont(i) for i in range(R)], R)
        if not torch.equal(oc, ref_out):
            raise RuntimeError("graph replay of the continuation differs from the eager result")
        # the same continuation over int8 artifacts of the rotated caches (>= 1 GiB of artifacts)
        nb8 = kvr.kvr_q8_bytes(desc)
        R8 = max(2, -(-(1 << 30) // (2 * nb8)))
        arts = []
        for i in range(R8):
            kq, vq, sc = kvr.q8_artifact(desc)
            c = pool[i % R]
            kvr.kvr_quantize_cache(desc, c[0], c[1], L, kq, vq, sc)
            arts.append((kq, vq, sc))
        oc8 = torch.empty_like(qs)

        def cont8(i):
            kq, vq, sc = arts[i % R8]
            kvr.kvr_continue_q8(desc, qs, ks, vs, kq, vq, sc, L, S, oc8, ws)
        for i in range(R8):
            cont8(i)
        cont(0)
        cont8(0)
        torch.cuda.synchronize()
        q8_dev = float((oc8.float() - oc.float()).abs().max())   # int8 artifact vs bf16 cache, same inputs
        cont8(R8 - 1)
        torch.cuda.synchronize()
        ref8 = oc8.clone()
        tc8 = graph_time(torch, stream, lambda: [cont8(i) for i in range(R8)], R8)
        if not torch.equal(oc8, ref8):
            raise RuntimeError("graph replay of the int8 continuation differs from the eager result")
        # one token (a decode step's attention) over the same caches and artifacts
        q1, k1, v1 = q[L:L + 1].contiguous(), k[L:L + 1].contiguous(), v[L:L + 1].contiguous()
        o1, o18 = torch.empty_like(q1), torch.empty_like(q1)

        def dec(i):
            c = pool[i % R]
            kvr.kvr_continue(desc, q1, k1, v1, c[0], c[1], L, 1, o1, ws)

        def dec8(i):
            kq, vq, sc = arts[i % R8]
            kvr.kvr_continue_q8(desc, q1, k1, v1, kq, vq, sc, L, 1, o18, ws)
        for i in range(max(R, R8)):
            dec(i)
            dec8(i)
        td = graph_time(torch, stream, lambda: [dec(i) for i in range(R)], R)
        td8 = graph_time(torch, stream, lambda: [dec8(i) for i in range(R8)], R8)
        del pool, arts
        tp_avg = sum(tp) / len(tp)
        tc_avg = tc
        tce_avg = sum(tc_eager) / len(tc_eager)
        fl = A.prefill_flops(n, Hq, D)
        by = A.continue_bytes(L, S, Hq, Hkv, D, 2)
        rows.append({
            "L_prefix": L, "S": S,
            "prefill_ms": round(tp_avg * 1e3, 4),
            "prefill_tflops": round(fl / tp_avg / 1e12, 2),
            "prefill_mfma_frac": round(fl / tp_avg / 1e12 / PEAK_BF16_TFLOPS, 4),
            "continue_us": round(tc_avg * 1e6, 2),
            "continue_GBps": round(by / tc_avg / 1e9, 1),
            "continue_hbm_frac": round(by / tc_avg / 1e9 / PEAK_HBM_GBPS, 4),
            "continue_rotated_caches": R,
            "continue_eager_us": round(tce_avg * 1e6, 2),
            "continue_timing": "HIP-graph replay of %d rotated calls (eager: host-issued, one event pair per call)" % R,
            "reuse_speedup": round(tp_avg / tc_avg, 2),
            "break_even_N": round(A.break_even(tp_avg, tc_avg), 4),
            "continue_q8_us": round(tc8 * 1e6, 2),
            "continue_q8_GBps": round(A.continue_q8_bytes(L, S, Hq, Hkv, D) / tc8 / 1e9, 1),
            "q8_speedup_vs_bf16_cache": round(tc_avg / tc8, 3),
            "q8_maxabs_vs_bf16_cache": round(q8_dev, 5),
            "continue_q8_rotated_artifacts": R8,
            "decode_us": round(td * 1e6, 2),
            "decode_hbm_frac": round(A.continue_bytes(L, 1, Hq, Hkv, D, 2) / td / 1e9 / PEAK_HBM_GBPS, 4),
            "decode_q8_us": round(td8 * 1e6, 2),
            "q8_decode_speedup_vs_bf16_cache": round(td / td8, 3),
        })
        del q, k, v, out, kc, vc
        torch.cuda.empty_cache()
    return rows


def decode36(torch, kvr, A, W, dev, stream):
    """36 layers x 24 decode steps: continue(S=1) over 32768+t cached rows and the cache update."""
    sh = W.QWEN
    Hq, Hkv, D = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    Lz, T, NL = W.DECODE_L, W.DECODE_STEPS, W.DECODE_LAYERS
    cap = Lz + T
    desc = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, cap)
    g = torch.Generator(device=dev)
    g.manual_seed(36)
    caches = torch.empty((NL, 2, Hkv, cap, D), dtype=torch.bfloat16, device=dev)
    for l in range(NL):
        caches[l].copy_(torch.randn((2, Hkv, cap, D), generator=g, device=dev))
    qkv = torch.randn((T, NL, Hq + 2 * Hkv, D), generator=g, device=dev).to(torch.bfloat16)
    out = torch.empty((1, Hq, D), dtype=torch.bfloat16, device=dev)
    ws = kvr.workspace_for(desc, cap, 1)

    def chain(fused):
        def run():
            for t in range(T):
                for l in range(NL):
                    x = qkv[t, l]
                    qq = x[:Hq].unsqueeze(0)
                    kk = x[Hq:Hq + Hkv].unsqueeze(0)
                    vv = x[Hq + Hkv:].unsqueeze(0)
                    if fused:     # attention and the cache update in one call
                        kvr.kvr_continue_append(desc, qq, kk, vv, caches[l, 0], caches[l, 1], Lz + t, 1, out, ws)
                    else:
                        kvr.kvr_continue(desc, qq, kk, vv, caches[l, 0], caches[l, 1], Lz + t, 1, out, ws)
                        kvr.kvr_cache_append(desc, kk, vv, 1, caches[l, 0], caches[l, 1], Lz + t)
        return run

    run_chain = chain(True)
    run_chain()
    torch.cuda.synchronize()
    ts = timed(torch, stream, lambda i: run_chain(), 3)
    t_eager = sum(ts) / len(ts)
    # the whole chain (864 calls) as one HIP graph; then the same work as
    # separate continue and append calls
    t_graph = graph_time(torch, stream, run_chain, 1, replays=3)
    t_sep = graph_time(torch, stream, chain(False), 1, replays=3)
    t_avg = min(t_graph, t_eager)
    by = sum(A.continue_bytes(Lz + t, 1, Hq, Hkv, D, 2) + A.append_bytes(1, Hkv, D, 2)
             for t in range(T)) * NL
    res = {
        "layers": NL, "prefix": Lz, "steps": T,
        "chain_ms": round(t_avg * 1e3, 3),
        "chain_graph_ms": round(t_graph * 1e3, 3),
        "chain_eager_ms": round(t_eager * 1e3, 3),
        "chain_separate_update_ms": round(t_sep * 1e3, 3),
        "per_call_us": round(t_avg / (T * NL) * 1e6, 2),
        "GBps": round(by / t_avg / 1e9, 1),
        "hbm_frac": round(by / t_avg / 1e9 / PEAK_HBM_GBPS, 4),
        "resident_cache_GB": round(caches.numel() * 2 / 1e9, 3),
        "note": "kvr_continue_append per layer per step (the attention and its cache update in one call); "
                "chain_ms is the faster of one HIP-graph replay of the chain (chain_graph_ms) and host-issued "
                "launches (chain_eager_ms); chain_separate_update_ms: kvr_continue then kvr_cache_append, "
                "graph-replayed",
    }
    del caches, qkv
    torch.cuda.empty_cache()
    return res


def artifact(torch, kvr, W, dev, stream):
    """The 36-layer artifact of the 3774-token context (Alg. 1 save, Alg. 2 load):
    device <-> pinned host memory, one strided copy per layer and tensor."""
    sh = W.QWEN
    NL, L = W.QWEN_LAYERS, W.LAYER_L
    desc = kvr.make_desc(sh.n_q_heads, sh.n_kv_heads, sh.head_dim, torch.bfloat16, L + 24)
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    kcs = [torch.randn((sh.n_kv_heads, L + 24, sh.head_dim), generator=g, device=dev).to(torch.bfloat16)
           for _ in range(NL)]
    vcs = [torch.randn((sh.n_kv_heads, L + 24, sh.head_dim), generator=g, device=dev).to(torch.bfloat16)
           for _ in range(NL)]
    nb = kvr.kvr_artifact_bytes(desc, NL, L)
    host = torch.empty(nb, dtype=torch.uint8).pin_memory()
    k2 = [torch.empty_like(x) for x in kcs]
    v2 = [torch.empty_like(x) for x in vcs]
    kvr.kvr_artifact_save(desc, "qwen3-4b", kcs, vcs, L, host)
    kvr.kvr_artifact_load(desc, "qwen3-4b", host, k2, v2)
    torch.cuda.synchronize()
    ts = timed(torch, stream, lambda i: kvr.kvr_artifact_save(desc, "qwen3-4b", kcs, vcs, L, host), 3)
    tl = timed(torch, stream, lambda i: kvr.kvr_artifact_load(desc, "qwen3-4b", host, k2, v2), 3)
    exact = all(torch.equal(a[:, :L], b[:, :L]) for a, b in zip(kcs + vcs, k2 + v2))
    t_s, t_l = sorted(ts)[1], sorted(tl)[1]
    res = {
        "layers": NL, "tokens": L, "MB": round(nb / 1e6, 2),
        "save_ms": round(t_s * 1e3, 3), "save_GBps": round(nb / t_s / 1e9, 2),
        "load_ms": round(t_l * 1e3, 3), "load_GBps": round(nb / t_l / 1e9, 2),
        "round_trip_exact": exact,
        "note": "pinned host memory, device <-> host over the host link; the paper's C_load for "
                "this artifact (Table 1 row 3774 tokens: 557 MB)",
    }
    del kcs, vcs, k2, v2, host
    torch.cuda.empty_cache()
    return res


def readers_sweep(torch, kvr, A, W, dev, stream, counts=(2, 4, 8, 16, 32, 64)):
    """N readers (S ~ U[24, 256], seeded) of one cached 3774-token prefix in one
    kvr_continue_batched call, against the same N continuations issued one by
    one (kvr_continue, each with its own key-split plan); medians of 3 x 10
    calls, alternated so that both see the same clock."""
    sh = W.QWEN
    Hq, Hkv, D = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    L = W.READERS_L
    desc = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, L)
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    kc = torch.randn((Hkv, L, D), generator=g, device=dev).to(torch.bfloat16)
    vc = torch.randn((Hkv, L, D), generator=g, device=dev).to(torch.bfloat16)
    rows = []
    for n in counts:
        lens = W.reader_lengths(n=n, seed=0)
        cu = W.cu_seqlens(lens)
        q, k, v = (x.to(torch.bfloat16) for x in W.qkv_device(cu[-1], sh, seed=n, device=dev))
        out = torch.empty_like(q)
        ws = kvr.workspace_for(desc, L, cu[-1], n)
        parts = [(q[a:b], k[a:b], v[a:b], out[a:b], kvr.workspace_for(desc, L, b - a))
                 for a, b in zip(cu[:-1], cu[1:])]

        def batched():
            kvr.kvr_continue_batched(desc, q, k, v, cu, kc, vc, L, out, ws)

        def singles():
            for (qi, ki, vi, oi, wi) in parts:
                kvr.kvr_continue(desc, qi, ki, vi, kc, vc, L, qi.shape[0], oi, wi)

        for f in (batched, singles):
            for _ in range(3):
                f()
        torch.cuda.synchronize()
        tb, ts = [], []
        for _ in range(3):
            tb += timed(torch, stream, lambda i: batched(), 10)
            ts += timed(torch, stream, lambda i: singles(), 10)
        t_b, t_s = sorted(tb)[len(tb) // 2], sorted(ts)[len(ts) // 2]
        fl = A.batched_flops(L, lens, Hq, D)
        rows.append({"readers": n, "tokens": cu[-1], "ms": round(t_b * 1e3, 4),
                     "tflops": round(fl / t_b / 1e12, 1), "mfma_frac": round(fl / t_b / 1e12 / PEAK_BF16_TFLOPS, 4),
                     "key_split": ws is not None, "singles_ms": round(t_s * 1e3, 4),
                     "batched_speedup_vs_singles": round(t_s / t_b, 2)})
        del q, k, v, out, parts, ws
    del kc, vc
    torch.cuda.empty_cache()
    return rows


def rope_calls(torch, kvr, A, W, dev, stream):
    """The step's calls with fused RoPE (positions 0.. for the prefill, L.. for
    the continuations) next to the same calls without it, alternated in blocks
    so that both see the same clock."""
    sh = W.QWEN
    Hq, Hkv, D = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    L, S = W.LAYER_L, W.LAYER_S
    n = L + S
    q, k, v = (x.to(dev) for x in W.qkv(n, sh, seed=0))
    desc = kvr.make_desc(Hq, Hkv, D, torch.bfloat16, n + 1)
    lens = W.reader_lengths()
    cu = W.cu_seqlens(lens)
    tab = kvr.RopeTable(D, n + 1 + max(lens))
    kc, vc = (torch.zeros((Hkv, n + 1, D), dtype=torch.bfloat16, device=dev) for _ in range(2))
    kc2, vc2 = torch.zeros_like(kc), torch.zeros_like(vc)
    out, out_r = torch.empty_like(q), torch.empty_like(q)
    qs, ks, vs = q[L:].contiguous(), k[L:].contiguous(), v[L:].contiguous()
    oc, oc_r = torch.empty_like(qs), torch.empty_like(qs)
    ws, ws_r = kvr.workspace_for(desc, L, S), kvr.workspace_for_rope(desc, L, S)
    rq, rk, rv = (x.to(dev) for x in W.qkv(cu[-1], sh, seed=1))
    ro = torch.empty_like(rq)
    ws_rd = kvr.workspace_for_rope(desc, L, cu[-1], len(lens))
    ws_rp = kvr.workspace_for(desc, L, cu[-1], len(lens))
    dq, dk, dv = (x.to(dev) for x in W.qkv(1, sh, seed=2))
    do = torch.empty_like(dq)
    ws_d, ws_dr = kvr.workspace_for(desc, n, 1), kvr.workspace_for_rope(desc, n, 1)
    calls = {
        "prefill": (lambda: kvr.kvr_prefill(desc, q, k, v, n, out, kc, vc),
                    lambda: kvr.kvr_prefill_rope(desc, tab, q, k, v, n, out_r, kc2, vc2)),
        "continue": (lambda: kvr.kvr_continue(desc, qs, ks, vs, kc, vc, L, S, oc, ws),
                     lambda: kvr.kvr_continue_rope(desc, tab, qs, ks, vs, kc2, vc2, L, S, oc_r, ws_r)),
        "readers": (lambda: kvr.kvr_continue_batched(desc, rq, rk, rv, cu, kc, vc, L, ro, ws_rp),
                    lambda: kvr.kvr_continue_batched_rope(desc, tab, rq, rk, rv, cu, kc2, vc2, L, ro, ws_rd)),
        "decode_step": (lambda: (kvr.kvr_continue(desc, dq, dk, dv, kc, vc, n, 1, do, ws_d),
                                 kvr.kvr_cache_append(desc, dk, dv, 1, kc, vc, n)),
                        lambda: kvr.kvr_continue_rope(desc, tab, dq, dk, dv, kc2, vc2, n, 1, do, ws_dr,
                                                      append=True)),
    }
    res = {}
    for name, (plain, roped) in calls.items():
        for f in (plain, roped):          # warm the clock up
            t_end = time.perf_counter() + 0.1
            while time.perf_counter() < t_end:
                f()
                torch.cuda.synchronize()
        tp, tr = [], []
        for _ in range(4):
            tp += timed(torch, stream, lambda i: plain(), 10)
            tr += timed(torch, stream, lambda i: roped(), 10)
        res[name] = (sorted(tp)[len(tp) // 2], sorted(tr)[len(tr) // 2])
    kvr.kvr_prefill_rope(desc, tab, q, k, v, n, out_r, kc2, vc2)
    kvr.kvr_continue_rope(desc, tab, qs, ks, vs, kc2, vc2, L, S, oc_r, ws_r)
    torch.cuda.synchronize()
    pf = A.prefill_flops(n, Hq, D)
    rd = A.batched_flops(L, lens, Hq, D)
    r = {
        "what": "the layer step's calls with RoPE fused (rotation at positions 0.. / L..; base 1e6) next to "
                "the same calls without; medians of 40 timed calls each",
        "prefill_ms": [round(res["prefill"][0] * 1e3, 4), round(res["prefill"][1] * 1e3, 4)],
        "prefill_tflops": [round(pf / res["prefill"][0] / 1e12, 1), round(pf / res["prefill"][1] / 1e12, 1)],
        "continue_us": [round(res["continue"][0] * 1e6, 2), round(res["continue"][1] * 1e6, 2)],
        "readers_ms": [round(res["readers"][0] * 1e3, 4), round(res["readers"][1] * 1e3, 4)],
        "readers_tflops": [round(rd / res["readers"][0] / 1e12, 1), round(rd / res["readers"][1] / 1e12, 1)],
        "decode_step_us": [round(res["decode_step"][0] * 1e6, 2), round(res["decode_step"][1] * 1e6, 2)],
        "pairs": "[without RoPE, with RoPE]",
        "claim1_maxabs": float((oc_r - out_r[L:]).abs().max()),
    }
    del q, k, v, kc, vc, kc2, vc2, out, out_r, rq, rk, rv, ro
    torch.cuda.empty_cache()
    return r


TABLE1 = os.path.join(ROOT, "tests", "golden", "table1_qwen3_4b_m1pro.txt")


def model_table1(torch, A, W, dev, lengths=(255, 485, 945, 1888, 3774)):
    """The paper's Table 1 on this GPU with a random-weight Qwen3-4B-shaped
    model (36 layers, hidden 2560, MLP 9728, 32/8 heads of 128, tied 151936-row
    output embedding, bf16): a full prefill of the L-token context (the last
    row's logits included) against ONE continuation step of one token over the
    resident caches (its logits included)."""
    from paper_2606_13361_amd import kvr_model as M
    cfg = dict(M.QWEN3_4B)
    H = cfg["hidden"]
    Lmax = max(lengths)
    m = M.Model(cfg, cfg["layers"], Lmax + 1, seed=0, vocab=cfg["vocab"], max_tokens=Lmax, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(3)
    h_all = torch.randn((Lmax + 1, H), generator=g, device=dev).to(torch.bfloat16)
    paper = {}
    for ln in open(TABLE1):
        if ln.strip() and not ln.startswith("#"):
            t, pf, rs, _, sp = ln.split()
            paper[int(t)] = (float(pf), float(rs), float(sp))
    layer_params = (H * (cfg["n_q_heads"] + 2 * cfg["n_kv_heads"]) * cfg["head_dim"]
                    + cfg["n_q_heads"] * cfg["head_dim"] * H + 3 * H * cfg["intermediate"])
    weight_bytes = 2 * (cfg["layers"] * layer_params + cfg["vocab"] * H)
    rows = []
    cur = torch.cuda.current_stream()
    for L in lengths:
        hp = torch.empty((L, H), dtype=torch.bfloat16, device=dev)
        h1 = torch.empty((1, H), dtype=torch.bfloat16, device=dev)

        def prefill():
            hp.copy_(h_all[:L])
            m.forward(hp, 0)
            m.logits(hp)

        def step():
            h1.copy_(h_all[L:L + 1])
            m.forward(h1, L)
            m.logits(h1)

        for _ in range(2):
            prefill()
        torch.cuda.synchronize()
        tp = timed(torch, cur, lambda i: prefill(), 5)
        for _ in range(5):
            step()
        torch.cuda.synchronize()
        ts = timed(torch, cur, lambda i: step(), 20)
        # the same step replayed from a HIP graph (no host launch cost)
        side = torch.cuda.Stream()
        side.wait_stream(cur)
        with torch.cuda.stream(side):
            step()
        cur.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        graph.replay()
        torch.cuda.synchronize()
        tg = timed(torch, cur, lambda i: graph.replay(), 20)
        del graph
        t_p, t_s, t_g = sorted(tp)[len(tp) // 2], sorted(ts)[len(ts) // 2], sorted(tg)[len(tg) // 2]
        flops = (2 * L * layer_params * cfg["layers"] + 2 * H * cfg["vocab"]
                 + cfg["layers"] * A.prefill_flops(L, cfg["n_q_heads"], cfg["head_dim"]))
        step_bytes = weight_bytes + cfg["layers"] * A.kv_bytes_per_token(cfg["n_kv_heads"], cfg["head_dim"], 2) * (L + 1)
        pp = paper.get(L)
        rows.append({
            "tokens": L,
            "prefill_ms": round(t_p * 1e3, 3), "prefill_tflops": round(flops / t_p / 1e12, 1),
            "step_ms": round(t_s * 1e3, 3), "step_graph_ms": round(t_g * 1e3, 3),
            "step_graph_GBps": round(step_bytes / t_g / 1e9, 1),
            "speedup": round(t_p / t_g, 2),
            "paper_prefill_s": pp[0] if pp else None, "paper_step_s": pp[1] if pp else None,
            "paper_speedup": pp[2] if pp else None,
        })
    res = {
        "what": "random-weight Qwen3-4B-shaped model, bf16, 36 layers (RMSNorm, QKV / O / gate-up / down "
                "products, q/k norm + RoPE, this library's attention), tied 151936-row output embedding: "
                "full prefill of the context (last row's logits; products on hipBLASLt) vs one continuation "
                "step of one token over the resident caches (its logits; the library's one-row product "
                "kernels with the norms and the activation fused); medians of 5 prefills and 20 steps",
        "weights_GB": round(weight_bytes / 1e9, 3),
        "rows": rows,
        "paper_context": "paper Table 1: Qwen3-4B fp16 on Apple M1 Pro (MPS), speedup 8.6-49.7x; the speedup "
                         "here uses the graph-replayed step",
    }
    del m, h_all
    torch.cuda.empty_cache()
    return res


def host_cpu():
    """The host's logical CPUs, the ones this process may run on, the cgroup CPU
    quota (if any) and the CPU model."""
    info = {"host_logical_cpus": os.cpu_count()}
    try:
        info["affinity_cpus"] = len(os.sched_getaffinity(0))
    except AttributeError:
        info["affinity_cpus"] = os.cpu_count()
    try:
        quota, period = open("/sys/fs/cgroup/cpu.max").read().split()[:2]
        info["cgroup_cpu_quota"] = None if quota == "max" else round(int(quota) / int(period), 2)
    except (OSError, ValueError):
        info["cgroup_cpu_quota"] = None
    model = None
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    info["cpu_model"] = model
    return info


def cpu_baseline(W, A, target_s):
    """The fp64 oracle, as it stands, on a strided sample of the rows of the
    32792-token prefill (the `value` workload), timed on the host cores: every
    CPU of the affinity mask (median of 3 runs) and one thread (median of 3, on
    a smaller sample).  Inputs are the same seeded bf16 values, drawn on the
    CPU, widened to fp64 once before timing."""
    import numpy as np
    from oracle import ref
    host = host_cpu()
    threads = max(1, host["affinity_cpus"] or 1)
    sh = W.QWEN
    n = W.SWEEP_L[3] + W.SWEEP_S
    Hq, D = sh.n_q_heads, sh.head_dim
    q, k, v = W.qkv(n, sh, seed=0)
    q, k, v = (ref._f64(x) for x in (q, k, v))

    def flops(rows):
        return sum(4 * Hq * D * (r + 1) for r in rows)

    def sample(rate, seconds):
        step = max(1, int(A.prefill_flops(n, Hq, D) / max(rate * seconds, 1.0)))
        return list(range(step // 2, n, step)), step

    def run(rows, nth):
        t0 = time.perf_counter()
        ref.prefill(q, k, v, rows=rows, nthreads=nth)
        return time.perf_counter() - t0

    res = {}
    for label, nth, secs in (("all", threads, target_s / 3.0), ("one", 1, target_s / 6.0)):
        probe = list(range(n - 1, 0, -n // (min(2 * nth, 64) + 2)))[:min(2 * nth, 64)]
        rate = flops(probe) / max(run(probe, nth), 1e-3)
        rows, step = sample(rate, secs)
        ts = sorted(run(rows, nth) for _ in range(3))
        res[label] = (flops(rows) / ts[1] / 1e12, rows, step, ts)
    v_all, rows, step, ts = res["all"]
    v_one, rows1, step1, ts1 = res["one"]
    return {
        "value": round(v_all, 6),
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "fp64 oracle prefill rows %d..%d step %d (%d of %d rows, all 32 heads) of the 32792-token "
                  "layer, median of 3 runs of %.1f-%.1f s on %d threads" % (rows[0], rows[-1], step, len(rows), n,
                                                                             ts[0], ts[2], threads),
        "single_thread_value": round(v_one, 6),
        "single_thread_sample": "rows step %d (%d rows), median of 3 runs of %.1f-%.1f s" % (
            step1, len(rows1), ts1[0], ts1[2]),
        "host": host,
    }


if __name__ == "__main__":
    main()

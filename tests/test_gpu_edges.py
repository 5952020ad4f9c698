"""GPU edge cases across entry points, against the fp64 oracles.

* more readers than one launch's segment table holds (128): the host splits
  them into groups of launches (and, with RoPE, groups of pre-pass launches),
  empty readers included, on every kernel family (two-group d = 128,
  register-staged d = 64, fp32);
* RoPE composed with the int8 artifact: rotated cache -> quantized artifact ->
  continuation whose rows were rotated at L_prefix.. by kvr_rope_apply;
* the decoder layer in fp16.
Bars as in the plain tests of each path (1e-2 bf16, 1e-5 fp32 against the
oracle; the layer's bars in test_gpu_model).
"""
import numpy as np
import pytest
import torch

from harness import workloads as W
from oracle import layer as LO
from oracle import quant as QO
from oracle import ref
from oracle import rope as ORope
from paper_2606_13361_amd import kvr

pytestmark = pytest.mark.gpu

DEV = "cuda"
TOL = {torch.bfloat16: 1e-2, torch.float32: 1e-5}


def say(msg):
    print(msg, flush=True)


def dev(*ts):
    return [t.to(DEV).contiguous() for t in ts]


def maxabs(gpu, want):
    return float(np.max(np.abs(gpu.double().cpu().numpy() - want))) if want.size else 0.0


def many_lengths(n, seed):
    g = torch.Generator()
    g.manual_seed(seed)
    lens = torch.randint(0, 10, (n,), generator=g).tolist()
    lens[0], lens[128], lens[n - 1] = 0, 0, 9          # empty readers at group edges
    return lens


def prefill(sh, q, k, v, cap):
    d = kvr.make_desc(sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.dtype, cap)
    qd, kd, vd = dev(q, k, v)
    out = torch.empty_like(qd)
    kc = torch.zeros((sh.n_kv_heads, cap, sh.head_dim), dtype=sh.dtype, device=DEV)
    vc = torch.zeros_like(kc)
    kvr.kvr_prefill(d, qd, kd, vd, q.shape[0], out, kc, vc)
    return kc, vc, d


@pytest.mark.parametrize("Hq,Hkv,D,dt", [(32, 8, 128, torch.bfloat16), (8, 2, 64, torch.bfloat16),
                                         (4, 2, 64, torch.float32)])
def test_readers_beyond_one_launch(Hq, Hkv, D, dt):
    say("300 readers %d/%d/%d %s" % (Hq, Hkv, D, dt))
    sh = W.Shape(Hq, Hkv, D, dt)
    Lp, n = 500, 300
    lens = many_lengths(n, D)
    cu = W.cu_seqlens(lens)
    g = W.gen(D + 1)
    qp, kp, vp = W.qkv(Lp, sh, generator=g)
    qs, ks, vs = W.qkv(cu[-1], sh, generator=g)
    kc, vc, d = prefill(sh, qp, kp, vp, Lp)
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.full_like(qd, float("nan"))
    kvr.kvr_continue_batched(d, qd, kd, vd, cu, kc, vc, Lp, out, kvr.workspace_for(d, Lp, cu[-1], n))
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()                   # every row of every reader written
    kc_o, vc_o = kp.transpose(0, 1).contiguous(), vp.transpose(0, 1).contiguous()
    for r in list(range(0, n, 7)) + [127, 128, 129, 255, 256, n - 1]:
        a, b = cu[r], cu[r + 1]
        if a == b:
            continue
        want, _ = ref.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp)
        assert maxabs(out[a:b], want) <= TOL[dt], r


def test_readers_rope_beyond_one_launch():
    say("300 readers with RoPE")
    sh = W.Shape(32, 8, 128, torch.bfloat16)
    Lp, n = 400, 300
    lens = many_lengths(n, 3)
    cu = W.cu_seqlens(lens)
    tab = kvr.RopeTable(128, Lp + 9)
    g = W.gen(4)
    qp, kp, vp = W.qkv(Lp, sh, generator=g)
    qs, ks, vs = W.qkv(cu[-1], sh, generator=g)
    d = kvr.make_desc(32, 8, 128, torch.bfloat16, Lp)
    qd, kd, vd = dev(qp, kp, vp)
    kc = torch.zeros((8, Lp, 128), dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    kvr.kvr_prefill_rope(d, tab, qd, kd, vd, Lp, torch.empty_like(qd), kc, vc)
    qd, kd, vd = dev(qs, ks, vs)
    out = torch.full_like(qd, float("nan"))
    kvr.kvr_continue_batched_rope(d, tab, qd, kd, vd, cu, kc, vc, Lp, out,
                                  kvr.workspace_for_rope(d, Lp, cu[-1], n))
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()
    k_rot = ORope.round_to(ORope.rotate(kp, np.arange(Lp), ORope.QWEN3_BASE), "bf16")
    kc_o = np.transpose(k_rot, (1, 0, 2)).copy()
    vc_o = vp.transpose(0, 1).contiguous()
    for r in list(range(0, n, 11)) + [127, 128, 129, n - 1]:
        a, b = cu[r], cu[r + 1]
        if a == b:
            continue
        want, _, _ = ORope.continue_(qs[a:b], ks[a:b], vs[a:b], kc_o, vc_o, Lp, ORope.QWEN3_BASE, fmt="bf16")
        assert maxabs(out[a:b], want) <= TOL[torch.bfloat16], r


def test_rope_with_int8_artifact():
    """A rotated cache quantized into the int8 artifact, continued by rows
    rotated at L_prefix.. (kvr_rope_apply), against the oracle's rotate ->
    round -> quantize -> continue."""
    say("RoPE + int8 artifact")
    sh = W.Shape(32, 8, 128, torch.bfloat16)
    Lp, S = 2000, 24
    n = Lp + S
    tab = kvr.RopeTable(128, n)
    q, k, v = W.qkv(n, sh, seed=8)
    d = kvr.make_desc(32, 8, 128, torch.bfloat16, n)
    qd, kd, vd = dev(q[:Lp], k[:Lp], v[:Lp])
    kc = torch.zeros((8, n, 128), dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    kvr.kvr_prefill_rope(d, tab, qd, kd, vd, Lp, torch.empty_like(qd), kc, vc)
    kq, vq, sc = kvr.q8_artifact(d)
    kvr.kvr_quantize_cache(d, kc, vc, Lp, kq, vq, sc)
    qs, ks, vs = dev(q[Lp:], k[Lp:], v[Lp:])
    qr = kvr.kvr_rope_apply(d, tab, qs, Lp, torch.empty_like(qs))
    kr = kvr.kvr_rope_apply(d, tab, ks, Lp, torch.empty_like(ks))
    out = torch.empty_like(qs)
    kvr.kvr_continue_q8(d, qr, kr, vs, kq, vq, sc, Lp, S, out, kvr.workspace_for(d, Lp, S))
    torch.cuda.synchronize()
    base = ORope.QWEN3_BASE
    k_rot = ORope.round_to(ORope.rotate(k[:Lp], np.arange(Lp), base), "bf16")
    kc_o = np.zeros((8, n, 128))
    kc_o[:, :Lp] = np.transpose(k_rot, (1, 0, 2))
    vc_o = np.zeros((8, n, 128))
    vc_o[:, :Lp] = v[:Lp].double().transpose(0, 1).numpy()
    k_codes, v_codes, sk, sv = QO.quantize_cache(kc_o, vc_o, Lp)
    pos = Lp + np.arange(S)
    qro = ORope.round_to(ORope.rotate(q[Lp:], pos, base), "bf16")
    kro = ORope.round_to(ORope.rotate(k[Lp:], pos, base), "bf16")
    want, _ = QO.continue_q8(qro, kro, v[Lp:], k_codes, v_codes, sk, sv, Lp)
    assert maxabs(out, want) <= TOL[torch.bfloat16]


def test_layer_fp16():
    """The decoder layer in fp16 (prefill, then a one-token step) against the
    layer oracle rounding every held tensor to fp16."""
    from paper_2606_13361_amd import kvr_model as M
    say("layer fp16")
    cfg = dict(M.QWEN3_4B)
    F = torch.float16
    Lp = 40
    n = Lp + 1
    g = torch.Generator(device=DEV)
    g.manual_seed(12)
    W_ = M.random_layer(cfg, F, g)
    h = torch.randn((n, cfg["hidden"]), generator=g, device=DEV).to(F)
    d = kvr.make_desc(32, 8, 128, F, n)
    kc = torch.zeros((8, n, 128), dtype=F, device=DEV)
    vc = torch.zeros_like(kc)
    tab = kvr.RopeTable(128, n, cfg["base"])
    blas = M.Blas()
    ws = torch.empty(M.kvr_layer_workspace_bytes(d, cfg, n, n), dtype=torch.uint8, device=DEV)
    hp, hs = h[:Lp].clone(), h[Lp:].clone()
    M.kvr_layer_forward(d, cfg, W_, tab, blas, hp, Lp, 0, kc, vc, ws)
    M.kvr_layer_forward(d, cfg, W_, tab, blas, hs, 1, Lp, kc, vc, ws)
    torch.cuda.synchronize()
    Wo = {k_: v_.double().cpu().numpy() for k_, v_ in W_.items()}
    hn = h.double().cpu().numpy()
    want_p, k_p, v_p = LO.layer(hn[:Lp], Wo, cfg, None, None, 0, fmt="fp16")
    kco = np.zeros((8, n, 128))
    vco = np.zeros_like(kco)
    kco[:, :Lp] = np.transpose(k_p, (1, 0, 2))
    vco[:, :Lp] = np.transpose(v_p, (1, 0, 2))
    want_s, _, _ = LO.layer(hn[Lp:], Wo, cfg, kco, vco, Lp, fmt="fp16")
    for got, want, name in ((hp, want_p, "prefill"), (hs, want_s, "step")):
        err = np.abs(got.double().cpu().numpy() - want)
        nrms = float(np.sqrt(np.mean(err ** 2)) / np.sqrt(np.mean(want ** 2)))
        say("  %s: max |d| %.3g, normalized rms %.3g" % (name, float(err.max()), nrms))
        # fp16 keeps three more bits than bf16: the layer's bars, a quarter of the ulp terms
        assert np.all(err <= 2.0 ** -8 * np.abs(want) + 1e-2), name
        assert nrms <= 2.0 ** -9, name

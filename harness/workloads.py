"""Seeded synthetic inputs with the shapes of the paper's workloads.

The paper measures Qwen3-4B on real documents of 255..3774 tokens (Table 1;
8 KV heads of width 128, Section "Artifact size").  Neither the weights nor
the documents are available, and attention cost does not depend on the data,
so Q/K/V are drawn i.i.d. N(0, 1) from a seeded CPU generator (fp32 draws in
the order Q, K, V, then rounded to the storage dtype).  The very same bits are
handed to the GPU and, widened exactly, to the oracle.

This module draws numbers only; it computes no attention.
"""
from dataclasses import dataclass

import torch

# Qwen3-4B-style attention layer: 32 query heads, 8 KV heads, head_dim 128.
QWEN_HQ, QWEN_HKV, QWEN_D = 32, 8, 128
QWEN_LAYERS = 36


@dataclass(frozen=True)
class Shape:
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: torch.dtype

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads


TINY = Shape(2, 1, 64, torch.float32)
QWEN = Shape(QWEN_HQ, QWEN_HKV, QWEN_D, torch.bfloat16)

# Workloads (prefix length L, suffix length S).
TINY_L, TINY_S = 128, 16
LAYER_L, LAYER_S = 3774, 24
SWEEP_L = (1024, 4096, 16384, 32768)
SWEEP_S = 24
READERS_N, READERS_L, READERS_SMIN, READERS_SMAX = 64, 3774, 24, 256
DECODE_LAYERS, DECODE_L, DECODE_STEPS = 36, 32768, 24


def gen(seed):
    g = torch.Generator()
    g.manual_seed(seed)
    return g


def qkv(n_tokens, shape, seed=0, generator=None):
    """Q [n,Hq,d], K [n,Hkv,d], V [n,Hkv,d] on the CPU, drawn N(0,1) in the order Q, K, V."""
    g = generator if generator is not None else gen(seed)
    q = torch.randn((n_tokens, shape.n_q_heads, shape.head_dim), generator=g)
    k = torch.randn((n_tokens, shape.n_kv_heads, shape.head_dim), generator=g)
    v = torch.randn((n_tokens, shape.n_kv_heads, shape.head_dim), generator=g)
    return q.to(shape.dtype), k.to(shape.dtype), v.to(shape.dtype)


def qkv_device(n_tokens, shape, seed, device):
    """Large inputs drawn on the device with a seeded device generator (bench sizes)."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    q = torch.randn((n_tokens, shape.n_q_heads, shape.head_dim), generator=g, device=device)
    k = torch.randn((n_tokens, shape.n_kv_heads, shape.head_dim), generator=g, device=device)
    v = torch.randn((n_tokens, shape.n_kv_heads, shape.head_dim), generator=g, device=device)
    return q.to(shape.dtype), k.to(shape.dtype), v.to(shape.dtype)


def reader_lengths(n=READERS_N, lo=READERS_SMIN, hi=READERS_SMAX, seed=0):
    """Suffix lengths of the many-readers workload, uniform on [lo, hi]."""
    return torch.randint(lo, hi + 1, (n,), generator=gen(seed)).tolist()


def cu_seqlens(lengths):
    cu = [0]
    for s in lengths:
        cu.append(cu[-1] + int(s))
    return cu


# ---------------------------------------------------------------- stress inputs
# N(0,1) inputs give nearly flat softmax rows.  These place large scores where
# an online softmax has to rescale: at the end of each key tile, rising across
# tiles, at the very first key, or everywhere (scores x8).

def stress(kind, n_tokens, shape, seed=0, tile=64):
    """Inputs whose softmax rows are far from flat.

    A per-kv-head unit direction u_g is added to every query of group g; keys
    get a multiple of u_g so that chosen keys score about +9 (in scaled units)
    above the N(0,1) background:
      "scaled"   -- all queries x8 (every score 8x wider);
      "sink"     -- key 0 is the large one;
      "tile_end" -- the last key of each tile, growing from tile to tile, so
                    every tile brings a new row maximum at its end;
      "rising"   -- a bump that grows linearly with the key index.
    """
    g = gen(seed + 7919)
    q, k, v = qkv(n_tokens, shape, seed)
    q32, k32 = q.float(), k.float()
    d = shape.head_dim
    u = torch.randn((shape.n_kv_heads, d), generator=g)
    u = u / u.norm(dim=1, keepdim=True)
    uq = u.repeat_interleave(shape.group, dim=0)            # [Hq, d]
    bump = 3.0 * (d ** 0.5)                                  # q.k/sqrt(d) ~ 3*3 = 9
    if kind == "scaled":
        q32 = q32 * 8.0
    elif kind == "sink":
        q32 = q32 + 3.0 * uq
        k32[0] = k32[0] + bump * u
    elif kind == "tile_end":
        q32 = q32 + 3.0 * uq
        for j in range(tile - 1, n_tokens, tile):
            k32[j] = k32[j] + bump * (1.0 + j / max(1, n_tokens)) * u
    elif kind == "rising":
        q32 = q32 + 3.0 * uq
        ramp = torch.linspace(0.0, 1.0, n_tokens).view(n_tokens, 1, 1)
        k32 = k32 + bump * ramp * u.unsqueeze(0)
    else:
        raise ValueError(kind)
    return q32.to(shape.dtype), k32.to(shape.dtype), v


def decode_step_inputs(generator, shape, n_layers):
    """Per-layer (q [1,Hq,d], k [1,Hkv,d], v [1,Hkv,d]) for one decode step, layer-major."""
    out = []
    for _ in range(n_layers):
        out.append(qkv(1, shape, generator=generator))
    return out

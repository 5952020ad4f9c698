"""Algorithmic work and cost-model accounting.

Counting conventions (algorithmic, never the executed work):

* FLOPs: 4 * n_q_heads * head_dim per visible (query, key) pair -- 2 for the
  score dot product, 2 for the value update.  exp is not counted, masked pairs
  and tile padding are not counted.
* Bytes of a continuation: the cached K and V rows that are read, the new
  Q/K/V rows and the output.  Split partials and re-reads are excluded.
* Bytes of a prefill: Q, K, V, output and the cache rows written.

The cost model is the paper's Section "Cost Model": per-call cost under
reuse, eqs. (1)-(2), and the break-even reuse count, eq. (3).
"""

ELT_BYTES = {"bf16": 2, "fp16": 2, "f32": 4}


def causal_pairs(n):
    """Visible (query, key) pairs of an n-token causal prefill: n(n+1)/2."""
    return n * (n + 1) // 2


def continue_pairs(L_prefix, S):
    """Pairs of a continuation: every new row sees the whole prefix, plus a causal suffix."""
    return S * L_prefix + causal_pairs(S)


def prefill_flops(n, n_q_heads, head_dim):
    return 4 * n_q_heads * head_dim * causal_pairs(n)


def continue_flops(L_prefix, S, n_q_heads, head_dim):
    return 4 * n_q_heads * head_dim * continue_pairs(L_prefix, S)


def kv_bytes_per_token(n_kv_heads, head_dim, elt, layers=1):
    """Bytes one token adds to the cache: a K and a V row per kv head per layer."""
    return 2 * n_kv_heads * head_dim * elt * layers


def continue_bytes(L_prefix, S, n_q_heads, n_kv_heads, head_dim, elt):
    cache = kv_bytes_per_token(n_kv_heads, head_dim, elt) * L_prefix
    new_q = S * n_q_heads * head_dim * elt
    new_kv = 2 * S * n_kv_heads * head_dim * elt
    out = S * n_q_heads * head_dim * elt
    return cache + new_q + new_kv + out


def q8_artifact_bytes(tokens, n_kv_heads, head_dim, layers=1):
    """Bytes of the int8 artifact: one byte per cached K/V element plus two fp32
    scales (K and V) per layer."""
    return kv_bytes_per_token(n_kv_heads, head_dim, 1, layers) * tokens + 2 * 4 * layers


def continue_q8_bytes(L_prefix, S, n_q_heads, n_kv_heads, head_dim):
    """Continuation over the int8 artifact: int8 cache rows, bf16 new rows and output."""
    cache = kv_bytes_per_token(n_kv_heads, head_dim, 1) * L_prefix
    return cache + continue_bytes(0, S, n_q_heads, n_kv_heads, head_dim, 2)


def prefill_bytes(n, n_q_heads, n_kv_heads, head_dim, elt):
    q_out = 2 * n * n_q_heads * head_dim * elt
    kv_in = 2 * n * n_kv_heads * head_dim * elt
    cache_write = 2 * n * n_kv_heads * head_dim * elt
    return q_out + kv_in + cache_write


def append_bytes(S, n_kv_heads, head_dim, elt):
    """Read the new K/V rows, write them into the cache."""
    return 2 * 2 * S * n_kv_heads * head_dim * elt


def batched_flops(L_prefix, lengths, n_q_heads, head_dim):
    return sum(continue_flops(L_prefix, s, n_q_heads, head_dim) for s in lengths)


def batched_bytes(L_prefix, lengths, n_q_heads, n_kv_heads, head_dim, elt):
    """Prefix read once plus every reader's own Q/K/V/out."""
    tot = kv_bytes_per_token(n_kv_heads, head_dim, elt) * L_prefix
    for s in lengths:
        tot += continue_bytes(0, s, n_q_heads, n_kv_heads, head_dim, elt)
    return tot


def per_call_cost(c_prefill, c_load, n, reuse):
    """Eqs. (1)-(2): per-call cost over n uses, from scratch or with KV reuse."""
    if not reuse:
        return c_prefill
    return c_prefill / n + c_load


def total_cost(c_prefill, c_load, n, reuse):
    return n * c_prefill if not reuse else c_prefill + n * c_load


def break_even(c_prefill, c_load):
    """Eq. (3): N* = C_prefill / (C_prefill - C_load)."""
    if c_load >= c_prefill:
        return float("inf")
    return c_prefill / (c_prefill - c_load)

"""Work accounting and the cost model, pinned to numbers the paper prints.

Golden file: tests/golden/table1_qwen3_4b_m1pro.txt (paper Table 1 plus the
break-even range printed in the Experiments section, paragraph "Scaling").
"""
import os

import pytest

from harness import accounting as A
from harness import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "table1_qwen3_4b_m1pro.txt")


def table1():
    rows = []
    for line in open(GOLD):
        line = line.strip()
        if line and not line.startswith("#"):
            t, p, r, mb, sp = line.split()
            rows.append((int(t), float(p), float(r), int(mb), float(sp)))
    return rows


def test_kv_bytes_per_token_matches_paper():
    """Section "Artifact size": about 0.148 MB per token for 36 layers x 8 kv heads x 128, fp16."""
    b = A.kv_bytes_per_token(8, 128, A.ELT_BYTES["fp16"], layers=36)
    assert b == 147456
    assert round(b / 1e6, 3) == 0.147 or round(b / 1e6, 3) == 0.148
    assert abs(b / 1e6 - 0.148) < 0.001
    # one layer of the bf16 Qwen-shaped workload
    assert A.kv_bytes_per_token(W.QWEN_HKV, W.QWEN_D, 2) == 4096


def test_kv_size_column_of_table1():
    """The analytic KV size column: tokens x 147,456 B, printed in MB.

    The 3774-token row prints 557 where 556.499 rounds to 556: the paper
    rounds twice (to 556.5, then up); allow 0.51 MB.
    """
    for tokens, _, _, mb, _ in table1():
        got = tokens * A.kv_bytes_per_token(8, 128, 2, layers=36) / 1e6
        assert abs(got - mb) <= 0.51, (tokens, got, mb)


def test_speedup_column_of_table1():
    """Speedup = prefill / reuse-step (the 1888 row prints 32.4 for 32.46)."""
    for _, p, r, _, sp in table1():
        assert abs(p / r - sp) <= 0.07


def test_break_even_range_of_table1():
    """Eq. (3) on Table 1 gives N* between 1.02 and 1.13 (Experiments, "Scaling")."""
    ns = [A.break_even(p, r) for _, p, r, _, _ in table1()]
    assert round(min(ns), 2) == 1.02 and round(max(ns), 2) == 1.13
    assert A.break_even(1.0, 1.0) == float("inf")


def test_savings_at_n_1000():
    """At N = 1000 reuse saves about 0.6e3 s (255 tokens) and 1.4e4 s (3774 tokens)."""
    rows = {t: (p, r) for t, p, r, _, _ in table1()}
    for tokens, want in ((255, 0.6e3), (3774, 1.4e4)):
        p, r = rows[tokens]
        saved = A.total_cost(p, r, 1000, reuse=False) - A.total_cost(p, r, 1000, reuse=True)
        assert abs(saved - want) / want < 0.06
        # per-call cost falls toward the reuse floor (eq. 2)
        assert A.per_call_cost(p, r, 1, True) > A.per_call_cost(p, r, 1000, True) > r


def test_pair_counts_brute_force():
    for n in range(0, 30):
        assert A.causal_pairs(n) == sum(1 for i in range(n) for j in range(n) if j <= i)
    for Lp in (0, 1, 7):
        for S in (0, 1, 5):
            brute = sum(1 for i in range(S) for j in range(Lp + S) if j <= Lp + i)
            assert A.continue_pairs(Lp, S) == brute


def test_workload_accounting_numbers():
    """Algorithmic work of the Qwen-layer workload: 3798-token prefill, 24 tokens over 3774."""
    assert A.prefill_flops(3798, 32, 128) == pytest.approx(1.182e11, rel=2e-3)
    assert A.continue_bytes(3774, 24, 32, 8, 128, 2) == pytest.approx(15.95e6, rel=2e-3)
    assert A.continue_flops(32768, 24, 32, 128) == 16384 * (24 * 32768 + 300)

"""A CPU model of the 16-bit kernels' online softmax, to fix what the bar
between two GPU results on peaky rows can be.

The kernels keep (m, l, O) per row in fp32 and round the weights
p = 2^(s c2 - m) to bf16 for the P V product.  Three rules for moving the
reference m are modelled:
  exact  -- a plain running maximum: m moves to every new row maximum, so the
            largest weight seen so far is exactly 1;
  lazy   -- m moves only when a tile's maximum exceeds it by more than 2^8
            (the first tile always): weights up to 2^8, the largest rounded;
  gated  -- the kernels' rule: lazy, plus m moves to a new maximum exactly
            whenever that maximum's weight exceeds a quarter of the row's mass
            so far (running sum plus the tile).
Each rule is run with the prefill's tiling (64-key tiles from key 0) and the
continuation's (key splits of 256 keys in 32-key stages taken alternately by
two states, then the log-sum-exp merge), and the two results are compared at
the Claim 1 bar between GPU results: 2e-3 plus one bf16 output ulp.

What it shows, on the stress inputs of the GPU parity test (seed 3): the lazy
rule alone misses the bar (its dominant weights are rounded), the exact and
gated rules meet it.  And on other peaky inputs even a plain running maximum
misses it (bf16 P rounds the non-maximal heavy weights), so on peaky rows the
plain bar is a property of the inputs, not a bound bf16 P guarantees.
"""
import numpy as np
import pytest

from harness import workloads as W

SLACK, SIG = 8.0, 0.25


def bf16(x):
    """Round fp32 values to bf16 (nearest, ties to even), returned as fp32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32)


def f32(x):
    return np.asarray(x, dtype=np.float32)


class Rows:
    """Online-softmax state of R rows (log2 domain, fp32)."""

    def __init__(self, R, D):
        self.m = np.full(R, -1e30, np.float32)
        self.l = np.zeros(R, np.float32)
        self.o = np.zeros((R, D), np.float32)

    def move(self, need, mx):
        m_new = np.where(need, mx, self.m).astype(np.float32)
        alpha = np.exp2(f32(self.m - m_new))
        self.m, self.l, self.o = m_new, f32(self.l * alpha), f32(self.o * alpha[:, None])

    def tile(self, s, v, c2, rule):
        """s [R, T] fp32 scores (-inf where masked), v [R, T, D]."""
        with np.errstate(over="ignore", invalid="ignore"):
            mx = f32(np.max(s, axis=1) * c2)
            if rule == "exact":
                self.move(mx > self.m, mx)
            else:
                self.move(mx > self.m + SLACK, mx)
                if rule == "gated":
                    part = np.exp2(f32(s * c2 - self.m[:, None])).sum(1)
                    pmax = np.exp2(f32(mx - self.m))
                    self.move((mx > self.m) & (pmax > SIG * (self.l + part)), mx)
            p = np.exp2(f32(s * c2 - self.m[:, None]))
        self.l = f32(self.l + p.sum(1))
        self.o = f32(self.o + np.einsum("rt,rtd->rd", bf16(p).astype(np.float64), v).astype(np.float32))


def attend(q, k, v, pos, heads, plan, rule):
    """Rows (pos[i], heads[i]); plan: per state, its key ranges in order; the
    states are merged by their log-sum-exp at the end, output rounded to bf16."""
    G = q.shape[1] // k.shape[1]
    D = q.shape[2]
    c2 = np.float32(np.float32(1.0 / np.sqrt(D)) * np.float32(1.4426950408889634))
    Q = q[pos, heads].astype(np.float64)
    g = heads // G
    states = []
    for ranges in plan:
        st = Rows(len(pos), D)
        for k0, k1 in ranges:
            s = np.einsum("rd,trd->rt", Q, k[k0:k1][:, g, :].astype(np.float64)).astype(np.float32)
            s = np.where(np.arange(k0, k1)[None, :] <= pos[:, None], s, -np.inf).astype(np.float32)
            st.tile(s, np.transpose(v[k0:k1][:, g, :], (1, 0, 2)).astype(np.float64), c2, rule)
        states.append(st)
    M = np.max(np.stack([st.m for st in states]), axis=0)
    l = sum(f32(st.l * np.exp2(f32(st.m - M))) for st in states)
    o = sum(f32(st.o * np.exp2(f32(st.m - M))[:, None]) for st in states)
    return bf16(f32(o / l[:, None])).astype(np.float64)


def prefill_plan(n):
    return [[(t, min(t + 64, n)) for t in range(0, n, 64)]]


def continue_plan(Lp, S, chunk=256):
    n = Lp + S
    nsplit = -(-Lp // chunk)
    plan = []
    for sp in range(nsplit):
        kb = sp * chunk
        ke = n if sp == nsplit - 1 else min(kb + chunk, Lp)
        stages = [(a, min(a + 32, ke)) for a in range(kb, ke, 32)]
        plan += [stages[0::2], stages[1::2]]
    return [p for p in plan if p]


def claim1_excess(kind, seed, rule, Lp=1500, S=24):
    """max over the continuation rows of |cont - prefill| - (2e-3 + |prefill| 2^-7)."""
    q, k, v = W.stress(kind, Lp + S, W.QWEN, seed=seed)
    q, k, v = q.float().numpy(), k.float().numpy(), v.float().numpy()
    pos = np.repeat(np.arange(Lp, Lp + S), q.shape[1])
    heads = np.tile(np.arange(q.shape[1]), S)
    a = attend(q, k, v, pos, heads, prefill_plan(Lp + S), rule)
    b = attend(q, k, v, pos, heads, continue_plan(Lp, S), rule)
    return float(np.max(np.abs(b - a) - (2e-3 + 2.0 ** -7 * np.abs(a))))


@pytest.mark.parametrize("kind", ["scaled", "tile_end"])
def test_lazy_rescale_alone_misses_the_bar(kind):
    assert claim1_excess(kind, 3, "lazy") > 1e-3


@pytest.mark.parametrize("kind", ["scaled", "tile_end"])
@pytest.mark.parametrize("rule", ["exact", "gated"])
def test_exact_and_gated_references_meet_the_bar(kind, rule):
    assert claim1_excess(kind, 3, rule) <= 0.0


def test_a_plain_running_maximum_can_miss_the_bar_too():
    """Other peaky inputs: bf16 P itself, with an exact running maximum."""
    assert 0.0 < claim1_excess("scaled", 6, "exact") < 1e-3

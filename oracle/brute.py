"""Brute-force attention in pure Python, for tiny shapes only.

TEST INFRASTRUCTURE ONLY: used by the test suite to pin the compiled oracle.
It shares nothing with the compiled oracle or with the GPU library: plain
nested lists and ``math.exp``, written from the textbook definition of
scaled-dot-product attention with a causal mask (paper: Method, "Setup and
notation": the entry for a position depends only on earlier positions), and
from Alg. 2's position ids (continuation row i sits at position L_prefix + i).
"""
import math


def attend(q_rows, keys, values, n_q_heads, n_kv_heads, scale, q_pos0):
    """Causal attention of query rows over a key sequence.

    q_rows[i][h] is a list of head_dim floats (query row i, head h) at absolute
    position q_pos0 + i; keys[j][g] / values[j][g] are key/value row j of kv
    head g at absolute position j.  Returns out[i][h] (list of floats) and
    lse[i][h].
    """
    group = n_q_heads // n_kv_heads
    out, lse = [], []
    for i, qi in enumerate(q_rows):
        pos = q_pos0 + i
        orow, lrow = [], []
        for h in range(n_q_heads):
            g = h // group
            z = []
            for j in range(pos + 1):
                z.append(scale * sum(a * b for a, b in zip(qi[h], keys[j][g])))
            m = max(z)
            w = [math.exp(x - m) for x in z]
            tot = sum(w)
            d = len(qi[h])
            o = [sum(w[j] * values[j][g][c] for j in range(pos + 1)) / tot for c in range(d)]
            orow.append(o)
            lrow.append(m + math.log(tot))
        out.append(orow)
        lse.append(lrow)
    return out, lse


def to_lists(a):
    """numpy array -> nested Python lists of floats."""
    return a.tolist()

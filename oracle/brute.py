"""Scalar-loop restatement of causal attention, used only to pin the oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper Sec. 2.1: softmax(Q K^T / sqrt(d_h) + M) V, M_ij = 0 for j <= i.
Every dot product and sum is a ``math.fsum`` over Python floats (correctly
rounded sums), every exponential a ``math.exp``; no numpy, no matrices.  It
is meant for a few dozen tokens at most.
"""

from __future__ import annotations

import math


def attention_brute(q, q_pos, k, v, k_pos, scale=None):
    """Same contract as ``oracle.attention.attend`` on nested sequences.

    q[i][h][d], k[j][g][d], v[j][g][d] indexable by Python ints (lists or
    float64 arrays).  Returns (O as nested lists, LSE as nested lists).
    """
    n = len(q)
    Hq = len(q[0]) if n else 0
    D = len(q[0][0]) if n else 0
    m = len(k)
    Hkv = len(k[0]) if m else 1
    if scale is None:
        scale = 1.0 / math.sqrt(D) if D else 1.0
    group = Hq // Hkv if Hkv else 1
    O = []
    LSE = []
    for i in range(n):
        o_row = []
        l_row = []
        for h in range(Hq):
            g = h // group
            logits = []
            keys = []
            for j in range(m):
                if k_pos[j] <= q_pos[i]:
                    dot = math.fsum(float(q[i][h][d]) * float(k[j][g][d]) for d in range(D))
                    logits.append(dot * scale)
                    keys.append(j)
            if not keys:
                o_row.append([0.0] * D)
                l_row.append(-math.inf)
                continue
            top = max(logits)
            weights = [math.exp(x - top) for x in logits]
            total = math.fsum(weights)
            o_row.append([
                math.fsum(w * float(v[j][g][d]) for w, j in zip(weights, keys)) / total
                for d in range(D)
            ])
            l_row.append(top + math.log(total))
        O.append(o_row)
        LSE.append(l_row)
    return O, LSE

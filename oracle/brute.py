"""Pure-Python brute-force attention for tiny inputs (test infrastructure only).

No numpy: plain nested lists and ``math.exp``, straight from the definition
o = sum_t e^{s_t} v_t / sum_t e^{s_t}, lse = log sum_t e^{s_t} with
s_t = q . k_t / sqrt(D) over keys t <= a (paper, Section 3: the cached prefix
must give the same result as recomputing it).  Used only to pin the
vectorised float64 oracle on shapes small enough that the unshifted
exponentials cannot overflow.
"""
from __future__ import annotations

import math


def attention(q, K, V, num_q_heads, num_kv_heads):
    """``q[i][h][d]`` for the last ``n = len(q)`` positions of a sequence whose
    keys/values are ``K[t][g][d]``, ``V[t][g][d]`` (``t < L``).  Returns
    ``(o[i][h][d], lse[i][h])``."""
    n, L = len(q), len(K)
    D = len(q[0][0])
    G = num_q_heads // num_kv_heads
    inv = 1.0 / math.sqrt(D)
    o, lse = [], []
    for i in range(n):
        a = L - n + i
        orow, lrow = [], []
        for h in range(num_q_heads):
            g = h // G
            w = []
            for t in range(a + 1):
                dot = 0.0
                for d in range(D):
                    dot += q[i][h][d] * K[t][g][d]
                w.append(math.exp(dot * inv))
            z = sum(w)
            orow.append([sum(w[t] * V[t][g][d] for t in range(a + 1)) / z for d in range(D)])
            lrow.append(math.log(z))
        o.append(orow)
        lse.append(lrow)
    return o, lse

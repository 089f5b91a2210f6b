"""Scalar brute-force attention for tiny shapes (oracle; test infrastructure only).

The Section 2 definition evaluated with plain Python loops and ``math`` only -- no
BLAS, no NumPy arithmetic -- so that it shares no code path with ``attention``.
Intended for S <= 16 and D <= 8.
"""
import math


def attention_brute(q, k, v, causal, scale=None):
    """q, k, v: nested lists [S][D] of one (batch, head).  Returns (o [S][D], lse [S])."""
    S, D = len(q), len(q[0])
    Dv = len(v[0])
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out, lse = [], []
    for r in range(S):
        scores = []
        for s in range(len(k)):
            if causal and s > r:
                continue
            acc = 0.0
            for d in range(D):
                acc += float(q[r][d]) * float(k[s][d])
            scores.append((s, acc * scale))
        m = max(x for _, x in scores)
        weights = [(s, math.exp(x - m)) for s, x in scores]
        den = sum(w for _, w in weights)
        row = []
        for d in range(Dv):
            num = 0.0
            for s, w in weights:
                num += w * float(v[s][d])
            row.append(num / den)
        out.append(row)
        lse.append(m + math.log(den))
    return out, lse

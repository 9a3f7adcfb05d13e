"""Brute-force softmax attention in pure Python (tiny inputs only).

Test infrastructure only.  Evaluates the definition of Section 6 element by
element with math.exp and math.fsum (correctly rounded sums), so it shares no
BLAS or numpy reduction with ``oracle.attention``.
"""
from __future__ import annotations

import math


def attention_brute(q, k, v, scale, causal):
    """q, k, v: nested sequences [B][H][L][d]; returns nested lists [B][H][L][d]."""
    out = []
    for qb, kb, vb in zip(q, k, v):
        heads = []
        for qh, kh, vh in zip(qb, kb, vb):
            L = len(qh)
            rows = []
            for i in range(L):
                keys = range(i + 1) if causal else range(len(kh))
                logits = [scale * math.fsum(a * b for a, b in zip(qh[i], kh[j])) for j in keys]
                mx = max(logits)
                w = [math.exp(s - mx) for s in logits]
                z = math.fsum(w)
                d = len(vh[0])
                rows.append([math.fsum(wj * vh[j][t] for wj, j in zip(w, keys)) / z for t in range(d)])
            heads.append(rows)
        out.append(heads)
    return out


def probabilities_brute(q, k, scale, causal):
    """q, k: nested sequences [L][d]; returns the L x L softmax weights as nested
    lists, P[i][j] = exp(s_ij - max_j' s_ij') / sum_j' exp(s_ij' - max), with
    s_ij = scale * <q_i, k_j> and masked entries (causal, j > i) exactly 0."""
    L, n = len(q), len(k)
    out = []
    for i in range(L):
        keys = range(i + 1) if causal else range(n)
        logits = [scale * math.fsum(a * b for a, b in zip(q[i], k[j])) for j in keys]
        mx = max(logits)
        w = [math.exp(s - mx) for s in logits]
        z = math.fsum(w)
        row = [0.0] * n
        for j, wj in zip(keys, w):
            row[j] = wj / z
        out.append(row)
    return out

"""Brute-force softmax attention in pure Python (tiny inputs only).

Test infrastructure only.  Evaluates the definition of Section 5 element by
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

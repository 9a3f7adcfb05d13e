"""Plain softmax attention, the definition the fused kernel must reproduce.

Test infrastructure only (see the package docstring).

Section 6 defines R = softmax(Q K^T / sqrt(d)) V for Q, K, V in R^{L x d};
the scale is an explicit argument here (the workloads pass 1/sqrt(d) as a
float32 value).  Causal masking is not defined in the paper; the reading used
throughout is top-left aligned: row i keeps keys j <= i, and masked logits are
-inf rather than 0 (Section 5.3 explains why a zero would add a spurious
positive weight).  Batches and heads are independent [B, H, L, d] slices.

Row blocks only limit memory: each block computes its full rows exactly
(max over the whole row, then exp, sum, normalise), so no reordering of the
definition is introduced.
"""
from __future__ import annotations

import numpy as np


def attention_head(q, k, v, scale, causal, rows=None, block_rows=512, dtype=np.float64):
    """One head.  q, k, v: [L, d] arrays; returns O[rows] (all rows if rows is None).

    O[i] = sum_j P[i, j] V[j], P[i, j] = exp(s_ij - m_i) / sum_j' exp(s_ij' - m_i),
    s_ij = scale * <Q[i], K[j]> (or -inf when causal and j > i), m_i = max_j s_ij.
    """
    q = np.asarray(q, dtype=dtype)
    k = np.asarray(k, dtype=dtype)
    v = np.asarray(v, dtype=dtype)
    L = q.shape[0]
    idx = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((idx.size, v.shape[1]), dtype=dtype)
    sc = dtype(scale)
    for s0 in range(0, idx.size, block_rows):
        r = idx[s0:s0 + block_rows]
        n = int(r.max()) + 1 if causal else k.shape[0]
        s = (q[r] @ k[:n].T) * sc
        if causal:
            s[np.arange(n)[None, :] > r[:, None]] = -np.inf
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        p = e / e.sum(axis=1, keepdims=True)
        out[s0:s0 + r.size] = p @ v[:n]
    return out


def attention(q, k, v, scale, causal, block_rows=512, dtype=np.float64):
    """All heads of [B, H, L, d] inputs; returns [B, H, L, d] in `dtype`."""
    B, H, L, d = q.shape
    out = np.empty((B, H, L, v.shape[-1]), dtype=dtype)
    for b in range(B):
        for h in range(H):
            out[b, h] = attention_head(q[b, h], k[b, h], v[b, h], scale, causal,
                                       block_rows=block_rows, dtype=dtype)
    return out


def probabilities_head(q, k, scale, causal, dtype=np.float64):
    """The full L x L matrix P of one head (small L only); used by invariant tests."""
    q = np.asarray(q, dtype=dtype)
    k = np.asarray(k, dtype=dtype)
    L = q.shape[0]
    s = (q @ k.T) * dtype(scale)
    if causal:
        s[np.triu(np.ones((L, k.shape[0]), dtype=bool), 1)] = -np.inf
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=1, keepdims=True)

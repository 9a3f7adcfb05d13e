"""Row softmax and the online softmax of Section 5.3, as plain float64 code.

Test infrastructure only: only tests/, the smoke check and the benchmark's CPU
leg may import this module, and it shares no code with the GPU library.

``softmax_rows`` is the definition, y_ij = exp(x_ij - max_j x_ij) / sum_j
exp(x_ij - max_j x_ij), row by row (optionally causal: column j > row index i
is masked to -inf, the top-left reading used for attention).

``online_stats`` follows the online algorithm of Section 5.3 over column tiles
of width t: a running maximum m (from -inf) and a running denominator d (from
0); for every tile the maximum rises to m_new = max(m, tile max), the old sum
is corrected by s = exp(m - m_new) and the tile's exponentials are added:
d <- d s + sum exp(x - m_new).  A tile that extends past the row is padded,
with -inf by default; the paper notes that padding with 0 instead adds exp(0 - m)
to the denominator, and ``pad`` lets the tests show that.

``merge`` is the associative operator of Section 5.3 on (m, d) pairs, and
``softmax_split`` cuts each row into contiguous column ranges, runs the online
algorithm on each range, folds the partial (m, d) with ``merge`` in a binary
tree (split-N) and writes exp(x - m) / d.
"""
from __future__ import annotations

import numpy as np


def softmax_rows(x, causal=False):
    """The definition, row by row, in float64."""
    x = np.array(x, dtype=np.float64)
    if causal:
        r, n = x.shape
        x[np.arange(n)[None, :] > np.arange(r)[:, None]] = -np.inf
    m = x.max(axis=1, keepdims=True)
    e = np.exp(x - m)
    return e / e.sum(axis=1, keepdims=True)


def _guard(m_new):
    # a row that has seen only -inf keeps m = -inf, d = 0: use 0 as the
    # reference so that exp(-inf - 0) = 0 rather than exp(nan)
    return np.where(np.isneginf(m_new), 0.0, m_new)


def online_stats(x, t, pad=-np.inf):
    """Running (m, d) over column tiles of width t, tail tile padded with `pad`."""
    x = np.asarray(x, dtype=np.float64)
    r, n = x.shape
    m = np.full(r, -np.inf)
    d = np.zeros(r)
    for j0 in range(0, n, t):
        tile = np.full((r, t), pad, dtype=np.float64)
        w = min(t, n - j0)
        tile[:, :w] = x[:, j0:j0 + w]
        m_new = np.maximum(m, tile.max(axis=1))
        ref = _guard(m_new)
        s = np.exp(m - ref)                           # correction factor
        d = d * s + np.exp(tile - ref[:, None]).sum(axis=1)
        m = m_new
    return m, d


def merge(a, b):
    """(m_a, d_a) (+) (m_b, d_b) = (max, d_a exp(m_a - max) + d_b exp(m_b - max))."""
    (ma, da), (mb, db) = a, b
    m = np.maximum(ma, mb)
    ref = _guard(m)
    return m, da * np.exp(ma - ref) + db * np.exp(mb - ref)


def softmax_split(x, t, n_split, causal=False):
    """Split-N: online statistics per column range, merged in a binary tree."""
    x = np.array(x, dtype=np.float64)
    r, n = x.shape
    if causal:
        x[np.arange(n)[None, :] > np.arange(r)[:, None]] = -np.inf
    bounds = np.linspace(0, n, n_split + 1).astype(int)
    parts = [online_stats(x[:, a:b], t) if b > a else (np.full(r, -np.inf), np.zeros(r))
             for a, b in zip(bounds[:-1], bounds[1:])]
    while len(parts) > 1:
        nxt = [merge(parts[i], parts[i + 1]) for i in range(0, len(parts) - 1, 2)]
        if len(parts) % 2:
            nxt.append(parts[-1])
        parts = nxt
    m, d = parts[0]
    return np.exp(x - _guard(m)[:, None]) / d[:, None]

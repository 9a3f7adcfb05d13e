"""Tile-by-tile evaluation of attention and the merge of partial results.

Test infrastructure only (see the package docstring).  Float64 throughout.

Section 6 writes each output row as a ratio of two sums over the key tiles
(Eq. r0): the numerator adds exponential weights times value rows, the
denominator adds the same weights.  So every key tile t has a partial result
of its own, measured against that tile's own row maxima:

    m_t     = largest logit of the row among the tile's keys (-inf if the row
              sees none of them),
    delta_t = sum over the tile's keys of exp(logit - m_t),
    O_t     = sum over the tile's keys of exp(logit - m_t) * (value row).

The operator of Section 5.3 combines two (m, delta) pairs taken against
different maxima by re-expressing both against the larger maximum; O rides
along with delta in the same way.  The operator is associative and
commutative, so folding the tiles' triples in any order and any bracketing
(one query tile walking its keys, or split-N: contiguous key ranges folded
first and the ranges merged afterwards) gives the row maximum, the whole
denominator and the whole numerator, and O / delta is the attention output.
The fused kernel performs one such fold per query tile.

Masked keys (causal: key index above the query index) and keys past the end
enter with logit -inf, never 0 (Section 5.3, padding rule).  A row that sees
no key of a tile contributes (-inf, 0, 0), the operator's identity.  Query
tiles only group rows: rows never interact.
"""
from __future__ import annotations

import numpy as np


def tile_triple(s, v_t):
    """Partial result (m_t, delta_t, O_t) of a logit tile s [rows, n] (-inf where
    a key is masked) with its value rows v_t [n, d]."""
    m = s.max(axis=1)
    # Against its own maximum every weight is at most 1; a row with no visible
    # key has only -inf logits and takes weight 0 everywhere.
    ref = np.where(np.isneginf(m), 0.0, m)
    w = np.exp(s - ref[:, None])
    return m, w.sum(axis=1), w @ v_t


def merge(a, b):
    """(m_a, delta_a, O_a) (+) (m_b, delta_b, O_b): the Section 5.3 operator on
    (m, delta), with O re-weighted exactly like delta."""
    m_a, d_a, o_a = a
    m_b, d_b, o_b = b
    m = np.maximum(m_a, m_b)
    ref = np.where(np.isneginf(m), 0.0, m)  # both parts empty: both weights 0
    w_a = np.exp(m_a - ref)
    w_b = np.exp(m_b - ref)
    return m, d_a * w_a + d_b * w_b, o_a * w_a[:, None] + o_b * w_b[:, None]


def identity(rows, d):
    """The operator's identity element for `rows` rows of width d."""
    return np.full(rows, -np.inf), np.zeros(rows), np.zeros((rows, d))


def _logits(q, k, rows, j0, j1, scale, causal):
    s = (q[rows] @ k[j0:j1].T) * scale
    if causal:
        s[np.arange(j0, j1)[None, :] > rows[:, None]] = -np.inf
    return s


def online_head(q, k, v, scale, causal, t_q, t_kv, kv_order=None, kv_range=None):
    """One head: for every query tile of t_q rows, the triples of its key tiles
    (t_kv keys each, the last one clipped) folded left to right in `kv_order`
    (default: ascending).  kv_range = (lo, hi) restricts the keys to [lo, hi).
    Returns (O, m, delta) for all rows, O not yet divided by delta."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    L = q.shape[0]
    lo, hi = (0, k.shape[0]) if kv_range is None else kv_range
    n_tiles = -(-(hi - lo) // t_kv) if hi > lo else 0
    order = list(range(n_tiles)) if kv_order is None else list(kv_order)
    assert sorted(order) == list(range(n_tiles)), "kv_order must visit every key tile once"
    o_all = np.zeros((L, v.shape[1]))
    m_all = np.full(L, -np.inf)
    d_all = np.zeros(L)
    for i0 in range(0, L, t_q):
        rows = np.arange(i0, min(L, i0 + t_q))
        acc = identity(rows.size, v.shape[1])
        for t in order:
            j0 = lo + t * t_kv
            j1 = min(hi, j0 + t_kv)
            acc = merge(acc, tile_triple(_logits(q, k, rows, j0, j1, scale, causal), v[j0:j1]))
        m_all[rows], d_all[rows], o_all[rows] = acc
    return o_all, m_all, d_all


def attention_online(q, k, v, scale, causal, t_q, t_kv, kv_order=None):
    """All heads of [B, H, L, d] inputs through the tile fold; returns O / delta."""
    B, H, L, d = q.shape
    out = np.empty((B, H, L, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            o, _, delta = online_head(q[b, h], k[b, h], v[b, h], scale, causal, t_q, t_kv, kv_order)
            out[b, h] = o / delta[:, None]
    return out


def attention_split(q, k, v, scale, causal, t_q, t_kv, n_split, tree=True):
    """Split-N (Section 5.3): the key tiles in n_split contiguous runs of equal
    tile count (the last run shorter, trailing runs possibly empty), each run
    folded on its own, then the runs merged pairwise (tree=True, a binary
    reduction) or left to right (tree=False)."""
    B, H, L, d = q.shape
    n_tiles = -(-k.shape[2] // t_kv)
    per = -(-n_tiles // n_split)
    out = np.empty((B, H, L, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            parts = []
            for s in range(n_split):
                lo = min(k.shape[2], s * per * t_kv)
                hi = min(k.shape[2], (s + 1) * per * t_kv)
                o, m, dl = online_head(q[b, h], k[b, h], v[b, h], scale, causal, t_q, t_kv,
                                       kv_range=(lo, hi))
                parts.append((m, dl, o))
            if tree:
                while len(parts) > 1:
                    nxt = [merge(parts[i], parts[i + 1]) for i in range(0, len(parts) - 1, 2)]
                    if len(parts) % 2:
                        nxt.append(parts[-1])
                    parts = nxt
                res = parts[0]
            else:
                res = parts[0]
                for p in parts[1:]:
                    res = merge(res, p)
            m, dl, o = res
            out[b, h] = o / dl[:, None]
    return out

"""Algorithm 1 (fused attention for one Q tile) and the online-softmax merge.

Test infrastructure only.  Float64 throughout.

``attention_online`` walks Algorithm 1 of Section 5 for every Q tile: the
running maximum m starts at -inf, the running denominator delta at 0 and the
accumulator O at 0; for each key/value tile t it forms S_t = scale Q_tile K_t^T,
raises m to include the tile's row maxima, takes the correction factor
s = exp(m - m_new), exponentiates the tile against m_new, rescales delta and O
by s and adds the tile's row sums and E_t V_t; it returns O / delta.  The last
tile in each dimension is clipped to the valid extent (Section 2, boundary
policy).  Causal masking sets logits with key index > query index to -inf
(Section 4.3: padding must be -inf, not 0).

Where every logit a row has seen so far is -inf (a fully masked tile before
any visible key) m_new is -inf and exp(m - m_new) would be exp(nan); the guard
used here takes the reference point as 0 in that case, so the row keeps
m = -inf, delta = 0, O = 0 until a visible key arrives.  Rows never reach the
end fully masked in the causal top-left reading (key 0 is visible to all).

``merge`` is the associative operator of Section 4.3 extended with the
accumulator O, and ``attention_split`` runs Algorithm 1 on contiguous key
ranges and folds the partial results with it (split-N, Section 4.3).
"""
from __future__ import annotations

import numpy as np


def _tile_update(m, delta, o, s, v_t):
    """One iteration of Algorithm 1 on a score tile s [rows, n] and its values v_t [n, d]."""
    m_new = np.maximum(m, s.max(axis=1))
    ref = np.where(np.isneginf(m_new), 0.0, m_new)
    corr = np.exp(m - ref)                 # s <- exp(m - m_new)
    e = np.exp(s - ref[:, None])           # E_t <- exp(S_t - m_new)
    delta = delta * corr + e.sum(axis=1)   # delta <- delta s + rowsum(E_t)
    o = o * corr[:, None] + e @ v_t        # O <- O s + E_t V_t
    return m_new, delta, o


def online_head(q, k, v, scale, causal, t_q, t_kv, kv_order=None, kv_range=None):
    """Algorithm 1 over one head; returns (O_unnormalised, m, delta) for all rows.

    kv_order permutes the key/value tiles (any order gives the same result
    in exact arithmetic); kv_range = (lo, hi) restricts the keys to [lo, hi).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    L, d = q.shape
    lo, hi = (0, k.shape[0]) if kv_range is None else kv_range
    n_tiles = -(-(hi - lo) // t_kv) if hi > lo else 0
    order = list(range(n_tiles)) if kv_order is None else list(kv_order)
    o_all = np.zeros((L, v.shape[1]))
    m_all = np.full(L, -np.inf)
    d_all = np.zeros(L)
    for i0 in range(0, L, t_q):
        i1 = min(L, i0 + t_q)
        rows = np.arange(i0, i1)
        m = np.full(i1 - i0, -np.inf)
        delta = np.zeros(i1 - i0)
        o = np.zeros((i1 - i0, v.shape[1]))
        for t in order:
            j0 = lo + t * t_kv
            j1 = min(hi, j0 + t_kv)
            s = (q[i0:i1] @ k[j0:j1].T) * scale
            if causal:
                s[np.arange(j0, j1)[None, :] > rows[:, None]] = -np.inf
            m, delta, o = _tile_update(m, delta, o, s, v[j0:j1])
        o_all[i0:i1], m_all[i0:i1], d_all[i0:i1] = o, m, delta
    return o_all, m_all, d_all


def attention_online(q, k, v, scale, causal, t_q, t_kv, kv_order=None):
    """Algorithm 1 for all heads of [B, H, L, d] inputs; returns O / delta."""
    B, H, L, d = q.shape
    out = np.empty((B, H, L, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            o, _, delta = online_head(q[b, h], k[b, h], v[b, h], scale, causal, t_q, t_kv, kv_order)
            out[b, h] = o / delta[:, None]
    return out


def merge(a, b):
    """(m_a, delta_a, O_a) (+) (m_b, delta_b, O_b), Section 4.3, carrying O like delta."""
    m_a, d_a, o_a = a
    m_b, d_b, o_b = b
    m_new = np.maximum(m_a, m_b)
    ref = np.where(np.isneginf(m_new), 0.0, m_new)
    w_a = np.exp(m_a - ref)
    w_b = np.exp(m_b - ref)
    return m_new, d_a * w_a + d_b * w_b, o_a * w_a[:, None] + o_b * w_b[:, None]


def attention_split(q, k, v, scale, causal, t_q, t_kv, n_split, tree=True):
    """Split-N: Algorithm 1 on n_split contiguous runs of key tiles, folded with `merge`.

    tree=True folds pairwise (a binary reduction); tree=False folds left to right.
    """
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

"""Closed-form HBM traffic and flop counts of fused vs unfused attention.

Test infrastructure only.  Section 6 (savings equation) and Section 6.2
("HBM traffic"): the fused kernel reads Q, K, V and writes the output once,
4 L d elem bytes per head; the unfused pipeline also writes the L x L score
matrix, reads it back, writes the probabilities and reads them back,
4 L^2 elem more bytes per head.  Their ratio is 1 + L/d (129 at L=16384,
d=128).  The paper's savings equation counts a single pass over S against the
fused traffic, L^2 elem / (4 L d elem) = L / (4d).
"""
from __future__ import annotations


def fused_bytes(B, H, L, d, elem):
    return 4 * B * H * L * d * elem


def score_matrix_bytes(B, H, L, elem):
    return B * H * L * L * elem


def unfused_bytes(B, H, L, d, elem):
    return fused_bytes(B, H, L, d, elem) + 4 * score_matrix_bytes(B, H, L, elem)


def savings_equation(L, d):
    """The printed savings equation, L / (4 d)."""
    return L / (4 * d)


def traffic_ratio(L, d):
    """unfused / fused bytes for one head: 1 + L/d."""
    return 1 + L / d


def attention_flops(B, H, L, d, causal):
    """Two products of 2 d flops per visible (query, key) pair."""
    pairs = L * (L + 1) // 2 if causal else L * L
    return 4 * B * H * pairs * d

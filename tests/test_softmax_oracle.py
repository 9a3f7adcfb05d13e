"""Pins of the row-softmax oracle (Section 5.3): definition, online algorithm,
merge and the padding rule, against brute force, a library routine and
closed forms."""
import math

import numpy as np
import pytest
from scipy import special

from oracle import softmax as SM


def _rand(shape, seed, scale=3.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _brute(x):
    out = []
    for row in x:
        mx = max(row)
        e = [math.exp(v - mx) for v in row]
        s = math.fsum(e)
        out.append([v / s for v in e])
    return np.array(out)


@pytest.mark.parametrize("shape", [(1, 1), (3, 5), (4, 17), (2, 64)])
def test_definition_matches_brute_force(shape):
    x = _rand(shape, sum(shape))
    assert np.allclose(SM.softmax_rows(x), _brute(x.tolist()), rtol=1e-12, atol=1e-15)


def test_definition_matches_scipy():
    x = _rand((16, 300), 4)
    assert np.allclose(SM.softmax_rows(x), special.softmax(x, axis=1), rtol=1e-12, atol=1e-16)


def test_hand_case():
    x = np.array([[0.0, math.log(2.0), math.log(3.0)]])
    assert np.allclose(SM.softmax_rows(x), [[1 / 6, 2 / 6, 3 / 6]], rtol=1e-14)


def test_closed_forms():
    x = _rand((5, 40), 9)
    y = SM.softmax_rows(x)
    assert np.allclose(y.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    # invariant to a per-row shift
    assert np.allclose(SM.softmax_rows(x + np.arange(5)[:, None] * 100.0), y, rtol=1e-12)
    # a constant row is uniform; a dominant entry takes all the weight
    assert np.allclose(SM.softmax_rows(np.full((2, 7), 3.5)), 1 / 7, rtol=1e-15)
    z = np.zeros((1, 9))
    z[0, 4] = 1000.0
    assert np.array_equal(SM.softmax_rows(z), np.eye(9)[4:5])


def test_causal_reading():
    y = SM.softmax_rows(np.zeros((6, 6)), causal=True)
    for i in range(6):
        assert np.allclose(y[i, :i + 1], 1 / (i + 1), rtol=1e-15) and np.all(y[i, i + 1:] == 0)


@pytest.mark.parametrize("t", [1, 3, 7, 64, 512, 1000])
def test_online_stats_equal_max_and_denominator(t):
    x = _rand((6, 333), t)
    m, d = SM.online_stats(x, t)
    assert np.array_equal(m, x.max(axis=1))
    assert np.allclose(d, np.exp(x - x.max(axis=1, keepdims=True)).sum(axis=1), rtol=1e-13)


@pytest.mark.parametrize("n_split,t", [(1, 64), (2, 7), (3, 512), (7, 16), (16, 8)])
def test_split_n_equals_definition(n_split, t):
    x = _rand((5, 700), n_split * 31 + t)
    assert np.allclose(SM.softmax_split(x, t, n_split), SM.softmax_rows(x), rtol=1e-12, atol=1e-16)
    assert np.allclose(SM.softmax_split(x, t, n_split, causal=True), SM.softmax_rows(x, causal=True),
                       rtol=1e-12, atol=1e-16)


def test_merge_is_associative_and_commutative():
    rng = np.random.default_rng(2)
    a, b, c = [(rng.standard_normal(8) * 5, rng.random(8) * 10 + 0.1) for _ in range(3)]
    l = SM.merge(SM.merge(a, b), c)
    r = SM.merge(a, SM.merge(b, c))
    assert np.array_equal(l[0], r[0]) and np.allclose(l[1], r[1], rtol=1e-13)
    ab, ba = SM.merge(a, b), SM.merge(b, a)
    assert np.array_equal(ab[0], ba[0]) and np.allclose(ab[1], ba[1], rtol=1e-15)
    # the identity element: a range with no entries
    e = (np.full(8, -np.inf), np.zeros(8))
    ae = SM.merge(a, e)
    assert np.array_equal(ae[0], a[0]) and np.allclose(ae[1], a[1], rtol=1e-15)


def test_padding_rule():
    """Section 5.3: a tail tile padded with 0 adds exp(0 - m) per padded entry to
    the denominator; padded with -inf it adds nothing."""
    x = np.abs(_rand((4, 100), 11)) + 1.0    # the row maximum stays above the pad value 0
    t = 64
    m_inf, d_inf = SM.online_stats(x, t)
    m_zero, d_zero = SM.online_stats(x, t, pad=0.0)
    assert np.array_equal(m_inf, m_zero)
    padded = (-100) % t
    assert np.allclose(d_zero - d_inf, padded * np.exp(-m_inf), rtol=1e-12)
    assert np.allclose(d_inf, np.exp(x - m_inf[:, None]).sum(axis=1), rtol=1e-13)

"""Pins of the CPU oracle against brute force, closed forms and invariants.

None of these compare the oracle with itself: each check is either an
independent evaluation (pure-Python fsum loops), a property the mathematics
fixes (softmax rows sum to one, shift invariance, constant V), a special case
with a known answer (the paper's structured Q[i,:]=i, K=I case of Section 3.1),
or a library routine (torch's bfloat16 rounding).
"""
import math

import numpy as np
import pytest

from oracle import attention as A
from oracle import brute, online
from paper_2609_10937_amd import inputs


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("L", [1, 2, 3, 7, 16])
@pytest.mark.parametrize("d", [1, 4, 8])
@pytest.mark.parametrize("causal", [False, True])
def test_matches_brute_force(L, d, causal):
    B, H = 2, 2
    q, k, v = (_rand((B, H, L, d), s) for s in (1, 2, 3))
    scale = 0.7
    ref = np.array(brute.attention_brute(q.tolist(), k.tolist(), v.tolist(), scale, causal))
    got = A.attention(q, k, v, scale, causal, block_rows=3)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_brute_force_hand_case():
    # L=2, d=1, scale=1: logits of row 0 are (0*0, 0*1) -> equal weights;
    # row 1 logits (1*0, 1*1) -> weights (1, e) / (1 + e).
    q = [[[[0.0], [1.0]]]]
    k = [[[[0.0], [1.0]]]]
    v = [[[[2.0], [4.0]]]]
    out = brute.attention_brute(q, k, v, 1.0, False)
    assert out[0][0][0][0] == pytest.approx(3.0, abs=1e-15)
    e = math.e
    assert out[0][0][1][0] == pytest.approx((2 + 4 * e) / (1 + e), abs=1e-15)
    outc = brute.attention_brute(q, k, v, 1.0, True)
    assert outc[0][0][0][0] == 2.0


# ---------------------------------------------------------------- invariants

@pytest.mark.parametrize("causal", [False, True])
def test_probability_rows_sum_to_one(causal):
    q, k = _rand((40, 16), 4), _rand((40, 16), 5) * 3
    p = A.probabilities_head(q, k, 0.25, causal)
    assert np.max(np.abs(p.sum(axis=1) - 1.0)) <= 1e-12
    if causal:
        assert np.all(p[np.triu(np.ones((40, 40), bool), 1)] == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_constant_v_gives_constant_o(causal):
    B, H, L, d = 1, 2, 50, 8
    q, k = _rand((B, H, L, d), 6), _rand((B, H, L, d), 7)
    c = _rand((d,), 8)
    v = np.broadcast_to(c, (B, H, L, d)).copy()
    o = A.attention(q, k, v, 0.3, causal, block_rows=16)
    assert np.max(np.abs(o - c)) <= 1e-12


@pytest.mark.parametrize("zero", ["q", "scale"])
def test_uniform_logits_give_column_means(zero):
    B, H, L, d = 1, 1, 37, 8
    q, k, v = _rand((B, H, L, d), 9), _rand((B, H, L, d), 10), _rand((B, H, L, d), 11)
    scale = 0.5
    if zero == "q":
        q[:] = 0.0
    else:
        scale = 0.0
    o = A.attention(q, k, v, scale, False)
    assert np.max(np.abs(o[0, 0] - v[0, 0].mean(axis=0))) <= 1e-12
    oc = A.attention(q, k, v, scale, True)
    prefix = np.cumsum(v[0, 0], axis=0) / np.arange(1, L + 1)[:, None]
    assert np.max(np.abs(oc[0, 0] - prefix)) <= 1e-12


def test_causal_first_row_is_v0_and_single_key_is_v():
    q, k, v = (_rand((2, 3, 20, 8), s) for s in (12, 13, 14))
    o = A.attention(q, k, v, 1.0, True)
    assert np.array_equal(o[:, :, 0], v[:, :, 0])
    q1, k1, v1 = q[:, :, :1], k[:, :, :1], v[:, :, :1]
    assert np.array_equal(A.attention(q1, k1, v1, 1.0, False), v1)


def test_permutation_equivariance_and_invariance():
    L, d = 30, 8
    q, k, v = _rand((L, d), 15), _rand((L, d), 16), _rand((L, d), 17)
    base = A.attention_head(q, k, v, 0.4, False)
    perm = np.random.default_rng(18).permutation(L)
    assert np.max(np.abs(A.attention_head(q[perm], k, v, 0.4, False) - base[perm])) <= 1e-12
    assert np.max(np.abs(A.attention_head(q, k[perm], v[perm], 0.4, False) - base)) <= 1e-12


@pytest.mark.parametrize("causal", [False, True])
def test_key_shift_invariance(causal):
    L, d = 30, 8
    q, k, v = _rand((L, d), 19), _rand((L, d), 20), _rand((L, d), 21)
    c = _rand((d,), 22) * 5
    a = A.attention_head(q, k, v, 0.4, causal)
    b = A.attention_head(q, k + c, v, 0.4, causal)
    assert np.max(np.abs(a - b)) <= 1e-11


def test_huge_scale_selects_argmax_value():
    # With scale 1e4 and distinct logits the softmax is one-hot on the argmax.
    # This also fails an implementation that skips the max subtraction
    # (exp overflows to inf and the result becomes nan).
    L, d = 25, 8
    q, k, v = _rand((L, d), 23), _rand((L, d), 24), _rand((L, d), 25)
    o = A.attention_head(q, k, v, 1e4, False)
    assert np.all(np.isfinite(o))
    logits = q @ k.T
    arg = np.argmax(logits, axis=1)
    top2 = np.sort(logits, axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) * 1e4 > 60.0  # runner-up weight below e^-60
    assert clear.sum() >= L - 3
    assert np.max(np.abs(o[clear] - v[arg[clear]])) <= 1e-12


def test_paper_structured_case():
    # Section 3.1: Q[i,:] = i and K = I (so L = d) give S[i,:] = i * scale,
    # constant along each row, hence uniform probabilities and O = column mean.
    d = 16
    q = np.repeat(np.arange(d, dtype=np.float64)[:, None], d, axis=1)
    k = np.eye(d)
    v = _rand((d, d), 26)
    s = q @ k.T
    assert np.array_equal(s, q)  # S[i, :] = i
    o = A.attention_head(q, k, v, 1.0 / math.sqrt(d), False)
    assert np.max(np.abs(o - v.mean(axis=0))) <= 1e-12


# ---------------------------------------------------------------- sampled rows and P

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("block_rows", [1, 3, 512])
def test_sampled_rows_match_brute_force(causal, block_rows):
    # attention_head(rows=r) evaluates arbitrary, unsorted rows (the GPU tests
    # compare sampled rows of large workloads through it): each must equal the
    # pure-Python evaluation of that row, causal rows seeing keys 0..i only.
    L, d = 23, 6
    q, k, v = _rand((L, d), 43), _rand((L, d), 44) * 2, _rand((L, d), 45)
    ref = np.array(brute.attention_brute([[q.tolist()]], [[k.tolist()]], [[v.tolist()]], 0.6, causal))[0, 0]
    rng = np.random.default_rng(46)
    for n in (1, 5, L):
        r = rng.permutation(L)[:n]
        got = A.attention_head(q, k, v, 0.6, causal, rows=r, block_rows=block_rows)
        assert got.shape == (n, d)
        assert np.max(np.abs(got - ref[r])) <= 1e-12
    # the last row alone, and the first row alone (causal: exactly V[0])
    assert np.max(np.abs(A.attention_head(q, k, v, 0.6, causal, rows=[L - 1]) - ref[L - 1:])) <= 1e-12
    if causal:
        assert np.array_equal(A.attention_head(q, k, v, 0.6, True, rows=[0])[0], v[0])


@pytest.mark.parametrize("causal", [False, True])
def test_probabilities_match_brute_force(causal):
    # The full weight matrix against the pure-Python softmax, with a scale that
    # is not 1: a missing or doubled scale moves every off-uniform entry.
    L, d = 17, 5
    q, k = _rand((L, d), 47), _rand((L, d), 48) * 2
    ref = np.array(brute.probabilities_brute(q.tolist(), k.tolist(), 0.35, causal))
    got = A.probabilities_head(q, k, 0.35, causal)
    assert np.max(np.abs(got - ref)) <= 1e-13
    wrong = A.probabilities_head(q, k, 0.7, causal)
    assert np.max(np.abs(wrong - ref)) > 1e-2


def test_probabilities_hand_case():
    # Two keys with logits 0 and scale * 2 = ln 3 give weights 1/4 and 3/4.
    q = np.array([[1.0]])
    k = np.array([[0.0], [2.0]])
    p = A.probabilities_head(q, k, math.log(3.0) / 2.0, False)
    assert p[0] == pytest.approx([0.25, 0.75], abs=1e-15)


# ---------------------------------------------------------------- tile fold

def test_tile_triple_hand_case():
    # One row, logits (0, ln 2) and a masked key: m = ln 2, weights (1/2, 1, 0),
    # delta = 3/2, O = 1/2 v0 + v1.
    s = np.array([[0.0, math.log(2.0), -np.inf]])
    v = np.array([[2.0, 0.0], [0.0, 4.0], [100.0, 100.0]])
    m, dl, o = online.tile_triple(s, v)
    assert m[0] == pytest.approx(math.log(2.0), abs=1e-15)
    assert dl[0] == pytest.approx(1.5, abs=1e-15)
    assert o[0] == pytest.approx([1.0, 4.0], abs=1e-15)
    # a fully masked row is the identity: merging it changes nothing
    e = online.tile_triple(np.full((1, 3), -np.inf), v)
    assert e[0][0] == -np.inf and e[1][0] == 0.0 and np.all(e[2] == 0.0)
    mm = online.merge((m, dl, o), e)
    assert mm[0][0] == m[0] and mm[1][0] == dl[0] and np.array_equal(mm[2], o)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("t_q,t_kv", [(16, 16), (48, 64), (32, 160), (7, 5)])
def test_algorithm1_equals_definition(causal, t_q, t_kv):
    B, H, L, d = 1, 2, 203, 16
    q, k, v = _rand((B, H, L, d), 27), _rand((B, H, L, d), 28) * 3, _rand((B, H, L, d), 29)
    ref = A.attention(q, k, v, 0.25, causal)
    got = online.attention_online(q, k, v, 0.25, causal, t_q, t_kv)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_algorithm1_any_kv_order():
    B, H, L, d = 1, 1, 150, 8
    q, k, v = _rand((B, H, L, d), 30), _rand((B, H, L, d), 31) * 3, _rand((B, H, L, d), 32)
    ref = A.attention(q, k, v, 0.5, True)
    order = np.random.default_rng(33).permutation(-(-L // 16))
    got = online.attention_online(q, k, v, 0.5, True, 16, 16, kv_order=order)
    assert np.max(np.abs(got - ref)) <= 1e-12


@pytest.mark.parametrize("n_split", [1, 2, 3, 5, 8])
@pytest.mark.parametrize("tree", [True, False])
@pytest.mark.parametrize("causal", [False, True])
def test_split_n_merge_equals_definition(n_split, tree, causal):
    B, H, L, d = 1, 1, 200, 8
    q, k, v = _rand((B, H, L, d), 34), _rand((B, H, L, d), 35) * 3, _rand((B, H, L, d), 36)
    ref = A.attention(q, k, v, 0.5, causal)
    got = online.attention_split(q, k, v, 0.5, causal, 32, 16, n_split, tree=tree)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_merge_is_associative():
    rng = np.random.default_rng(37)
    parts = []
    for _ in range(3):
        m = rng.standard_normal(6) * 4
        m[0] = -np.inf  # an empty part for row 0
        dl = np.where(np.isneginf(m), 0.0, rng.random(6) + 0.5)
        o = rng.standard_normal((6, 4)) * dl[:, None]
        parts.append((m, dl, o))
    a, b, c = parts
    left = online.merge(online.merge(a, b), c)
    right = online.merge(a, online.merge(b, c))
    for x, y in zip(left, right):
        assert np.allclose(x, y, rtol=1e-14, atol=0)


def test_zero_padding_would_corrupt_denominator():
    # Section 5.3: a padded key with logit 0 instead of -inf adds exp(0 - m) > 0
    # to the denominator.  Plant that mistake in a fold over padded tiles and
    # check it moves the result away from the definition; -inf padding does not.
    L, d, t_kv = 10, 4, 8  # the second key tile has 6 padded slots
    q, k, v = _rand((L, d), 38), _rand((L, d), 39), _rand((L, d), 40)
    ref = A.attention_head(q, k, v, 1.0, False)
    pad = 2 * t_kv - L
    kp = np.vstack([k, np.zeros((pad, d))])
    vp = np.vstack([v, np.zeros((pad, d))])

    def run(pad_value):
        acc = online.identity(L, d)
        for j0 in (0, t_kv):
            s = q @ kp[j0:j0 + t_kv].T
            s[:, max(0, L - j0):] = pad_value
            acc = online.merge(acc, online.tile_triple(s, vp[j0:j0 + t_kv]))
        return acc[2] / acc[1][:, None]

    assert np.max(np.abs(run(-np.inf) - ref)) <= 1e-12
    assert np.max(np.abs(run(0.0) - ref)) > 1e-3


# ---------------------------------------------------------------- inputs

def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(41)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -0.0, 65504.0, 1e-40],
                                 dtype=np.float32)])
    ours = inputs.f32_to_bf16_bits(x)
    theirs = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, theirs)


def test_f16_roundtrip_and_widening_is_exact():
    x = np.random.default_rng(42).standard_normal(1000).astype(np.float32)
    bits = inputs.f32_to_f16_bits(x)
    assert np.array_equal(inputs.bits_to_f64(bits, "f16"), x.astype(np.float16).astype(np.float64))
    b16 = inputs.f32_to_bf16_bits(x)
    w = inputs.bits_to_f64(b16, "bf16")
    assert np.max(np.abs(w - x) / np.abs(x)) <= 2.0 ** -8


def test_generator_is_seeded_and_ordered():
    q1, k1, v1 = inputs.make_qkv(1, 2, 8, 4, "bf16", 7)
    q2, k2, v2 = inputs.make_qkv(1, 2, 8, 4, "bf16", 7)
    assert np.array_equal(q1, q2) and np.array_equal(k1, k2) and np.array_equal(v1, v2)
    _, k3, _ = inputs.make_qkv(1, 2, 8, 4, "bf16", 7, k_scale=3.0)
    rng = np.random.Generator(np.random.PCG64(7))
    rng.standard_normal((1, 2, 8, 4), dtype=np.float32)
    kk = rng.standard_normal((1, 2, 8, 4), dtype=np.float32) * np.float32(3.0)
    assert np.array_equal(k3, inputs.f32_to_bf16_bits(kk))

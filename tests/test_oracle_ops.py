"""Pins for the oracle's plain ops: GELU (erf form), RMSNorm, causal attention.

Pinned against closed forms, textbook values, pure-Python brute force using
the ``math`` module, and independent library routines (torch float64 on the
CPU), never against the oracle itself.
"""
import math

import numpy as np
import pytest
import torch

from oracle import partir_oracle as O


# ---------------------------------------------------------------------------
# GELU
# ---------------------------------------------------------------------------
# erf at a few points, to 16 digits (Abramowitz & Stegun, Table 7.1)
ERF_TABLE = {0.5: 0.5204998778130465, 1.0: 0.8427007929497149, 2.0: 0.9953222650189527}


def test_gelu_textbook_points():
    # gelu(t*sqrt 2) = (t*sqrt 2)/2 * (1 + erf t)
    for t, e in ERF_TABLE.items():
        x = t * math.sqrt(2.0)
        assert abs(O.gelu_erf(np.array([x]))[0] - 0.5 * x * (1 + e)) < 1e-15


def test_gelu_closed_forms():
    assert O.gelu_erf(np.array([0.0]))[0] == 0.0
    x = np.linspace(-6, 6, 97)
    # erf is odd, so gelu(x) - gelu(-x) = x
    assert np.max(np.abs(O.gelu_erf(x) - O.gelu_erf(-x) - x)) < 1e-14
    big = np.array([12.0, 40.0])
    assert np.array_equal(O.gelu_erf(big), big)
    assert np.all(np.abs(O.gelu_erf(-big)) < 1e-30)


def test_gelu_matches_math_erf_and_torch():
    x = np.random.default_rng(0).standard_normal(257) * 3
    brute = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in x])
    assert np.max(np.abs(O.gelu_erf(x) - brute)) < 1e-15
    t = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    assert np.max(np.abs(O.gelu_erf(x) - t)) < 1e-14


def test_gelu_is_not_tanh_form():
    x = np.array([1.0])
    tanh_form = 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))
    assert abs(O.gelu_erf(x)[0] - tanh_form[0]) > 1e-5


# ---------------------------------------------------------------------------
# RMSNorm
# ---------------------------------------------------------------------------
def test_rmsnorm_constant_row_closed_form():
    eps = 1e-6
    g = np.array([1.0, -2.0, 0.5, 3.0])
    for c in (-2.5, 0.1, 7.0):
        y = O.rmsnorm(np.full((1, 4), c), g, eps)[0]
        expect = g * math.copysign(1.0, c) / math.sqrt(1 + eps / c ** 2)
        assert np.max(np.abs(y - expect)) < 1e-15


def test_rmsnorm_brute_force_and_scale_invariance():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 10))
    g = rng.standard_normal(10)
    eps = 1e-5
    for i in range(3):
        ms = sum(v * v for v in x[i]) / 10
        brute = [g[j] * x[i][j] / math.sqrt(ms + eps) for j in range(10)]
        assert np.max(np.abs(O.rmsnorm(x, g, eps)[i] - brute)) < 1e-14
    # with eps = 0 the norm is invariant to positive row scaling
    assert np.allclose(O.rmsnorm(5 * x, g, 0.0), O.rmsnorm(x, g, 0.0), rtol=1e-14, atol=0)


# ---------------------------------------------------------------------------
# causal attention
# ---------------------------------------------------------------------------
def brute_attention(q, k, v, scale, causal=True):
    out = []
    for i in range(len(q)):
        js = range(i + 1) if causal else range(len(k))
        s = [scale * sum(a * b for a, b in zip(q[i], k[j])) for j in js]
        m = max(s)
        e = [math.exp(t - m) for t in s]
        z = sum(e)
        out.append([sum(e[t] / z * v[j][d] for t, j in enumerate(js)) for d in range(len(v[0]))])
    return np.array(out)


@pytest.mark.parametrize("causal", [True, False])
def test_attention_brute_force(causal):
    rng = np.random.default_rng(9)
    q, k, v = (rng.standard_normal((7, 5)) for _ in range(3))
    got = O.causal_attention(q, k, v, 0.37, causal)
    assert np.max(np.abs(got - brute_attention(q, k, v, 0.37, causal))) < 1e-14


def test_attention_first_position_is_v0_exactly():
    rng = np.random.default_rng(1)
    q, k, v = (rng.standard_normal((6, 4)) for _ in range(3))
    assert np.array_equal(O.causal_attention(q, k, v, 0.5)[0], v[0])


def test_attention_zero_queries_give_prefix_means():
    rng = np.random.default_rng(2)
    k, v = rng.standard_normal((9, 4)), rng.integers(-4, 5, (9, 4)).astype(np.float64)
    o = O.causal_attention(np.zeros((9, 4)), k, v, 1.0)
    for i in range(9):
        assert np.max(np.abs(o[i] - v[:i + 1].mean(axis=0))) < 1e-14


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((33, 16)) for _ in range(3))
    scale = 16 ** -0.5
    t = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
        is_causal=True, scale=scale)[0].numpy()
    assert np.max(np.abs(O.causal_attention(q, k, v, scale) - t)) < 1e-13


def test_attention_query_positions_subset():
    rng = np.random.default_rng(5)
    q, k, v = (rng.standard_normal((12, 8)) for _ in range(3))
    full = O.causal_attention(q, k, v, 0.3)
    pos = np.array([0, 4, 11])
    part = O.causal_attention(q[pos], k, v, 0.3, q_pos=pos)
    assert np.max(np.abs(part - full[pos])) < 1e-15
    # a query only needs the keys up to its own position
    part2 = O.causal_attention(q[[4]], k[:5], v[:5], 0.3, q_pos=np.array([4]))
    assert np.max(np.abs(part2[0] - full[4])) < 1e-15


def test_attention_large_scores_stay_finite():
    q = np.full((4, 2), 300.0)
    k = np.array([[1.0, 1.0], [2.0, 2.0], [-1.0, 0.0], [3.0, 3.0]])
    v = np.arange(8.0).reshape(4, 2)
    o = O.causal_attention(q, k, v, 1.0)
    assert np.all(np.isfinite(o))
    assert np.array_equal(o[1], v[1]) and np.array_equal(o[3], v[3])


# ---------------------------------------------------------------------------
# the key axis as a loop with the softmax combiner (custom associative #sum)
# ---------------------------------------------------------------------------
def test_split_kv_attention_equals_attention():
    """Folding the shards' (m, l, o) with the combiner gives softmax
    attention over all keys, for every shard count and with a causal mask
    (shards past a query contribute the identity)."""
    rng = np.random.default_rng(31)
    q, k, v = (rng.standard_normal((64, 16)) for _ in range(3))
    for causal in (True, False):
        ref = O.causal_attention(q, k, v, 0.25, causal)
        for R in (1, 2, 4, 8, 64):
            got = O.attention_split_kv(q, k, v, 0.25, causal, R)
            assert np.abs(got - ref).max() <= 1e-13


def test_softmax_combiner_is_associative_and_commutative_with_identity():
    rng = np.random.default_rng(32)
    q = rng.standard_normal((8, 4))
    parts = []
    for r in range(3):
        k, v = rng.standard_normal((5, 4)), rng.standard_normal((5, 4))
        parts.append(O.softmax_partial(q, k, v, 1.3, False, np.arange(8), np.arange(5)))
    a, b, c = parts

    def close(x, y):
        return all(np.allclose(u, w, rtol=1e-13, atol=1e-13) for u, w in zip(x, y))
    assert close(O.softmax_combine(O.softmax_combine(a, b), c), O.softmax_combine(a, O.softmax_combine(b, c)))
    assert close(O.softmax_combine(a, b), O.softmax_combine(b, a))
    ident = (np.full(8, -np.inf), np.zeros(8), np.zeros((8, 4)))
    assert close(O.softmax_combine(a, ident), a) and close(O.softmax_combine(ident, a), a)


def test_softmax_partial_brute_force():
    """(m, l, o) of one shard against pure-Python loops."""
    rng = np.random.default_rng(33)
    q, k, v = rng.standard_normal((3, 4)), rng.standard_normal((5, 4)), rng.standard_normal((5, 4))
    m, l, o = O.softmax_partial(q, k, v, 0.5, True, np.array([1, 3, 9]), np.arange(2, 7))
    for i, qp in enumerate([1, 3, 9]):
        s = [0.5 * sum(q[i][t] * k[j][t] for t in range(4)) for j in range(5) if 2 + j <= qp]
        js = [j for j in range(5) if 2 + j <= qp]
        if not s:
            assert m[i] == -np.inf and l[i] == 0 and not o[i].any()
            continue
        mm = max(s)
        assert m[i] == pytest.approx(mm, rel=1e-14)
        assert l[i] == pytest.approx(sum(math.exp(x - mm) for x in s), rel=1e-13)
        for t in range(4):
            assert o[i][t] == pytest.approx(sum(math.exp(x - mm) * v[j][t] for x, j in zip(s, js)), rel=1e-12, abs=1e-14)

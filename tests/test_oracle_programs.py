"""Pins for the oracle's partitioned programs (MLP, attention, decoder).

The shard interpreter is compared with the unpartitioned evaluator (the
correctness theorem of the lowering: a partitioned loop equals the
unpartitioned op), with pure-Python brute force on tiny inputs, bitwise on
integer-exact inputs, across partition sizes, and on sampled rows.
"""
import math

import numpy as np
import pytest

from oracle import partir_oracle as O


def ints(rng, shape, lo=-1, hi=1):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float64)


# ---------------------------------------------------------------------------
# MLP
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("Rb,Rm", [(1, 1), (1, 2), (1, 8), (2, 4), (4, 8)])
def test_mlp_integer_exact_across_partitions(Rb, Rm):
    rng = np.random.default_rng(Rb * 10 + Rm)
    X, W1, W2 = ints(rng, (32, 16)), ints(rng, (16, 64)), ints(rng, (64, 16))
    ref = O.matmul(O.matmul(X, W1), W2)
    assert np.array_equal(O.mlp_block(X, W1, W2, act="none", R_batch=Rb, R_model=Rm), ref)


def test_mlp_brute_force_gelu_with_biases():
    rng = np.random.default_rng(0)
    T, D, F = 4, 3, 8
    X, W1, W2 = rng.standard_normal((T, D)), rng.standard_normal((D, F)), rng.standard_normal((F, D))
    b1, b2 = rng.standard_normal(F), rng.standard_normal(D)
    brute = np.zeros((T, D))
    for i in range(T):
        h = [sum(X[i][d] * W1[d][f] for d in range(D)) + b1[f] for f in range(F)]
        h = [0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in h]
        for j in range(D):
            brute[i][j] = sum(h[f] * W2[f][j] for f in range(F)) + b2[j]
    for Rb, Rm in [(1, 1), (2, 4), (4, 2)]:
        got = O.mlp_block(X, W1, W2, b1, b2, "gelu", Rb, Rm)
        assert np.max(np.abs(got - brute)) < 1e-13


def test_mlp_bias_of_sum_loop_is_added_once():
    """Adding a replicated b2 inside the #sum body would add it R times."""
    rng = np.random.default_rng(1)
    X, W1, W2 = rng.standard_normal((8, 4)), rng.standard_normal((4, 16)), rng.standard_normal((16, 4))
    b2 = np.ones(4)
    with_bias = O.mlp_block(X, W1, W2, None, b2, "gelu", 1, 4)
    without = O.mlp_block(X, W1, W2, None, None, "gelu", 1, 4)
    assert np.allclose(with_bias - without, 1.0, rtol=0, atol=1e-13)
    wrong = O.loop_sum(4, lambda m: O.matmul(O.gelu_erf(O.matmul(X, O.slice_(W1, 1, m, 4))),
                                             O.slice_(W2, 0, m, 4)) + b2)
    assert np.allclose(wrong - without, 4.0, rtol=0, atol=1e-12)


def test_mlp_rows_match_full_and_norm_bounds_output():
    rng = np.random.default_rng(2)
    X, W1, W2 = rng.standard_normal((64, 8)), rng.standard_normal((8, 32)), rng.standard_normal((32, 8))
    full, norm = O.mlp_block(X, W1, W2, R_batch=4, R_model=8, return_norm=True)
    rows = [0, 15, 16, 31, 47, 63]
    part, pnorm = O.mlp_block(X, W1, W2, R_batch=4, R_model=8, rows=rows, return_norm=True)
    # (BLAS may block a row subset differently: equal up to rounding)
    assert np.max(np.abs(part - full[rows]) / norm[rows]) < 1e-14
    assert np.max(np.abs(pnorm - norm[rows]) / norm[rows]) < 1e-14
    assert np.all(np.abs(full) <= norm * (1 + 1e-12))
    h = O.gelu_erf(O.matmul(X, W1))
    assert np.allclose(norm, O.abs_product(h, W2), rtol=1e-13, atol=0)


def test_mlp_rejects_indivisible():
    with pytest.raises(ValueError):
        O.mlp_block(np.zeros((6, 2)), np.zeros((2, 8)), np.zeros((8, 2)), R_batch=4)
    with pytest.raises(ValueError):
        O.mlp_block(np.zeros((8, 2)), np.zeros((2, 6)), np.zeros((6, 2)), R_model=4)


# ---------------------------------------------------------------------------
# attention block
# ---------------------------------------------------------------------------
def brute_attn_block(X, Wq, Wk, Wv, Wo, B, S, H, dh):
    """Per-sequence, per-head loops written out directly."""
    Q, K, V = X @ Wq, X @ Wk, X @ Wv
    A = np.zeros_like(Q)
    for s in range(B):
        for h in range(H):
            for i in range(S):
                qi = Q[s * S + i, h * dh:(h + 1) * dh]
                sc = [float(qi @ K[s * S + j, h * dh:(h + 1) * dh]) / math.sqrt(dh) for j in range(i + 1)]
                m = max(sc)
                e = [math.exp(t - m) for t in sc]
                z = sum(e)
                A[s * S + i, h * dh:(h + 1) * dh] = sum(e[j] / z * V[s * S + j, h * dh:(h + 1) * dh]
                                                        for j in range(i + 1))
    return A @ Wo


@pytest.mark.parametrize("Rb,Rm", [(1, 1), (1, 4), (2, 2), (2, 4)])
def test_attn_block_brute_force(Rb, Rm):
    rng = np.random.default_rng(Rb + 3 * Rm)
    B, S, H, dh = 2, 6, 4, 3
    D = H * dh
    X = rng.standard_normal((B * S, D))
    Ws = [rng.standard_normal((D, D)) / math.sqrt(D) for _ in range(4)]
    ref = brute_attn_block(X, *Ws, B, S, H, dh)
    got = O.attn_block(X, *Ws, B, S, H, dh, R_batch=Rb, R_model=Rm)
    assert np.max(np.abs(got - ref)) < 1e-13
    assert np.max(np.abs(O.attn_ref(X, *Ws, B, S, H, dh) - ref)) < 1e-13


def test_attn_block_rows_and_norm():
    rng = np.random.default_rng(8)
    B, S, H, dh = 2, 16, 4, 8
    D = H * dh
    X = rng.standard_normal((B * S, D))
    Ws = [rng.standard_normal((D, D)) / math.sqrt(D) for _ in range(4)]
    full, norm = O.attn_block(X, *Ws, B, S, H, dh, R_batch=2, R_model=2, return_norm=True)
    rows = [0, 5, 15, 16, 31]
    part, pn = O.attn_block(X, *Ws, B, S, H, dh, R_batch=2, R_model=2, rows=rows, return_norm=True)
    assert np.max(np.abs(part - full[rows])) < 1e-14
    assert np.max(np.abs(pn - norm[rows])) < 1e-14
    assert np.all(np.abs(full) <= norm * (1 + 1e-12))


def test_attn_heads_tile_is_concatenation_of_single_heads():
    rng = np.random.default_rng(6)
    B, S, H, dh = 1, 5, 4, 2
    D = H * dh
    X = rng.standard_normal((S, D))
    Wq, Wk, Wv = (rng.standard_normal((D, D)) for _ in range(3))
    eye = np.eye(D)
    a = O.attn_block(X, Wq, Wk, Wv, eye, B, S, H, dh, R_model=2)
    for h in range(H):
        cs = slice(h * dh, (h + 1) * dh)
        one = O.causal_attention((X @ Wq)[:, cs], (X @ Wk)[:, cs], (X @ Wv)[:, cs], dh ** -0.5)
        assert np.max(np.abs(a[:, cs] - one)) < 1e-14


# ---------------------------------------------------------------------------
# decoder
# ---------------------------------------------------------------------------
def make_layer(rng, D, F, gains=True):
    p = {n: rng.standard_normal((D, D)) / math.sqrt(D) for n in ("Wq", "Wk", "Wv", "Wo")}
    p["W1"] = rng.standard_normal((D, F)) / math.sqrt(D)
    p["W2"] = rng.standard_normal((F, D)) / math.sqrt(F)
    p["g1"] = rng.standard_normal(D) if gains else np.ones(D)
    p["g2"] = rng.standard_normal(D) if gains else np.ones(D)
    return p


def brute_decoder_layer(x, p, B, S, H, dh, eps):
    def rms(t, g):
        return np.stack([g * r / math.sqrt(sum(v * v for v in r) / len(r) + eps) for r in t])
    h = x + brute_attn_block(rms(x, p["g1"]), p["Wq"], p["Wk"], p["Wv"], p["Wo"], B, S, H, dh)
    u = rms(h, p["g2"]) @ p["W1"]
    u = np.vectorize(lambda v: 0.5 * v * (1 + math.erf(v / math.sqrt(2))))(u)
    return h + u @ p["W2"]


@pytest.mark.parametrize("Rb,Rm", [(1, 1), (2, 2), (2, 4)])
def test_decoder_layer_brute_force(Rb, Rm):
    rng = np.random.default_rng(Rb * 7 + Rm)
    B, S, H, dh, F = 2, 5, 4, 2, 12
    D = H * dh
    x = rng.standard_normal((B * S, D))
    p = make_layer(rng, D, F)
    ref = brute_decoder_layer(x, p, B, S, H, dh, 1e-6)
    got, norm = O.decoder_layer(x, p, B, S, H, dh, 1e-6, Rb, Rm, return_norm=True)
    assert np.max(np.abs(got - ref)) < 1e-12
    assert np.all(np.abs(got) <= norm * (1 + 1e-12))


def test_decoder_stack_rows_match_full():
    rng = np.random.default_rng(12)
    B, S, H, dh, F = 2, 8, 4, 4, 24
    D = H * dh
    x = rng.standard_normal((B * S, D))
    layers = [make_layer(rng, D, F), make_layer(rng, D, F)]
    full, norm = O.decoder(x, layers, B, S, H, dh, R_batch=2, R_model=4, return_norm=True)
    assert np.max(np.abs(full - O.decoder_ref(x, layers, B, S, H, dh))) < 1e-12
    rows = [0, 3, 8, 15]
    part, pn = O.decoder(x, layers, B, S, H, dh, R_batch=2, R_model=4, rows=rows, return_norm=True)
    assert np.max(np.abs(part - full[rows])) < 1e-13
    assert np.max(np.abs(pn - norm[rows])) < 1e-13
    assert list(O.decoder_rows_needed([3, 8, 10], B * S, S)) == [0, 1, 2, 3, 8, 9, 10]


def test_decoder_independent_of_model_partition():
    rng = np.random.default_rng(13)
    B, S, H, dh, F = 2, 4, 8, 2, 16
    D = H * dh
    x = rng.standard_normal((B * S, D))
    p = make_layer(rng, D, F)
    outs = [O.decoder_layer(x, p, B, S, H, dh, 1e-6, Rb, Rm) for Rb in (1, 2) for Rm in (1, 2, 4, 8)]
    for o in outs[1:]:
        assert np.max(np.abs(o - outs[0])) < 1e-12


def test_mlp_with_empty_ffn_is_the_output_bias():
    """F = 0: every model shard holds no hidden units, the #sum over m adds R
    empty contributions (0), and only the bias added after the loop remains."""
    rng = np.random.default_rng(7)
    X = rng.standard_normal((16, 8))
    b2 = rng.standard_normal(8)
    for Rm in (1, 4):
        Y = O.mlp_block(X, np.zeros((8, 0)), np.zeros((0, 8)), None, b2, "gelu", 1, Rm)
        assert np.array_equal(Y, np.broadcast_to(b2, (16, 8)))
    assert np.array_equal(O.mlp_block(X, np.zeros((8, 0)), np.zeros((0, 8)), act="gelu", R_model=2),
                          np.zeros((16, 8)))


def test_decoder_with_empty_ffn_equals_zero_down_projection():
    """F = 0 adds the empty sum; a width-8 FFN whose down-projection is all
    zeros adds exactly 0 as well, so the two layers agree bit for bit, and
    the normaliser falls back to the attention residual add (>= |x|)."""
    rng = np.random.default_rng(11)
    B, S, H, dh = 2, 8, 2, 4
    D = H * dh
    x = rng.standard_normal((B * S, D))
    p = {"g1": np.ones(D), "g2": np.ones(D)}
    for k in ("Wq", "Wk", "Wv", "Wo"):
        p[k] = rng.standard_normal((D, D)) / math.sqrt(D)
    empty = dict(p, W1=np.zeros((D, 0)), W2=np.zeros((0, D)))
    zero = dict(p, W1=rng.standard_normal((D, 8)), W2=np.zeros((8, D)))
    for Rm in (1, 2):
        a, na = O.decoder_layer(x, empty, B, S, H, dh, R_batch=2, R_model=Rm, return_norm=True)
        b = O.decoder_layer(x, zero, B, S, H, dh, R_batch=2, R_model=Rm)
        assert np.array_equal(a, b)
        assert np.all(na >= np.abs(x) - 1e-15) and np.all(na > 0)

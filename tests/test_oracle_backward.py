"""Pins for the oracle's MLP backward pass (gradients as loop nests).

The gradients are pinned to things other than the oracle's own formulas:
closed forms of GELU's derivative, central finite differences of the
(separately pinned) forward shard interpreter, torch's fp64 autograd of the
same forward, and bitwise integer arithmetic for the identity activation
across partition sizes.
"""
import math

import numpy as np
import pytest
import torch

from oracle import partir_oracle as O

KEYS = ("dX", "dW1", "dW2", "db1", "db2")


def ints(rng, shape, lo=-2, hi=2):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float64)


def problem(seed, T=16, D=8, F=32, scale=1.0):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, D)) * scale
    W1 = rng.standard_normal((D, F)) / math.sqrt(D)
    W2 = rng.standard_normal((F, D)) / math.sqrt(F)
    dY = rng.standard_normal((T, D))
    b1 = rng.standard_normal(F) * 0.5
    return X, W1, W2, dY, b1


# ---------------------------------------------------------------------------
# GELU derivative
# ---------------------------------------------------------------------------
def test_gelu_grad_closed_forms():
    assert O.activation_grad(np.array([0.0]), "gelu")[0] == 0.5
    x = np.linspace(-7, 7, 113)
    # Phi(x) + Phi(-x) = 1 and x phi(x) is odd: gelu'(x) + gelu'(-x) = 1
    assert np.max(np.abs(O.activation_grad(x, "gelu") + O.activation_grad(-x, "gelu") - 1)) < 1e-15
    assert np.all(np.abs(O.activation_grad(np.array([40.0]), "gelu") - 1) < 1e-15)
    assert np.all(np.abs(O.activation_grad(np.array([-40.0]), "gelu")) < 1e-30)
    assert np.array_equal(O.activation_grad(x, "none"), np.ones_like(x))
    # the minimum of gelu' (near x = -1.4142) equals 1 - Phi(sqrt2) - sqrt2 phi(sqrt2)
    s2 = math.sqrt(2.0)
    closed = 0.5 * math.erfc(1.0) - s2 * math.exp(-1.0) / math.sqrt(2 * math.pi)
    assert abs(O.activation_grad(np.array([-s2]), "gelu")[0] - closed) < 1e-16


def test_gelu_grad_matches_central_differences_and_torch():
    x = np.random.default_rng(3).standard_normal(301) * 3
    h = 1e-5
    fd = (O.gelu_erf(x + h) - O.gelu_erf(x - h)) / (2 * h)
    assert np.max(np.abs(O.activation_grad(x, "gelu") - fd)) < 1e-9
    t = torch.from_numpy(x).requires_grad_(True)
    torch.nn.functional.gelu(t, approximate="none").sum().backward()
    assert np.max(np.abs(O.activation_grad(x, "gelu") - t.grad.numpy())) < 1e-15


# ---------------------------------------------------------------------------
# MLP gradients
# ---------------------------------------------------------------------------
def torch_grads(X, W1, W2, dY, b1, act):
    ts = {k: torch.from_numpy(np.array(v)).requires_grad_(True)
          for k, v in dict(X=X, W1=W1, W2=W2, b1=b1, b2=np.zeros(W2.shape[1])).items()}
    z = ts["X"] @ ts["W1"] + ts["b1"]
    h = torch.nn.functional.gelu(z, approximate="none") if act == "gelu" else z
    y = h @ ts["W2"] + ts["b2"]
    y.backward(torch.from_numpy(dY))
    return {"dX": ts["X"].grad.numpy(), "dW1": ts["W1"].grad.numpy(), "dW2": ts["W2"].grad.numpy(),
            "db1": ts["b1"].grad.numpy(), "db2": ts["b2"].grad.numpy()}


@pytest.mark.parametrize("act", ["gelu", "none"])
@pytest.mark.parametrize("Rb,Rm", [(1, 1), (2, 4), (4, 2), (1, 8)])
def test_mlp_backward_matches_torch_autograd(act, Rb, Rm):
    X, W1, W2, dY, b1 = problem(10 + Rb * 8 + Rm)
    want = torch_grads(X, W1, W2, dY, b1, act)
    got = O.mlp_block_backward(X, W1, W2, dY, b1, act, Rb, Rm)
    ref = O.mlp_backward_ref(X, W1, W2, dY, b1, act)
    for k in KEYS:
        assert got[k].shape == want[k].shape
        assert np.max(np.abs(got[k] - want[k])) < 1e-12, k
        assert np.max(np.abs(ref[k] - want[k])) < 1e-12, k


def test_mlp_backward_central_differences_of_the_forward():
    """dL/dtheta for L = <mlp_block(theta), dY>, entry by entry."""
    T, D, F = 4, 3, 8
    X, W1, W2, dY, b1 = problem(5, T, D, F)
    b2 = np.zeros(D)
    g = O.mlp_block_backward(X, W1, W2, dY, b1, "gelu", 2, 4)
    args = dict(X=X, W1=W1, W2=W2, b1=b1, b2=b2)
    names = {"dX": "X", "dW1": "W1", "dW2": "W2", "db1": "b1", "db2": "b2"}
    h = 1e-6

    def loss(a):
        return float(np.sum(O.mlp_block(a["X"], a["W1"], a["W2"], a["b1"], a["b2"], "gelu", 2, 4) * dY))

    for gk, ak in names.items():
        base = args[ak]
        for idx in np.ndindex(base.shape):
            up, dn = base.copy(), base.copy()
            up[idx] += h
            dn[idx] -= h
            fd = (loss(dict(args, **{ak: up})) - loss(dict(args, **{ak: dn}))) / (2 * h)
            assert abs(g[gk][idx] - fd) < 1e-7 * max(1.0, abs(fd)), (gk, idx)


@pytest.mark.parametrize("Rb,Rm", [(1, 1), (2, 2), (4, 8), (8, 1)])
def test_mlp_backward_integer_exact_bitwise(Rb, Rm):
    """Identity activation on small integers: every gradient is an integer
    matrix product, exact in fp64 whatever the partition."""
    rng = np.random.default_rng(Rb * 16 + Rm)
    T, D, F = 32, 8, 64
    X, W1, W2, dY = ints(rng, (T, D)), ints(rng, (D, F)), ints(rng, (F, D)), ints(rng, (T, D))
    b1 = ints(rng, F)
    g = O.mlp_block_backward(X, W1, W2, dY, b1, "none", Rb, Rm)
    dZ = dY @ W2.T
    assert np.array_equal(g["dX"], dZ @ W1.T)
    assert np.array_equal(g["dW1"], X.T @ dZ)
    assert np.array_equal(g["dW2"], (X @ W1 + b1).T @ dY)
    assert np.array_equal(g["db1"], dZ.sum(axis=0))
    assert np.array_equal(g["db2"], dY.sum(axis=0))


def test_mlp_backward_sum_loops_visit_every_shard():
    """Each #sum loop adds exactly R terms: with the batch loop of 4 shards,
    scaling one shard's cotangent by 2 moves dW2 by that shard's term once."""
    X, W1, W2, dY, b1 = problem(6, T=16)
    base = O.mlp_block_backward(X, W1, W2, dY, b1, "gelu", 4, 2)
    dY2 = dY.copy()
    dY2[4:8] *= 2
    moved = O.mlp_block_backward(X, W1, W2, dY2, b1, "gelu", 4, 2)
    h = O.gelu_erf(X[4:8] @ W1 + b1)
    assert np.max(np.abs(moved["dW2"] - base["dW2"] - h.T @ dY[4:8])) < 1e-12
    assert np.max(np.abs(moved["db2"] - base["db2"] - dY[4:8].sum(axis=0))) < 1e-12


def test_mlp_backward_norms_bound_the_gradients():
    X, W1, W2, dY, b1 = problem(7)
    g, n = O.mlp_block_backward(X, W1, W2, dY, b1, "gelu", 2, 4, return_norm=True)
    for k in KEYS:
        assert n[k].shape == g[k].shape
        assert np.all(np.abs(g[k]) <= n[k] * (1 + 1e-12)), k
    # identity activation: the normalisers are plain |A|.|B| of each product
    g, n = O.mlp_block_backward(X, W1, W2, dY, b1, "none", 1, 1, return_norm=True)
    dZa = np.abs(dY) @ np.abs(W2).T
    assert np.allclose(n["dX"], dZa @ np.abs(W1).T, rtol=1e-13, atol=0)
    assert np.allclose(n["dW2"], (np.abs(X) @ np.abs(W1) + np.abs(b1)).T @ np.abs(dY), rtol=1e-13, atol=0)


def test_mlp_backward_norms_exact_on_nonnegative_operands():
    """Two-sided pin of the GELU-case normalisers: with X, W1, b1, W2, dY >= 0
    every |A||B| product equals AB, so each normaliser reduces to a closed
    form written here from plain definitions (scipy's normal cdf and pdf for
    GELU and its derivative): the dX, dW1, db1 normalisers exceed |grad| by
    exactly the first-order term dH * Z carried through the same product,
    and dW2's is (2 z Phi(z) + z^2 phi(z))^T dY.  An inflated or deflated
    normaliser fails."""
    from scipy.stats import norm
    rng = np.random.default_rng(31)
    T, D, F = 12, 6, 20
    X = rng.uniform(0.0, 1.5, (T, D))
    W1 = rng.uniform(0.0, 1.0, (D, F)) / math.sqrt(D)
    W2 = rng.uniform(0.0, 1.0, (F, D)) / math.sqrt(F)
    dY = rng.uniform(0.0, 1.0, (T, D))
    b1 = rng.uniform(0.0, 0.5, F)
    g, n = O.mlp_block_backward(X, W1, W2, dY, b1, "gelu", 2, 2, return_norm=True)
    z = X @ W1 + b1                      # >= 0
    dh = dY @ W2.T                       # >= 0
    gp = norm.cdf(z) + z * norm.pdf(z)   # GELU'(z) > 0 for z >= 0
    dz = dh * gp
    extra = dh * z                       # |dH| nZ with nZ = Z here
    assert np.allclose(g["dX"], dz @ W1.T, rtol=1e-12, atol=0)
    assert np.allclose(n["dX"], (dz + extra) @ W1.T, rtol=1e-12, atol=0)
    assert np.allclose(n["dW1"], X.T @ (dz + extra), rtol=1e-12, atol=0)
    assert np.allclose(n["db1"], (dz + extra).sum(axis=0), rtol=1e-12, atol=0)
    nh = 2.0 * z * norm.cdf(z) + z * z * norm.pdf(z)   # GELU'(z) z + GELU(z)
    assert np.allclose(n["dW2"], nh.T @ dY, rtol=1e-12, atol=0)
    assert np.allclose(n["db2"], dY.sum(axis=0), rtol=1e-13, atol=0)
    # the sampled loop nests (the full-size GPU tests' reference) give the
    # same normalisers at the rows and units they evaluate
    rows, units = [0, 5, 11], [1, 7, 19]
    _, sn = O.mlp_block_backward_sampled(X, W1, W2, dY, b1, "gelu", 2, 2, rows, units)
    assert np.allclose(sn["dX"], ((dz + extra) @ W1.T)[rows], rtol=1e-12, atol=0)
    assert np.allclose(sn["dW1"], (X.T @ (dz + extra))[:, units], rtol=1e-12, atol=0)
    assert np.allclose(sn["db1"], (dz + extra).sum(axis=0)[units], rtol=1e-12, atol=0)
    assert np.allclose(sn["dW2"], (nh.T @ dY)[units], rtol=1e-12, atol=0)


def test_mlp_backward_empty_sizes():
    rng = np.random.default_rng(9)
    D, F = 8, 16
    W1, W2 = rng.standard_normal((D, F)), rng.standard_normal((F, D))
    # no tokens: the weight gradients are empty sums over the batch
    g = O.mlp_block_backward(np.zeros((0, D)), W1, W2, np.zeros((0, D)), np.ones(F), "gelu", 2, 4)
    assert g["dX"].shape == (0, D)
    for k, shape in (("dW1", (D, F)), ("dW2", (F, D)), ("db1", (F,)), ("db2", (D,))):
        assert g[k].shape == shape and np.array_equal(g[k], np.zeros(shape))
    # no hidden units: dX is the empty sum over the model loop
    X, dY = rng.standard_normal((16, D)), rng.standard_normal((16, D))
    g = O.mlp_block_backward(X, np.zeros((D, 0)), np.zeros((0, D)), dY, None, "gelu", 2, 4)
    assert np.array_equal(g["dX"], np.zeros((16, D)))
    assert g["dW1"].shape == (D, 0) and g["dW2"].shape == (0, D) and g["db1"].shape == (0,)
    assert np.allclose(g["db2"], dY.sum(axis=0), rtol=1e-15, atol=1e-15)


def test_mlp_backward_rejects_indivisible():
    with pytest.raises(ValueError):
        O.mlp_block_backward(np.zeros((6, 2)), np.zeros((2, 8)), np.zeros((8, 2)), np.zeros((6, 2)), R_batch=4)
    with pytest.raises(ValueError):
        O.mlp_block_backward(np.zeros((8, 2)), np.zeros((2, 6)), np.zeros((6, 2)), np.zeros((8, 2)), R_model=4)


@pytest.mark.parametrize("act", ["gelu", "none"])
def test_mlp_backward_sampled_matches_full(act):
    """Entries evaluated one by one by their owning shards equal the full
    evaluation, normalisers included."""
    X, W1, W2, dY, b1 = problem(8, T=32, D=8, F=64)
    g, n = O.mlp_block_backward(X, W1, W2, dY, b1, act, 4, 8, return_norm=True)
    rows, units = [0, 7, 8, 31], [0, 7, 8, 63, 40]
    s, sn = O.mlp_block_backward_sampled(X, W1, W2, dY, b1, act, 4, 8, rows, units)
    pick = {"dX": (g["dX"][rows], n["dX"][rows]), "dW1": (g["dW1"][:, units], n["dW1"][:, units]),
            "dW2": (g["dW2"][units], n["dW2"][units]), "db1": (g["db1"][units], n["db1"][units]),
            "db2": (g["db2"], n["db2"])}
    for k, (val, nv) in pick.items():
        assert s[k].shape == val.shape
        assert np.max(np.abs(s[k] - val) / nv) < 1e-13, k
        assert np.max(np.abs(sn[k] - nv) / nv) < 1e-13, k


# ---------------------------------------------------------------------------
# attention core gradients
# ---------------------------------------------------------------------------
def attn_problem(seed, n=12, dh=4):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((n, dh)) for _ in range(4)]


@pytest.mark.parametrize("causal", [True, False])
def test_attention_backward_matches_torch_autograd(causal):
    q, k, v, do = attn_problem(20)
    scale = 0.5
    dq, dk, dv = O.attention_backward(q, k, v, do, scale, causal)
    ts = [torch.from_numpy(a.copy()).requires_grad_(True) for a in (q, k, v)]
    s = ts[0] @ ts[1].T * scale
    if causal:
        s = s.masked_fill(torch.triu(torch.ones(12, 12, dtype=torch.bool), 1), float("-inf"))
    (torch.softmax(s, dim=1) @ ts[2]).backward(torch.from_numpy(do))
    for got, t in zip((dq, dk, dv), ts):
        assert np.max(np.abs(got - t.grad.numpy())) < 1e-12


def test_attention_backward_central_differences():
    """<causal_attention(q, k, v), do> differentiated entry by entry."""
    q, k, v, do = attn_problem(21, n=6, dh=3)
    scale, h = 0.7, 1e-6
    g = O.attention_backward(q, k, v, do, scale, True)
    args = [q, k, v]
    loss = lambda a: float(np.sum(O.causal_attention(a[0], a[1], a[2], scale, True) * do))
    for which in range(3):
        for idx in np.ndindex(args[which].shape):
            up = [a.copy() for a in args]
            dn = [a.copy() for a in args]
            up[which][idx] += h
            dn[which][idx] -= h
            fd = (loss(up) - loss(dn)) / (2 * h)
            assert abs(g[which][idx] - fd) < 1e-7 * max(1.0, abs(fd)), (which, idx)


def test_attention_backward_closed_forms():
    q, k, v, do = attn_problem(22)
    # query 0 sees only key 0 (p = 1): its score gradient vanishes, so dq_0 = 0,
    # and dv gets do_0 in full from it
    dq, dk, dv = O.attention_backward(q, k, v, do, 0.3, True)
    assert np.max(np.abs(dq[0])) < 1e-15
    # the last key is seen only by the last query: dv_last = p_last,last do_last
    s = q[-1] @ k.T * 0.3
    p = np.exp(s - s.max())
    p /= p.sum()
    assert np.max(np.abs(dv[-1] - p[-1] * do[-1])) < 1e-14
    # a constant shift of v's rows changes o by the same constant: dq, dk unchanged
    dq2, dk2, _ = O.attention_backward(q, k, v + 5.0, do, 0.3, True)
    assert np.max(np.abs(dq2 - dq)) < 1e-11 and np.max(np.abs(dk2 - dk)) < 1e-11
    # softmax is shift-invariant along a row, so each row of ds sums to zero:
    # sum_j dk_j = scale sum_i (sum_j ds_ij) q_i = 0, and with all-equal keys
    # dq = scale ds k is zero
    kk = np.tile(k[:1], (12, 1))
    dq3, _, _ = O.attention_backward(q, kk, v, do, 0.3, False)
    assert np.max(np.abs(dq3)) < 1e-13
    assert np.max(np.abs(np.sum(dk, axis=0))) < 1e-12


def test_attention_backward_norms_bound():
    q, k, v, do = attn_problem(23, n=16, dh=8)
    (dq, dk, dv), (nq, nk, nv) = O.attention_backward(q, k, v, do, 0.35, True, return_norm=True)
    for g, n in ((dq, nq), (dk, nk), (dv, nv)):
        assert np.all(np.abs(g) <= n * (1 + 1e-12))


@pytest.mark.parametrize("causal", [True, False])
def test_attention_backward_norms_exact_on_nonnegative_operands(causal):
    """Two-sided pin of the attention-backward normalisers: with q, k, v,
    do >= 0 the magnitudes equal the values, so nv = dv exactly and nq, nk
    exceed dq, dk by exactly 2 scale (P * D) K and 2 scale (P * D)^T Q, with
    P = softmax(scale q k^T) (scipy) and D_i = sum_d do_id o_id, o = P v."""
    from scipy.special import softmax
    rng = np.random.default_rng(41)
    n, dh, scale = 10, 4, 0.4
    q, k, v, do = (rng.uniform(0.0, 1.0, (n, dh)) for _ in range(4))
    (dq, dk, dv), (nq, nk, nv) = O.attention_backward(q, k, v, do, scale, causal, return_norm=True)
    s = scale * (q @ k.T)
    if causal:
        s = np.where(np.tril(np.ones((n, n), bool)), s, -np.inf)
    P = softmax(s, axis=1)
    D = np.sum(do * (P @ v), axis=1, keepdims=True)
    assert np.allclose(nv, dv, rtol=1e-12, atol=0)
    assert np.allclose(nq, dq + 2.0 * scale * (P * D) @ k, rtol=1e-11, atol=1e-15)
    assert np.allclose(nk, dk + 2.0 * scale * (P * D).T @ q, rtol=1e-11, atol=1e-15)


# ---------------------------------------------------------------------------
# attention block gradients
# ---------------------------------------------------------------------------
def attn_block_problem(seed, B=2, S=4, H=2, dh=2):
    rng = np.random.default_rng(seed)
    D = H * dh
    X = rng.standard_normal((B * S, D))
    Ws = [rng.standard_normal((D, D)) / math.sqrt(D) for _ in range(4)]
    dY = rng.standard_normal((B * S, D))
    return X, Ws, dY


def torch_attn_block_grads(X, Ws, dY, B, S, H, dh, causal):
    ts = [torch.from_numpy(a.copy()).requires_grad_(True) for a in [X] + Ws]
    Xt, Wq, Wk, Wv, Wo = ts
    Q, K, V = Xt @ Wq, Xt @ Wk, Xt @ Wv
    A = torch.zeros_like(Q)
    outs = []
    for s in range(B):
        row = []
        for h in range(H):
            rs, cs = slice(s * S, (s + 1) * S), slice(h * dh, (h + 1) * dh)
            sc = Q[rs, cs] @ K[rs, cs].T / math.sqrt(dh)
            if causal:
                sc = sc.masked_fill(torch.triu(torch.ones(S, S, dtype=torch.bool), 1), float("-inf"))
            row.append(torch.softmax(sc, dim=1) @ V[rs, cs])
        outs.append(torch.cat(row, dim=1))
    A = torch.cat(outs, dim=0)
    (A @ Wo).backward(torch.from_numpy(dY))
    return {k: t.grad.numpy() for k, t in zip(("dX", "dWq", "dWk", "dWv", "dWo"), ts)}


@pytest.mark.parametrize("Rb,Rm", [(1, 1), (2, 2), (1, 2), (2, 1)])
@pytest.mark.parametrize("causal", [True, False])
def test_attn_block_backward_matches_torch_autograd(Rb, Rm, causal):
    B, S, H, dh = 2, 4, 2, 2
    X, Ws, dY = attn_block_problem(30 + Rb * 4 + Rm, B, S, H, dh)
    want = torch_attn_block_grads(X, Ws, dY, B, S, H, dh, causal)
    got = O.attn_block_backward(X, *Ws, dY, B, S, H, dh, causal, None, Rb, Rm)
    for k in want:
        assert got[k].shape == want[k].shape
        assert np.max(np.abs(got[k] - want[k])) < 1e-12, k


def test_attn_block_backward_central_differences():
    B, S, H, dh = 2, 3, 2, 2
    X, Ws, dY = attn_block_problem(31, B, S, H, dh)
    g = O.attn_block_backward(X, *Ws, dY, B, S, H, dh, True, None, 2, 2)
    args = [X] + Ws
    names = ("dX", "dWq", "dWk", "dWv", "dWo")
    loss = lambda a: float(np.sum(O.attn_block(a[0], a[1], a[2], a[3], a[4], B, S, H, dh, True, None, 2, 2) * dY))
    rng = np.random.default_rng(0)
    for which, key in enumerate(names):
        for _ in range(4):
            idx = tuple(int(rng.integers(n)) for n in args[which].shape)
            up = [a.copy() for a in args]
            dn = [a.copy() for a in args]
            up[which][idx] += 1e-6
            dn[which][idx] -= 1e-6
            fd = (loss(up) - loss(dn)) / 2e-6
            assert abs(g[key][idx] - fd) < 1e-7 * max(1.0, abs(fd)), (key, idx)


def test_attn_block_backward_norms_bound():
    B, S, H, dh = 2, 8, 4, 4
    X, Ws, dY = attn_block_problem(32, B, S, H, dh)
    g, n = O.attn_block_backward(X, *Ws, dY, B, S, H, dh, True, None, 2, 2, return_norm=True)
    for k in g:
        assert n[k].shape == g[k].shape
        assert np.all(np.abs(g[k]) <= n[k] * (1 + 1e-12)), k


def test_attn_block_backward_sampled_matches_full():
    B, S, H, dh = 4, 8, 4, 2
    X, Ws, dY = attn_block_problem(33, B, S, H, dh)
    g, n = O.attn_block_backward(X, *Ws, dY, B, S, H, dh, True, None, 2, 2, return_norm=True)
    seq, rows, head = 3, [0, 5, 7], 2
    sg, sn = O.attn_block_backward_sampled(X, *Ws, dY, B, S, H, dh, True, None, 2, 2, seq, rows, head)
    cs = slice(head * dh, (head + 1) * dh)
    pick = {"dX": (g["dX"][seq * S + np.array(rows)], n["dX"][seq * S + np.array(rows)]),
            "dWq": (g["dWq"][:, cs], n["dWq"][:, cs]), "dWk": (g["dWk"][:, cs], n["dWk"][:, cs]),
            "dWv": (g["dWv"][:, cs], n["dWv"][:, cs]), "dWo": (g["dWo"][cs], n["dWo"][cs])}
    for k, (val, nv) in pick.items():
        assert sg[k].shape == val.shape, k
        assert np.max(np.abs(sg[k] - val) / nv) < 1e-12, k
        assert np.max(np.abs(sn[k] - nv) / nv) < 1e-12, k

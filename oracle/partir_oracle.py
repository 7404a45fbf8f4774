"""Plain CPU oracle for loop-partitioned tensor programs (PartIR:Core semantics).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module; only the test suite, the smoke check and the CPU-baseline
leg of the benchmark do.  It shares no code with the HIP library.

What it computes
----------------
PartIR:Core (paper Sec. 5 and App. C, figure "Interpretation of PartIR:Core")
gives a denotational meaning to three constructs:

* ``slice d x[r]``  -- the r-th of n equal contiguous chunks of x along dim d,
  i.e. ``x[..., r*n_d:(r+1)*n_d, ...]`` with ``n_d = x.shape[d] / n`` (typing
  rule TSlice requires n to divide the dimension exactly);
* ``loop a [#tile<d>] e`` -- the direct sum (concatenation along dim d) of the
  body evaluated at r = 0..n-1 (typing rule TTile multiplies dim d by n);
* ``loop a [#sum] e`` -- the sum of the body over r = 0..n-1 (rule TSum keeps
  the type).

Any other op is evaluated by its plain definition.  This module evaluates the
loop nests of the partitioned programs *literally*, enumerating every virtual
shard (the "shard interpreter"), and separately evaluates the same programs
unpartitioned on whole tensors (the "unpartitioned evaluator").  By the
paper's correctness theorem for the lowering (App. C, theorem "correctness of
translation") and the matmul program equivalences (Sec. 5.2.1, figure
"matmul-examples"), both must agree up to rounding.

Arithmetic is float64 throughout.  Inputs arrive already decoded (exactly)
from their float32 / bfloat16 storage; no intermediate is rounded.  Library
primitives used as single steps: ``numpy.matmul`` (fp64 matrix product),
``numpy.exp``, ``numpy.sqrt`` and ``scipy.special.erf``.

Readings of the paper that this module fixes (where it is silent):
* the sum of a ``#sum`` loop is taken in increasing r;
* GELU is the exact erf form 0.5*x*(1+erf(x/sqrt 2));
* causal attention lets query i see keys j <= i of its own sequence, with
  scores scaled by ``scale`` and a max-subtracted softmax;
* RMSNorm is g * x / sqrt(mean(x^2) + eps) over the last dim;
* a bias of a ``#sum`` loop is added once, after the loop; a bias of a
  ``#tile`` loop is sliced with the tiled operand (add's tile-mapping entry
  needs both operands tiled alike, Sec. 5.2.1);
* weight matrices are passed in their logical [fan_in, fan_out] orientation.

Parity pins for every function here live in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import math
from typing import Callable, Optional, Sequence

import numpy as np
from scipy.special import erf as _erf

AXIS_NONE, AXIS_M, AXIS_N, AXIS_K = -1, 0, 1, 2


# ---------------------------------------------------------------------------
# PartIR:Core constructs (App. C, figure "Interpretation of PartIR:Core")
# ---------------------------------------------------------------------------
def slice_(x: np.ndarray, d: int, r: int, n: int) -> np.ndarray:
    """``slice d x[r]`` over an axis of size n (rule TSlice)."""
    size = x.shape[d]
    if n <= 0 or size % n != 0:
        raise ValueError(f"axis size {n} does not divide dim {d} of size {size}")
    if not 0 <= r < n:
        raise ValueError(f"range value {r} outside range<{n}>")
    nd = size // n
    index = [slice(None)] * x.ndim
    index[d] = slice(r * nd, (r + 1) * nd)
    return x[tuple(index)]


def loop_tile(n: int, d: int, body: Callable[[int], np.ndarray]) -> np.ndarray:
    """``loop a [#tile<d>] (r: range<n>) { body }``: direct sum along dim d."""
    parts = [body(r) for r in range(n)]
    return np.concatenate(parts, axis=d)


def loop_sum(n: int, body: Callable[[int], np.ndarray]) -> np.ndarray:
    """``loop a [#sum] (r: range<n>) { body }``: sum over r, r increasing."""
    acc = np.array(body(0), dtype=np.float64, copy=True)
    for r in range(1, n):
        acc = acc + body(r)
    return acc


# ---------------------------------------------------------------------------
# Plain ops (fp64)
# ---------------------------------------------------------------------------
def matmul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    return np.matmul(np.asarray(a, np.float64), np.asarray(b, np.float64))


def gelu_erf(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1.0 + _erf(x / math.sqrt(2.0)))


def activation(x: np.ndarray, act: str) -> np.ndarray:
    if act == "none":
        return np.asarray(x, np.float64)
    if act == "gelu":
        return gelu_erf(x)
    raise ValueError(f"unknown activation {act!r}")


def activation_grad(x: np.ndarray, act: str) -> np.ndarray:
    """d act(x) / dx.  GELU-erf is x Phi(x), so by the product rule its
    derivative is Phi(x) + x phi(x) with phi the standard normal density."""
    x = np.asarray(x, np.float64)
    if act == "none":
        return np.ones_like(x)
    if act == "gelu":
        cdf = 0.5 * (1.0 + _erf(x / math.sqrt(2.0)))
        pdf = np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
        return cdf + x * pdf
    raise ValueError(f"unknown activation {act!r}")


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    x = np.asarray(x, np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return np.asarray(g, np.float64) * x / np.sqrt(ms + eps)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                     causal: bool = True, q_pos: Optional[np.ndarray] = None) -> np.ndarray:
    """Softmax attention of one head of one sequence.

    q: [nq, dh] queries at positions ``q_pos`` (default 0..nq-1);
    k, v: [nk, dh] keys/values at positions 0..nk-1.
    o_i = sum_j p_ij v_j with p_ij = exp(s_ij - max_j s_ij) / sum_j(...),
    s_ij = scale * q_i . k_j over keys j <= pos(i) when causal.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    if q_pos is None:
        q_pos = np.arange(q.shape[0])
    s = matmul(q, k.T) * scale
    if causal:
        key_pos = np.arange(k.shape[0])
        s = np.where(key_pos[None, :] <= np.asarray(q_pos)[:, None], s, -np.inf)
    m = np.max(s, axis=1, keepdims=True)
    p = np.exp(s - m)
    p = p / np.sum(p, axis=1, keepdims=True)
    return matmul(p, v)


def attention_backward(q, k, v, do, scale: float, causal: bool = True, return_norm: bool = False):
    """Gradients of o = causal_attention(q, k, v) for the cotangent do, one
    head of one sequence (positions 0..n-1), by the chain rule through
    s = scale q k^T, p = softmax_rows(s), o = p v:

      dv = p^T do;  dp = do v^T;  ds = p * (dp - rowsum(do * o));
      dq = scale ds k;  dk = scale ds^T q.

    (rowsum(do * o)_i = sum_j p_ij dp_ij: the softmax Jacobian applied to dp.)
    With return_norm also first-order error normalisers: for each gradient
    its last product with ds replaced by p * (|do||v|^T + rowsum|do * o|)
    (the magnitude of dp - D) and every other operand by its magnitude.
    Returns (dq, dk, dv) or ((dq, dk, dv), (nq, nk, nv)).
    """
    q, k, v, do = (np.asarray(a, np.float64) for a in (q, k, v, do))
    n = q.shape[0]
    s = matmul(q, k.T) * scale
    if causal:
        pos = np.arange(n)
        s = np.where(pos[None, :] <= pos[:, None], s, -np.inf)
    p = np.exp(s - np.max(s, axis=1, keepdims=True))
    p = p / np.sum(p, axis=1, keepdims=True)
    o = matmul(p, v)
    dv = matmul(p.T, do)
    dp = matmul(do, v.T)
    d = np.sum(do * o, axis=1, keepdims=True)
    ds = p * (dp - d)
    dq = scale * matmul(ds, k)
    dk = scale * matmul(ds.T, q)
    if not return_norm:
        return dq, dk, dv
    nds = p * (abs_product(do, v.T) + np.sum(np.abs(do * o), axis=1, keepdims=True))
    return (dq, dk, dv), (scale * matmul(nds, np.abs(k)), scale * matmul(nds.T, np.abs(q)),
                          matmul(p.T, np.abs(do)))


# ---------------------------------------------------------------------------
# The key axis as a loop: a custom associative #sum (Sec. 5.2.1 footnote)
# ---------------------------------------------------------------------------
def softmax_partial(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, causal: bool,
                    q_pos: np.ndarray, k_pos: np.ndarray):
    """One key shard of softmax attention, per query: (m, l, o) with
    m = max_j s_ij over the keys j of the shard the query may see,
    l = sum_j exp(s_ij - m), o = sum_j exp(s_ij - m) v_j.  A query that sees
    no key of the shard gets (-inf, 0, 0), the identity of the combiner."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    s = matmul(q, k.T) * scale
    if causal:
        s = np.where(np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None], s, -np.inf)
    m = np.max(s, axis=1) if s.shape[1] else np.full(s.shape[0], -np.inf)
    seen = np.isfinite(m)
    e = np.where(seen[:, None], np.exp(s - np.where(seen, m, 0.0)[:, None]), 0.0)
    return m, e.sum(axis=1), matmul(e, v)


def softmax_combine(a, b):
    """(m, l, o) (+) (m', l', o') = (M, e^(m-M) l + e^(m'-M) l', e^(m-M) o + e^(m'-M) o'),
    M = max(m, m'); a shard with m = -inf carries weight 0."""
    (m1, l1, o1), (m2, l2, o2) = a, b
    M = np.maximum(m1, m2)
    w1 = np.where(np.isfinite(m1), np.exp(m1 - np.where(np.isfinite(M), M, 0.0)), 0.0)
    w2 = np.where(np.isfinite(m2), np.exp(m2 - np.where(np.isfinite(M), M, 0.0)), 0.0)
    return M, w1 * l1 + w2 * l2, w1[:, None] * o1 + w2[:, None] * o2


def attention_split_kv(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, causal: bool, R: int,
                       q_pos: Optional[np.ndarray] = None) -> np.ndarray:
    """loop s [#sum softmax](R) { softmax_partial(q, slice 0 k[s], slice 0 v[s]) },
    folded with softmax_combine in shard order, then o / l."""
    nk = k.shape[0]
    if q_pos is None:
        q_pos = np.arange(q.shape[0])
    acc = None
    for r in range(R):
        pos = np.arange(r * (nk // R), (r + 1) * (nk // R))
        part = softmax_partial(q, slice_(k, 0, r, R), slice_(v, 0, r, R), scale, causal, q_pos, pos)
        acc = part if acc is None else softmax_combine(acc, part)
    return acc[2] / acc[1][:, None]


# ---------------------------------------------------------------------------
# Single partitioned matmul: the three TMR forms of matmul (Sec. 5.2.1)
# ---------------------------------------------------------------------------
def loop_matmul(A: np.ndarray, B: np.ndarray, tile_axis: int, sum_axis: int, R: int) -> np.ndarray:
    """C = A @ B written as a loop over R virtual shards.

    tile_axis M: ``loop [#tile<0>] { matmul(slice 0 A[r], B) }``
    tile_axis N: ``loop [#tile<1>] { matmul(A, slice 1 B[r]) }``
    sum_axis  K: ``loop [#sum]     { matmul(slice 1 A[r], slice 0 B[r]) }``
    tile and sum together: the tile loop outside, the sum loop inside, over two
    distinct axes of size R each (nested loops over one axis are forbidden,
    Sec. 5.2.3).
    """
    if tile_axis not in (AXIS_NONE, AXIS_M, AXIS_N):
        raise ValueError("tile_axis must be NONE, M or N")
    if sum_axis not in (AXIS_NONE, AXIS_K):
        raise ValueError("sum_axis must be NONE or K")

    def summed(a, b):
        if sum_axis == AXIS_K:
            return loop_sum(R, lambda r: matmul(slice_(a, 1, r, R), slice_(b, 0, r, R)))
        return matmul(a, b)

    if tile_axis == AXIS_M:
        return loop_tile(R, 0, lambda r: summed(slice_(A, 0, r, R), B))
    if tile_axis == AXIS_N:
        return loop_tile(R, 1, lambda r: summed(A, slice_(B, 1, r, R)))
    return summed(A, B)


def abs_product(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """|A|.|B|: the elementwise error normaliser of a product (Higham Sec. 3.5)."""
    return matmul(np.abs(A), np.abs(B))


# ---------------------------------------------------------------------------
# Megatron MLP block, optionally nested in a batch #tile
# ---------------------------------------------------------------------------
def mlp_block(X, W1, W2, b1=None, b2=None, act="gelu", R_batch=1, R_model=1,
              rows: Optional[Sequence[int]] = None, return_norm=False):
    """Y = loop b [#tile<0>](R_batch) { loop m [#sum](R_model) {
              act(slice 0 X[b] @ slice 1 W1[m] + slice 0 b1[m]) @ slice 0 W2[m] } + b2 }

    X [T, D], W1 [D, F], W2 [F, D], b1 [F] or None, b2 [D] or None.
    ``rows``: evaluate only these output rows (each row is computed by the batch
    shard that owns it, exactly as in the full evaluation).
    With ``return_norm`` also returns the normaliser |H|.|W2| (+|b2|) of the
    last contraction.
    """
    T = X.shape[0]
    F = W1.shape[1]
    sel = np.arange(T) if rows is None else np.asarray(rows)
    out = np.zeros((len(sel), W2.shape[1]))
    norm = np.zeros_like(out)
    Tb = T // R_batch
    if T % R_batch or F % R_model:
        raise ValueError("indivisible partition")
    for b in range(R_batch):
        xb = slice_(X, 0, b, R_batch)
        mine = [(i, r - b * Tb) for i, r in enumerate(sel) if b * Tb <= r < (b + 1) * Tb]
        if not mine:
            continue
        local = np.array([t for _, t in mine])
        xr = xb[local]

        def shard(m):
            h = matmul(xr, slice_(W1, 1, m, R_model))
            if b1 is not None:
                h = h + slice_(np.asarray(b1), 0, m, R_model)
            h = activation(h, act)
            w2 = slice_(W2, 0, m, R_model)
            return matmul(h, w2), (abs_product(h, w2) if return_norm else None)

        parts = [shard(m) for m in range(R_model)]
        y = loop_sum(R_model, lambda m: parts[m][0])
        nrm = loop_sum(R_model, lambda m: parts[m][1]) if return_norm else None
        if b2 is not None:
            y = y + np.asarray(b2, np.float64)
            if return_norm:
                nrm = nrm + np.abs(np.asarray(b2, np.float64))
        idx = np.array([i for i, _ in mine])
        out[idx] = y
        if return_norm:
            norm[idx] = nrm
    return (out, norm) if return_norm else out


def mlp_ref(X, W1, W2, b1=None, b2=None, act="gelu"):
    """Unpartitioned MLP: act(X W1 + b1) W2 + b2."""
    h = matmul(X, W1)
    if b1 is not None:
        h = h + b1
    y = matmul(activation(h, act), W2)
    if b2 is not None:
        y = y + b2
    return y


def mlp_block_backward(X, W1, W2, dY, b1=None, act="gelu", R_batch=1, R_model=1, return_norm=False):
    """Gradients of mlp_block for the output cotangent dY, as loop nests over
    the same batch (b, R_batch) and model (m, R_model) shards as the forward.

    Reverse-mode differentiation of a partitioned program is again a
    partitioned program (the paper partitions whole training steps, Sec. 7):
    every product of the backward pass is a matmul whose operands are sliced
    exactly as the matmul tile-mapping entries of Sec. 5.2.1 demand, so a
    gradient that contracts over a sliced dimension is a #sum loop:

      Z[b][:, m]  = slice 0 X[b] @ slice 1 W1[m] + slice 0 b1[m]      (recomputed)
      dH[b][:, m] = slice 0 dY[b] @ (slice 0 W2[m])^T
      dZ[b][:, m] = dH[b][:, m] * act'(Z[b][:, m])
      dW2 = loop m [#tile<0>] { loop b [#sum] { act(Z[b][:, m])^T @ slice 0 dY[b] } }
      dW1 = loop m [#tile<1>] { loop b [#sum] { (slice 0 X[b])^T @ dZ[b][:, m] } }
      dX  = loop b [#tile<0>] { loop m [#sum] { dZ[b][:, m] @ (slice 1 W1[m])^T } }
      db1 = loop m [#tile<0>] { loop b [#sum] { column sums of dZ[b][:, m] } }
      db2 = loop b [#sum] { column sums of slice 0 dY[b] }

    X [T, D], W1 [D, F], W2 [F, D], dY [T, D], b1 [F] or None.  Returns a dict
    with dX [T, D], dW1 [D, F], dW2 [F, D], db1 [F], db2 [D].  With
    ``return_norm`` also a dict of elementwise normalisers: each gradient's
    last contraction with every operand replaced by a first-order bound on
    its own magnitude and error sensitivity (see mlp_backward_norms).
    """
    T = X.shape[0]
    F = W1.shape[1]
    if T % R_batch or F % R_model:
        raise ValueError("indivisible partition")
    b1v = None if b1 is None else np.asarray(b1, np.float64)
    shard = {}
    for b in range(R_batch):
        xb, dyb = slice_(X, 0, b, R_batch), slice_(dY, 0, b, R_batch)
        for m in range(R_model):
            z = matmul(xb, slice_(W1, 1, m, R_model))
            if b1v is not None:
                z = z + slice_(b1v, 0, m, R_model)
            dh = matmul(dyb, slice_(W2, 0, m, R_model).T)
            dz = dh * activation_grad(z, act)
            shard[b, m] = dict(x=xb, dy=dyb, z=z, h=activation(z, act), dh=dh, dz=dz)
    w1 = lambda m: slice_(W1, 1, m, R_model)
    g = {
        "dW2": loop_tile(R_model, 0, lambda m: loop_sum(
            R_batch, lambda b: matmul(shard[b, m]["h"].T, shard[b, m]["dy"]))),
        "dW1": loop_tile(R_model, 1, lambda m: loop_sum(
            R_batch, lambda b: matmul(shard[b, m]["x"].T, shard[b, m]["dz"]))),
        "dX": loop_tile(R_batch, 0, lambda b: loop_sum(
            R_model, lambda m: matmul(shard[b, m]["dz"], w1(m).T))),
        "db1": loop_tile(R_model, 0, lambda m: loop_sum(
            R_batch, lambda b: np.sum(shard[b, m]["dz"], axis=0))),
        "db2": loop_sum(R_batch, lambda b: np.sum(shard[b, 0]["dy"], axis=0)),
    }
    if not return_norm:
        return g
    return g, mlp_backward_norms(X, W1, W2, dY, b1, act)


def mlp_block_backward_sampled(X, W1, W2, dY, b1=None, act="gelu", R_batch=1, R_model=1,
                               rows=(), units=()):
    """The loop nests of mlp_block_backward evaluated only where asked, each
    entry by the shards that own it: dX at token ``rows`` (batch shard b of
    the row, #sum over every model shard m) and, at hidden ``units`` f (model
    shard m of the unit, #sum over every batch shard b), dW1[:, f], dW2[f, :]
    and db1[f]; db2 in full.  Returns (values, normalisers), both dicts with
    dX [len(rows), D], dW1 [D, len(units)], dW2 [len(units), D],
    db1 [len(units)], db2 [D].
    """
    T, D = X.shape
    F = W1.shape[1]
    if T % R_batch or F % R_model:
        raise ValueError("indivisible partition")
    X, W1, W2, dY = (np.asarray(a, np.float64) for a in (X, W1, W2, dY))
    b1v = np.zeros(F) if b1 is None else np.asarray(b1, np.float64)
    Tb, Fm = T // R_batch, F // R_model
    rows, units = np.asarray(rows, int), np.asarray(units, int)

    def unit_grads(x, dy, w1, b1s, w2):
        """z, h, dz of one shard's tokens x over one shard's hidden units."""
        z = matmul(x, w1) + b1s
        dh = matmul(dy, w2.T)
        return z, activation(z, act), dh, dh * activation_grad(z, act)

    out = {"dX": np.zeros((len(rows), D)), "dW1": np.zeros((D, len(units))),
           "dW2": np.zeros((len(units), D)), "db1": np.zeros(len(units))}
    nrm = {k: np.zeros_like(v) for k, v in out.items()}
    for i, t in enumerate(rows):
        b = t // Tb
        x, dy = slice_(X, 0, b, R_batch)[t - b * Tb][None], slice_(dY, 0, b, R_batch)[t - b * Tb][None]

        def shard(m):
            w1, w2 = slice_(W1, 1, m, R_model), slice_(W2, 0, m, R_model)
            z, _, dh, dz = unit_grads(x, dy, w1, slice_(b1v, 0, m, R_model), w2)
            n = _dz_norm(x, dy, w1, slice_(b1v, 0, m, R_model), w2, z, dh, act)
            return matmul(dz, w1.T)[0], matmul(n, np.abs(w1).T)[0]

        parts = [shard(m) for m in range(R_model)]
        out["dX"][i] = loop_sum(R_model, lambda m: parts[m][0])
        nrm["dX"][i] = loop_sum(R_model, lambda m: parts[m][1])
    for j, f in enumerate(units):
        m = f // Fm
        w1, w2 = slice_(W1, 1, m, R_model)[:, [f - m * Fm]], slice_(W2, 0, m, R_model)[[f - m * Fm]]
        b1s = slice_(b1v, 0, m, R_model)[[f - m * Fm]]

        def shard(b):
            x, dy = slice_(X, 0, b, R_batch), slice_(dY, 0, b, R_batch)
            z, h, dh, dz = unit_grads(x, dy, w1, b1s, w2)
            ndz = _dz_norm(x, dy, w1, b1s, w2, z, dh, act)
            nh = abs_product(x, w1) + np.abs(b1s)
            if act != "none":
                nh = np.abs(activation_grad(z, act)) * nh + np.abs(h)
            return (matmul(x.T, dz)[:, 0], matmul(h.T, dy)[0], np.sum(dz),
                    matmul(np.abs(x).T, ndz)[:, 0], matmul(nh.T, np.abs(dy))[0], np.sum(ndz))

        parts = [shard(b) for b in range(R_batch)]
        for k, key in enumerate(("dW1", "dW2", "db1")):
            val = loop_sum(R_batch, lambda b: np.asarray(parts[b][k]))
            nv = loop_sum(R_batch, lambda b: np.asarray(parts[b][k + 3]))
            if key == "dW1":
                out[key][:, j], nrm[key][:, j] = val, nv
            else:
                out[key][j], nrm[key][j] = val, nv
    out["db2"] = loop_sum(R_batch, lambda b: np.sum(slice_(dY, 0, b, R_batch), axis=0))
    nrm["db2"] = loop_sum(R_batch, lambda b: np.sum(np.abs(slice_(dY, 0, b, R_batch)), axis=0))
    return out, nrm


def _dz_norm(x, dy, w1, b1s, w2, z, dh, act):
    """First-order normaliser of dZ for one shard (mlp_backward_norms)."""
    ndh = abs_product(dy, w2.T)
    if act == "none":
        return ndh
    nz = abs_product(x, w1) + np.abs(b1s)
    return ndh * np.abs(activation_grad(z, act)) + np.abs(dh) * nz


def mlp_backward_norms(X, W1, W2, dY, b1=None, act="gelu"):
    """Elementwise error normalisers for the MLP gradients, by first-order
    error propagation through the unpartitioned backward pass:

      nZ  = |X| |W1| + |b1|                  (normaliser of Z's contraction)
      ndH = |dY| |W2|^T
      ndZ = ndH |act'(Z)| + |dH| nZ          (sup |GELU''| = 2 phi(0) < 1)
      nH  = |act'(Z)| nZ + |act(Z)|
      dW2: nH^T |dY|,  dW1: |X|^T ndZ,  dX: ndZ |W1|^T,
      db1: column sums of ndZ,  db2: column sums of |dY|.
    For the identity activation ndZ = ndH and nH = nZ.
    """
    nz = abs_product(X, W1)
    z = matmul(X, W1)
    if b1 is not None:
        nz = nz + np.abs(np.asarray(b1, np.float64))
        z = z + np.asarray(b1, np.float64)
    ndh = abs_product(dY, np.asarray(W2, np.float64).T)
    dh = matmul(dY, np.asarray(W2, np.float64).T)
    if act == "none":
        ndz, nh = ndh, nz
    else:
        gp = np.abs(activation_grad(z, act))
        ndz = ndh * gp + np.abs(dh) * nz
        nh = gp * nz + np.abs(activation(z, act))
    return {"dW2": matmul(nh.T, np.abs(dY)), "dW1": matmul(np.abs(X).T, ndz),
            "dX": matmul(ndz, np.abs(W1).T), "db1": np.sum(ndz, axis=0),
            "db2": np.sum(np.abs(np.asarray(dY, np.float64)), axis=0)}


def mlp_backward_ref(X, W1, W2, dY, b1=None, act="gelu"):
    """Unpartitioned gradients of act(X W1 + b1) W2 + b2 for cotangent dY."""
    z = matmul(X, W1)
    if b1 is not None:
        z = z + np.asarray(b1, np.float64)
    dz = matmul(dY, np.asarray(W2, np.float64).T) * activation_grad(z, act)
    return {"dW2": matmul(activation(z, act).T, dY), "dW1": matmul(np.asarray(X, np.float64).T, dz),
            "dX": matmul(dz, np.asarray(W1, np.float64).T), "db1": np.sum(dz, axis=0),
            "db2": np.sum(np.asarray(dY, np.float64), axis=0)}


# ---------------------------------------------------------------------------
# Attention block: heads #tile inside a Megatron #sum, in a batch #tile
# ---------------------------------------------------------------------------
def _attend_shard(xb, Wq_m, Wk_m, Wv_m, n_seq, S, heads, d_head, scale, causal, sel_local):
    """Heads-#tile loop of one model shard over the sequences of one batch shard.

    Returns the attention output rows ``sel_local`` ([n_sel, heads*d_head]).
    For each sequence only its key prefix up to the largest selected position is
    projected (keys beyond it are masked for every selected query)."""
    out = np.zeros((len(sel_local), heads * d_head))
    for s in range(n_seq):
        mine = [(i, t - s * S) for i, t in enumerate(sel_local) if s * S <= t < (s + 1) * S]
        if not mine:
            continue
        pos = np.array([p for _, p in mine])
        nk = (int(pos.max()) + 1) if causal else S
        xs = xb[s * S: s * S + nk]
        q_rows = xs[pos]
        Q = matmul(q_rows, Wq_m)
        K = matmul(xs, Wk_m)
        V = matmul(xs, Wv_m)
        o = loop_tile(heads, 1, lambda h: causal_attention(
            slice_(Q, 1, h, heads), slice_(K, 1, h, heads), slice_(V, 1, h, heads),
            scale, causal, q_pos=pos))
        out[np.array([i for i, _ in mine])] = o
    return out


def attn_block(X, Wq, Wk, Wv, Wo, B, S, n_heads, d_head, causal=True, scale=None,
               R_batch=1, R_model=1, rows=None, return_norm=False):
    """Y = loop b [#tile<0>](R_batch) { loop m [#sum](R_model) {
              (loop h [#tile<1>](heads/R_model) { attn(q_h, k_h, v_h) }) @ slice 0 Wo[m] } }
    with q = slice 0 X[b] @ slice 1 Wq[m] (and k, v likewise); X is [B*S, D]
    sequence-major.  Batch shards hold whole sequences."""
    if scale is None:
        scale = 1.0 / math.sqrt(d_head)
    T, D = X.shape
    if T != B * S or n_heads * d_head != Wq.shape[1]:
        raise ValueError("shape mismatch")
    if B % R_batch or n_heads % R_model:
        raise ValueError("indivisible partition")
    sel = np.arange(T) if rows is None else np.asarray(rows)
    out = np.zeros((len(sel), Wo.shape[1]))
    norm = np.zeros_like(out)
    Tb = T // R_batch
    hps = n_heads // R_model
    for b in range(R_batch):
        xb = slice_(X, 0, b, R_batch)
        mine = [(i, r - b * Tb) for i, r in enumerate(sel) if b * Tb <= r < (b + 1) * Tb]
        if not mine:
            continue
        local = np.array([t for _, t in mine])

        def shard(m):
            a = _attend_shard(xb, slice_(Wq, 1, m, R_model), slice_(Wk, 1, m, R_model),
                              slice_(Wv, 1, m, R_model), B // R_batch, S, hps, d_head,
                              scale, causal, local)
            wo = slice_(Wo, 0, m, R_model)
            return matmul(a, wo), (abs_product(a, wo) if return_norm else None)

        parts = [shard(m) for m in range(R_model)]
        y = loop_sum(R_model, lambda m: parts[m][0])
        idx = np.array([i for i, _ in mine])
        out[idx] = y
        if return_norm:
            norm[idx] = loop_sum(R_model, lambda m: parts[m][1])
    return (out, norm) if return_norm else out


def attn_ref(X, Wq, Wk, Wv, Wo, B, S, n_heads, d_head, causal=True, scale=None):
    """Unpartitioned attention block on whole tensors."""
    if scale is None:
        scale = 1.0 / math.sqrt(d_head)
    Q, K, V = matmul(X, Wq), matmul(X, Wk), matmul(X, Wv)
    A = np.zeros_like(Q)
    for s in range(B):
        rs = slice(s * S, (s + 1) * S)
        for h in range(n_heads):
            cs = slice(h * d_head, (h + 1) * d_head)
            A[rs, cs] = causal_attention(Q[rs, cs], K[rs, cs], V[rs, cs], scale, causal)
    return matmul(A, Wo)


def attn_block_backward(X, Wq, Wk, Wv, Wo, dY, B, S, n_heads, d_head, causal=True, scale=None,
                        R_batch=1, R_model=1, return_norm=False):
    """Gradients of attn_block for the output cotangent dY, as loop nests over
    the forward's batch (b) and model (m, heads) shards:

      q|k|v[b, m] = slice 0 X[b] @ slice 1 W{q,k,v}[m];  a[b, m] = heads' attention
      dA[b, m]    = slice 0 dY[b] @ (slice 0 Wo[m])^T          (#tile<0> b, #tile<1> m)
      dq|dk|dv[b, m] = per (sequence, head) attention_backward(q, k, v, dA)
      dX  = loop b [#tile<0>] { loop m [#sum] { dq Wq[m]^T + dk Wk[m]^T + dv Wv[m]^T } }
      dWq = loop m [#tile<1>] { loop b [#sum] { (slice 0 X[b])^T dq[b, m] } }  (k, v alike)
      dWo = loop m [#tile<0>] { loop b [#sum] { a[b, m]^T slice 0 dY[b] } }

    Weights in their logical [fan_in, fan_out] orientation.  Returns a dict
    dX, dWq, dWk, dWv, dWo; with return_norm also a dict of normalisers that
    propagate magnitudes through the same nests (attention_backward's bounds
    with dA replaced by |dY| |Wo|^T, the attention output by p |v|).
    """
    if scale is None:
        scale = 1.0 / math.sqrt(d_head)
    T, D = X.shape
    if T != B * S or n_heads * d_head != Wq.shape[1]:
        raise ValueError("shape mismatch")
    if B % R_batch or n_heads % R_model:
        raise ValueError("indivisible partition")
    X, Wq, Wk, Wv, Wo, dY = (np.asarray(a, np.float64) for a in (X, Wq, Wk, Wv, Wo, dY))
    nseq, hps = B // R_batch, n_heads // R_model
    sh = {}
    for b in range(R_batch):
        xb, dyb = slice_(X, 0, b, R_batch), slice_(dY, 0, b, R_batch)
        for m in range(R_model):
            w = [slice_(W, 1, m, R_model) for W in (Wq, Wk, Wv)]
            wo = slice_(Wo, 0, m, R_model)
            q, k, v = (matmul(xb, wi) for wi in w)
            da = matmul(dyb, wo.T)
            nda = abs_product(dyb, wo.T)
            grads = [np.zeros_like(q) for _ in range(3)]
            norms = [np.zeros_like(q) for _ in range(3)]
            a, na = np.zeros_like(q), np.zeros_like(q)
            for sq in range(nseq):
                rs = slice(sq * S, (sq + 1) * S)
                for hh in range(hps):
                    cs = slice(hh * d_head, (hh + 1) * d_head)
                    a[rs, cs] = causal_attention(q[rs, cs], k[rs, cs], v[rs, cs], scale, causal)
                    na[rs, cs] = causal_attention(q[rs, cs], k[rs, cs], np.abs(v[rs, cs]), scale, causal)
                    g = attention_backward(q[rs, cs], k[rs, cs], v[rs, cs], da[rs, cs], scale, causal)
                    _, n = attention_backward(q[rs, cs], k[rs, cs], v[rs, cs], nda[rs, cs], scale, causal,
                                              return_norm=True)
                    for i in range(3):
                        grads[i][rs, cs] = g[i]
                        norms[i][rs, cs] = n[i]
            sh[b, m] = dict(x=xb, dy=dyb, w=w, a=a, na=na, g=grads, n=norms)
    out = {
        "dX": loop_tile(R_batch, 0, lambda b: loop_sum(R_model, lambda m: sum(
            matmul(sh[b, m]["g"][i], sh[b, m]["w"][i].T) for i in range(3)))),
        "dWo": loop_tile(R_model, 0, lambda m: loop_sum(R_batch, lambda b: matmul(sh[b, m]["a"].T, sh[b, m]["dy"]))),
    }
    for i, key in enumerate(("dWq", "dWk", "dWv")):
        out[key] = loop_tile(R_model, 1, lambda m, i=i: loop_sum(
            R_batch, lambda b: matmul(sh[b, m]["x"].T, sh[b, m]["g"][i])))
    if not return_norm:
        return out
    nrm = {
        "dX": loop_tile(R_batch, 0, lambda b: loop_sum(R_model, lambda m: sum(
            abs_product(sh[b, m]["n"][i], sh[b, m]["w"][i].T) for i in range(3)))),
        "dWo": loop_tile(R_model, 0, lambda m: loop_sum(R_batch, lambda b: matmul(sh[b, m]["na"].T,
                                                                                 np.abs(sh[b, m]["dy"])))),
    }
    for i, key in enumerate(("dWq", "dWk", "dWv")):
        nrm[key] = loop_tile(R_model, 1, lambda m, i=i: loop_sum(
            R_batch, lambda b: abs_product(sh[b, m]["x"].T, sh[b, m]["n"][i])))
    return out, nrm


def attn_block_backward_sampled(X, Wq, Wk, Wv, Wo, dY, B, S, n_heads, d_head, causal=True, scale=None,
                                R_batch=1, R_model=1, seq=0, rows=(), head=0):
    """The nests of attn_block_backward evaluated only where asked, each entry
    through the shards that own it: dX at positions ``rows`` of sequence
    ``seq`` (its batch shard; #sum over every model shard and head), and the
    weight gradients of one ``head`` (its model shard; #sum over every batch
    shard): dWq|dWk|dWv[:, head columns] and dWo[head rows, :].  Returns
    (values, normalisers) as dicts with dX [len(rows), D], dWq/dWk/dWv
    [D, d_head], dWo [d_head, D]."""
    if scale is None:
        scale = 1.0 / math.sqrt(d_head)
    T, D = X.shape
    if B % R_batch or n_heads % R_model:
        raise ValueError("indivisible partition")
    X, Wq, Wk, Wv, Wo, dY = (np.asarray(a, np.float64) for a in (X, Wq, Wk, Wv, Wo, dY))
    Tb, hps, nseq = T // R_batch, n_heads // R_model, B // R_batch
    rows = np.asarray(rows, int)

    def head_grads(xs, dys, m, hh):
        """One (sequence, head) of model shard m: attention inputs and gradients."""
        cs = slice(hh * d_head, (hh + 1) * d_head)
        w = [slice_(W, 1, m, R_model)[:, cs] for W in (Wq, Wk, Wv)]
        wo = slice_(Wo, 0, m, R_model)[cs]
        q, k, v = (matmul(xs, wi) for wi in w)
        da, nda = matmul(dys, wo.T), abs_product(dys, wo.T)
        g = attention_backward(q, k, v, da, scale, causal)
        _, n = attention_backward(q, k, v, nda, scale, causal, return_norm=True)
        a = causal_attention(q, k, v, scale, causal)
        na = causal_attention(q, k, np.abs(v), scale, causal)
        return w, g, n, a, na

    # dX rows: batch shard of the sequence, #sum over model shards and their heads
    b = seq // nseq
    xb, dyb = slice_(X, 0, b, R_batch), slice_(dY, 0, b, R_batch)
    sl = slice((seq - b * nseq) * S, (seq - b * nseq + 1) * S)
    xs, dys = xb[sl], dyb[sl]

    def dx_shard(m):
        val, nv = np.zeros((len(rows), D)), np.zeros((len(rows), D))
        for hh in range(hps):
            w, g, n, _, _ = head_grads(xs, dys, m, hh)
            for i in range(3):
                val += matmul(g[i][rows], w[i].T)
                nv += abs_product(n[i][rows], w[i].T)
        return val, nv

    parts = [dx_shard(m) for m in range(R_model)]
    out = {"dX": loop_sum(R_model, lambda m: parts[m][0])}
    nrm = {"dX": loop_sum(R_model, lambda m: parts[m][1])}
    # weight gradients of one head: its model shard, #sum over batch shards
    m, hh = head // hps, head % hps

    def w_shard(bb):
        xbb, dybb = slice_(X, 0, bb, R_batch), slice_(dY, 0, bb, R_batch)
        acc = [np.zeros((D, d_head)) for _ in range(3)] + [np.zeros((d_head, D))]
        nac = [np.zeros((D, d_head)) for _ in range(3)] + [np.zeros((d_head, D))]
        for sq in range(nseq):
            rs = slice(sq * S, (sq + 1) * S)
            _, g, n, a, na = head_grads(xbb[rs], dybb[rs], m, hh)
            for i in range(3):
                acc[i] += matmul(xbb[rs].T, g[i])
                nac[i] += abs_product(xbb[rs].T, n[i])
            acc[3] += matmul(a.T, dybb[rs])
            nac[3] += matmul(na.T, np.abs(dybb[rs]))
        return acc, nac

    wp = [w_shard(bb) for bb in range(R_batch)]
    for i, key in enumerate(("dWq", "dWk", "dWv", "dWo")):
        out[key] = loop_sum(R_batch, lambda bb: wp[bb][0][i])
        nrm[key] = loop_sum(R_batch, lambda bb: wp[bb][1][i])
    return out, nrm


# ---------------------------------------------------------------------------
# Pre-norm decoder layer / stack (residual stream kept unrounded)
# ---------------------------------------------------------------------------
def decoder_layer(x, p, B, S, n_heads, d_head, eps=1e-6, R_batch=1, R_model=1,
                  rows=None, return_norm=False):
    """x' = loop b [#tile<0>](R_batch) { xb = slice 0 x[b];
              h  = xb + loop m [#sum](R_model) { attn_m(rms(xb, g1)) @ slice 0 Wo[m] };
              h + loop m [#sum](R_model) { gelu(rms(h, g2) @ slice 1 W1[m]) @ slice 0 W2[m] } }

    p: dict with g1, g2 [D], Wq, Wk, Wv, Wo [D, D], W1 [D, F], W2 [F, D].
    rms(xb, g1) is a replicated value of the batch shard: every model shard
    reads the same normalised rows.  ``rows`` restricts the output rows; the
    attention then reads every key position of the touched sequences up to the
    largest requested one.  The normaliser returned with ``return_norm`` is
    |h| + |gelu(.)|.|W2| of the final residual add (|x| + |attn|.|Wo| of the
    attention residual add when the FFN has width 0)."""
    T, D = x.shape
    if T != B * S or B % R_batch or n_heads % R_model or p["W1"].shape[1] % R_model:
        raise ValueError("indivisible partition")
    scale = 1.0 / math.sqrt(d_head)
    x = np.asarray(x, np.float64)
    sel = np.arange(T) if rows is None else np.asarray(rows)
    out = np.zeros((len(sel), D))
    norm = np.zeros_like(out)
    Tb = T // R_batch
    hps = n_heads // R_model
    for b in range(R_batch):
        xb = slice_(x, 0, b, R_batch)
        mine = [(i, r - b * Tb) for i, r in enumerate(sel) if b * Tb <= r < (b + 1) * Tb]
        if not mine:
            continue
        local = np.array([t for _, t in mine])
        xn = rmsnorm(xb, p["g1"], eps)

        att = []
        for m in range(R_model):
            a = _attend_shard(xn, slice_(p["Wq"], 1, m, R_model), slice_(p["Wk"], 1, m, R_model),
                              slice_(p["Wv"], 1, m, R_model), B // R_batch, S, hps, d_head,
                              scale, True, local)
            wo = slice_(p["Wo"], 0, m, R_model)
            att.append((matmul(a, wo), abs_product(a, wo) if return_norm else None))
        h = xb[local] + loop_sum(R_model, lambda m: att[m][0])
        hn = rmsnorm(h, p["g2"], eps)
        parts = []
        for m in range(R_model):
            g = gelu_erf(matmul(hn, slice_(p["W1"], 1, m, R_model)))
            w2 = slice_(p["W2"], 0, m, R_model)
            parts.append((matmul(g, w2), abs_product(g, w2) if return_norm else None))
        idx = np.array([i for i, _ in mine])
        out[idx] = h + loop_sum(R_model, lambda m: parts[m][0])
        if return_norm:
            if p["W1"].shape[1] == 0:
                # an FFN of width 0 contracts over nothing: the last contraction
                # is the attention out-projection
                norm[idx] = np.abs(xb[local]) + loop_sum(R_model, lambda m: att[m][1])
            else:
                norm[idx] = np.abs(h) + loop_sum(R_model, lambda m: parts[m][1])
    return (out, norm) if return_norm else out


def decoder_rows_needed(rows, T, S):
    """Rows of a layer's input that its attention needs for output ``rows``:
    every position up to the largest requested one in each touched sequence."""
    need = set()
    for r in np.asarray(rows):
        s0 = (int(r) // S) * S
        need.update(range(s0, int(r) + 1))
    return np.array(sorted(need))


def decoder(x, layers, B, S, n_heads, d_head, eps=1e-6, R_batch=1, R_model=1,
            rows=None, return_norm=False):
    """A stack of decoder layers applied in order.  With ``rows``, each layer
    is evaluated on the rows the following layers need (prefixes of the touched
    sequences), and the last layer on ``rows`` only."""
    T = x.shape[0]
    x = np.asarray(x, np.float64)
    if rows is None:
        out, nrm = x, None
        for p in layers:
            out, nrm = decoder_layer(out, p, B, S, n_heads, d_head, eps, R_batch, R_model,
                                     return_norm=True)
        return (out, nrm) if return_norm else out
    rows = np.asarray(rows)
    need = decoder_rows_needed(rows, T, S)
    # x restricted to the needed prefix rows; positions keep their sequence index
    cur = {int(r): x[r] for r in need}
    for li, p in enumerate(layers):
        last = li == len(layers) - 1
        want = rows if last else need
        full = np.zeros_like(x)
        for r, v in cur.items():
            full[r] = v
        # rows outside `need` are never read: attention of a needed row only
        # looks at earlier positions of its own sequence, all of which are needed
        res, nrm = decoder_layer(full, p, B, S, n_heads, d_head, eps, R_batch, R_model,
                                 rows=want, return_norm=True)
        cur = {int(r): res[i] for i, r in enumerate(want)}
    out = np.stack([cur[int(r)] for r in rows])
    return (out, nrm) if return_norm else out


def decoder_ref(x, layers, B, S, n_heads, d_head, eps=1e-6):
    """Unpartitioned decoder stack."""
    x = np.asarray(x, np.float64)
    for p in layers:
        h = x + attn_ref(rmsnorm(x, p["g1"], eps), p["Wq"], p["Wk"], p["Wv"], p["Wo"],
                         B, S, n_heads, d_head)
        x = h + mlp_ref(rmsnorm(h, p["g2"], eps), p["W1"], p["W2"])
    return x


# ---------------------------------------------------------------------------
# PartIR:SPMD collectives on device-local arrays (Sec. 6)
# ---------------------------------------------------------------------------
# A mesh is a list [(axis name, size), ...]; device-local values are dicts
# {device coordinates (tuple, one entry per axis in mesh order): array}.
def mesh_devices(mesh):
    devs = [()]
    for _, n in mesh:
        devs = [d + (r,) for d in devs for r in range(n)]
    return devs


def _axis(mesh, axis):
    names = [a for a, _ in mesh]
    k = names.index(axis)
    return k, mesh[k][1]


def _peers(dev, k, n):
    return [dev[:k] + (r,) + dev[k + 1:] for r in range(n)]


def replicated(x, mesh):
    return {d: np.asarray(x, np.float64) for d in mesh_devices(mesh)}


def all_slice(local, mesh, dim, axis):
    """Each device keeps the chunk of its array along `dim` given by its own
    coordinate on `axis` (equal contiguous chunks, no padding)."""
    k, n = _axis(mesh, axis)
    return {d: slice_(x, dim, d[k], n) for d, x in local.items()}


def all_gather(local, mesh, dim, axis):
    """Each device gets the concatenation along `dim` of the arrays of the
    devices that differ from it only on `axis`, in axis order (the dual of
    all_slice: the dim grows by the axis size)."""
    k, n = _axis(mesh, axis)
    return {d: np.concatenate([np.asarray(local[p], np.float64) for p in _peers(d, k, n)], axis=dim)
            for d in local}


def all_reduce(local, mesh, axis):
    """Each device gets the sum, in axis order, of the arrays of the devices
    that differ from it only on `axis` (the result is replicated on it)."""
    k, n = _axis(mesh, axis)
    out = {}
    for d in local:
        acc = np.array(local[_peers(d, k, n)[0]], dtype=np.float64, copy=True)
        for p in _peers(d, k, n)[1:]:
            acc = acc + local[p]
        out[d] = acc
    return out


def reduce_scatter(local, mesh, dim, axis):
    """The device with coordinate r on `axis` gets the sum over its axis
    group of every member's r-th chunk along `dim` (the chunks are summed,
    not the whole arrays: the collective's own definition)."""
    k, n = _axis(mesh, axis)
    out = {}
    for d in local:
        parts = [slice_(local[p], dim, d[k], n) for p in _peers(d, k, n)]
        acc = np.array(parts[0], dtype=np.float64, copy=True)
        for q in parts[1:]:
            acc = acc + q
        out[d] = acc
    return out


def mlp_block_z3(X_loc, W1_loc, W2_loc, b1=None, b2=None, act="gelu", R_batch=1, R_model=1,
                 sequence_sharded=True):
    """The lowered SPMD program of the MLP under BP + MP + Z3 on the mesh
    {B: R_batch, M: R_model} (Sec. 3, the data-parallel fully sharded chain):
    per device (b, m), with W1_loc = W1[dim 0 block b, dim 1 block m] and
    W2_loc = W2[dim 0 block m, dim 1 block b]:

      w1 = all_gather<B>(W1_loc, dim 0);  w2 = all_gather<B>(W2_loc, dim 1)
      x  = all_gather<M>(X_loc, dim 0)    if the activations are sharded on M
           X_loc                          otherwise (the batch block b)
      h  = act(x w1 + slice 0 b1[m]);  p = h w2
      y  = reduce_scatter<M>(p, dim 0) + b2   if sharded on M (the all_reduce
           all_reduce<M>(p) + b2              fused with the all_slice)
    Returns {device: y}.
    """
    mesh = [("B", R_batch), ("M", R_model)]
    x = all_gather(X_loc, mesh, 0, "M") if sequence_sharded else {d: np.asarray(v, np.float64)
                                                                    for d, v in X_loc.items()}
    w1 = all_gather(W1_loc, mesh, 0, "B")
    w2 = all_gather(W2_loc, mesh, 1, "B")
    b1_loc = None if b1 is None else all_slice(replicated(b1, mesh), mesh, 0, "M")
    p = {}
    for d in mesh_devices(mesh):
        z = matmul(x[d], w1[d])
        if b1_loc is not None:
            z = z + b1_loc[d]
        p[d] = matmul(activation(z, act), w2[d])
    y = reduce_scatter(p, mesh, 0, "M") if sequence_sharded else all_reduce(p, mesh, "M")
    if b2 is not None:
        y = {d: v + np.asarray(b2, np.float64) for d, v in y.items()}
    return y


def z3_local_operands(X, W1, W2, R_batch, R_model, sequence_sharded=True):
    """Value tiling of the whole operands into the device-local arrays the
    lowering takes as arguments (Sec. 6: arguments used by all_slice become
    device-local): X by tokens over B (and M), W1 dim 0 over B and dim 1 over
    M, W2 dim 0 over M and dim 1 over B."""
    mesh = [("B", R_batch), ("M", R_model)]
    x = all_slice(replicated(X, mesh), mesh, 0, "B")
    if sequence_sharded:
        x = all_slice(x, mesh, 0, "M")
    w1 = all_slice(all_slice(replicated(W1, mesh), mesh, 0, "B"), mesh, 1, "M")
    w2 = all_slice(all_slice(replicated(W2, mesh), mesh, 0, "M"), mesh, 1, "B")
    return x, w1, w2


def decoder_layer_z3(x_loc, p_loc, g1, g2, B, S, n_heads, d_head, eps=1e-6, R_batch=1, R_model=1):
    """The lowered SPMD program of decoder_layer under BP + MP + Z3 with the
    residual stream sharded over the model axis as well (sequence-parallel
    norms), per device (b, m) of the mesh {B, M}:

      xn = all_gather<M>(rmsnorm(x_loc, g1), dim 0)        the norm on the local tokens
      q|k|v = xn @ all_gather<B>(W{q,k,v}_loc, dim 0)       the shard's heads
      a  = causal attention of those heads over the batch block's sequences
      x_loc += reduce_scatter<M>(a @ all_gather<B>(Wo_loc, dim 1), dim 0)
      hn = all_gather<M>(rmsnorm(x_loc, g2), dim 0)
      x_loc += reduce_scatter<M>(gelu(hn @ all_gather<B>(W1_loc, dim 0))
                                 @ all_gather<B>(W2_loc, dim 1), dim 0)

    x_loc {device: [T/(R_batch R_model), D]}; p_loc {name: {device: block}}
    with Wq, Wk, Wv, W1 blocks (dim 0 block b, dim 1 block m) and Wo, W2
    blocks (dim 0 block m, dim 1 block b).  Returns the new x_loc."""
    mesh = [("B", R_batch), ("M", R_model)]
    scale = 1.0 / math.sqrt(d_head)
    hps, nseq = n_heads // R_model, B // R_batch
    x = {d: np.asarray(v, np.float64) for d, v in x_loc.items()}
    gathered = {k: all_gather(p_loc[k], mesh, 0, "B") for k in ("Wq", "Wk", "Wv", "W1")}
    gathered.update({k: all_gather(p_loc[k], mesh, 1, "B") for k in ("Wo", "W2")})
    xn = all_gather({d: rmsnorm(v, g1, eps) for d, v in x.items()}, mesh, 0, "M")
    part = {}
    for d in mesh_devices(mesh):
        q, k, v = (matmul(xn[d], gathered[w][d]) for w in ("Wq", "Wk", "Wv"))
        a = np.zeros_like(q)
        for sq in range(nseq):
            rs = slice(sq * S, (sq + 1) * S)
            for hh in range(hps):
                cs = slice(hh * d_head, (hh + 1) * d_head)
                a[rs, cs] = causal_attention(q[rs, cs], k[rs, cs], v[rs, cs], scale, True)
        part[d] = matmul(a, gathered["Wo"][d])
    rs_ = reduce_scatter(part, mesh, 0, "M")
    x = {d: x[d] + rs_[d] for d in x}
    hn = all_gather({d: rmsnorm(v, g2, eps) for d, v in x.items()}, mesh, 0, "M")
    part = {d: matmul(gelu_erf(matmul(hn[d], gathered["W1"][d])), gathered["W2"][d]) for d in mesh_devices(mesh)}
    rs_ = reduce_scatter(part, mesh, 0, "M")
    return {d: x[d] + rs_[d] for d in x}


def z3_local_decoder(x, p, R_batch, R_model):
    """Value tiling of a decoder layer's whole operands into device-local
    arrays: x by tokens over B then M; Wq, Wk, Wv, W1 dim 0 over B and dim 1
    over M; Wo, W2 dim 0 over M and dim 1 over B (Sec. 6: sliced arguments
    become device-local)."""
    mesh = [("B", R_batch), ("M", R_model)]
    x_loc = all_slice(all_slice(replicated(x, mesh), mesh, 0, "B"), mesh, 0, "M")
    p_loc = {}
    for k in ("Wq", "Wk", "Wv", "W1"):
        p_loc[k] = all_slice(all_slice(replicated(p[k], mesh), mesh, 0, "B"), mesh, 1, "M")
    for k in ("Wo", "W2"):
        p_loc[k] = all_slice(all_slice(replicated(p[k], mesh), mesh, 0, "M"), mesh, 1, "B")
    return x_loc, p_loc


# ---------------------------------------------------------------------------
# Parity measure (the elementwise forward-error form)
# ---------------------------------------------------------------------------
def normalised_error(got, ref, norm):
    """max_ij |got - ref|_ij / norm_ij; entries with norm 0 must match exactly
    (they contribute +inf otherwise)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    norm = np.asarray(norm, np.float64)
    diff = np.abs(got - ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.where(norm > 0, diff / np.where(norm > 0, norm, 1.0),
                     np.where(diff == 0, 0.0, np.inf))
    return float(np.max(e)) if e.size else 0.0

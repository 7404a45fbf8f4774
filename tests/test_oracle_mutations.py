"""Planted mistakes in the oracle must be caught by its pins.

Each case swaps one oracle function for a plausibly wrong variant (on the
CPU, inside this process only) and runs the pins that should notice; at least
one of them has to fail.  This shows the pins constrain every part of the
oracle rather than only re-deriving it.
"""
import math

import numpy as np
import pytest

from oracle import partir_oracle as O
from tests import test_oracle_backward as BW
from tests import test_oracle_core as C
from tests import test_oracle_spmd as SP
from tests import test_oracle_ops as P
from tests import test_oracle_programs as G

_real = {name: getattr(O, name) for name in dir(O) if callable(getattr(O, name))}


def _slice_shifted(x, d, r, n):
    return _real["slice_"](x, d, (r + 1) % n, n)


def _tile_reversed(n, d, body):
    return np.concatenate([body(r) for r in reversed(range(n))], axis=d)


def _sum_drops_last(n, body):
    acc = np.array(body(0), dtype=np.float64, copy=True)
    for r in range(1, n - 1):
        acc = acc + body(r)
    return acc


def _matmul_bt(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return a @ (b.T if b.shape[0] == b.shape[1] else b[:, ::-1])


def _gelu_tanh(x):
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))


def _gelu_no_sqrt2(x):
    from scipy.special import erf
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1 + erf(x))


def _rms_sum(x, g, eps):
    x = np.asarray(x, np.float64)
    return g * x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)


def _rms_eps_outside(x, g, eps):
    x = np.asarray(x, np.float64)
    return g * x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps)


def _attn_variant(mask, scaled=True):
    def f(q, k, v, scale, causal=True, q_pos=None):
        q, k, v = (np.asarray(t, np.float64) for t in (q, k, v))
        if q_pos is None:
            q_pos = np.arange(q.shape[0])
        s = q @ k.T * (scale if scaled else 1.0)
        if causal:
            kp = np.arange(k.shape[0])[None, :]
            qp = np.asarray(q_pos)[:, None]
            s = np.where(mask(kp, qp), s, -np.inf)
        with np.errstate(invalid="ignore"):
            m = np.max(s, axis=1, keepdims=True)
            p = np.exp(s - m)
            p = p / np.sum(p, axis=1, keepdims=True)
        return p @ v
    return f


def _mlp_bias_inside(X, W1, W2, b1=None, b2=None, act="gelu", R_batch=1, R_model=1,
                     rows=None, return_norm=False):
    if b2 is not None:
        out = _real["mlp_block"](X, W1, W2, b1, None, act, R_batch, R_model, rows, return_norm)
        bump = R_model * np.asarray(b2, np.float64)
        return (out[0] + bump, out[1]) if return_norm else out + bump
    return _real["mlp_block"](X, W1, W2, b1, b2, act, R_batch, R_model, rows, return_norm)


def _gelu_grad_cdf_only(x, act):
    from scipy.special import erf
    x = np.asarray(x, np.float64)
    return np.ones_like(x) if act == "none" else 0.5 * (1 + erf(x / math.sqrt(2)))


def _gelu_grad_minus(x, act):
    from scipy.special import erf
    x = np.asarray(x, np.float64)
    if act == "none":
        return np.ones_like(x)
    return 0.5 * (1 + erf(x / math.sqrt(2))) - x * np.exp(-0.5 * x * x) / math.sqrt(2 * math.pi)


def _gather_reversed(local, mesh, dim, axis):
    k = [a for a, _ in mesh].index(axis)
    n = mesh[k][1]
    return {d: np.concatenate([local[d[:k] + (r,) + d[k + 1:]] for r in reversed(range(n))], axis=dim)
            for d in local}


def _scatter_wrong_chunk(local, mesh, dim, axis):
    k = [a for a, _ in mesh].index(axis)
    n = mesh[k][1]
    out = {}
    for d in local:
        peers = [d[:k] + (r,) + d[k + 1:] for r in range(n)]
        out[d] = sum(_real["slice_"](local[p], dim, (d[k] + 1) % n, n) for p in peers)
    return out


def _attn_bwd_without_rowsum(q, k, v, do, scale, causal=True, return_norm=False):
    """The softmax Jacobian applied without its rank-one term: ds = p * dp."""
    q, k, v, do = (np.asarray(a, np.float64) for a in (q, k, v, do))
    n = q.shape[0]
    s = q @ k.T * scale
    if causal:
        s = np.where(np.arange(n)[None, :] <= np.arange(n)[:, None], s, -np.inf)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    ds = p * (do @ v.T)
    return scale * ds @ k, scale * ds.T @ q, p.T @ do


def _attend_k_from_q(xb, Wq_m, Wk_m, Wv_m, *rest):
    return _real["_attend_shard"](xb, Wq_m, Wq_m, Wv_m, *rest)


def _run(pins, golden):
    failures = 0
    for pin in pins:
        kwargs = {"golden": golden} if "golden" in pin.__code__.co_varnames[:pin.__code__.co_argcount] else {}
        try:
            if pin.__name__ == "test_loop_matmul_brute_force":
                pin(O.AXIS_M, O.AXIS_K, 2, **kwargs)
                pin(O.AXIS_N, O.AXIS_NONE, 4, **kwargs)
            elif pin.__name__ == "test_loop_matmul_integer_exact_bitwise":
                pin(4, **kwargs)
            elif pin.__name__ in ("test_attention_brute_force",):
                pin(True)
            elif pin.__name__ == "test_attn_block_brute_force":
                pin(2, 4)
            elif pin.__name__ == "test_mlp_integer_exact_across_partitions":
                pin(2, 4)
            elif pin.__name__ == "test_mlp_backward_matches_torch_autograd":
                pin("gelu", 2, 4)
            elif pin.__name__ == "test_attention_backward_matches_torch_autograd":
                pin(True)
            elif pin.__name__ == "test_z3_mlp_integer_exact_equals_unpartitioned":
                pin(4, 2, True)
            elif pin.__name__ == "test_reduce_scatter_is_all_reduce_fused_with_all_slice":
                pin(0, "M")
            else:
                pin(**kwargs)
        except (AssertionError, ValueError, FloatingPointError):
            failures += 1
    return failures


CASES = {
    "slice picks the wrong chunk": ("slice_", _slice_shifted,
                                    [C.test_slice_is_rth_contiguous_chunk, C.test_value_tiling_shapes]),
    "tile concatenates out of order": ("loop_tile", _tile_reversed,
                                       [C.test_loop_tile_is_concatenation_in_r_order, C.test_loop_matmul_brute_force]),
    "sum drops an iteration": ("loop_sum", _sum_drops_last,
                               [C.test_loop_sum_sums_every_iteration_once, C.test_loop_matmul_integer_exact_bitwise]),
    "matmul transposes an operand": ("matmul", _matmul_bt,
                                     [C.test_matmul_equivalences_shapes_and_values, C.test_loop_matmul_brute_force]),
    "gelu uses the tanh form": ("gelu_erf", _gelu_tanh,
                                [P.test_gelu_textbook_points, P.test_gelu_matches_math_erf_and_torch]),
    "gelu drops 1/sqrt2": ("gelu_erf", _gelu_no_sqrt2, [P.test_gelu_textbook_points]),
    "rmsnorm sums instead of averaging": ("rmsnorm", _rms_sum, [P.test_rmsnorm_constant_row_closed_form]),
    "rmsnorm adds eps outside the root": ("rmsnorm", _rms_eps_outside, [P.test_rmsnorm_constant_row_closed_form]),
    "causal mask excludes the diagonal": ("causal_attention", _attn_variant(lambda kp, qp: kp < qp),
                                          [P.test_attention_first_position_is_v0_exactly]),
    "causal mask points the wrong way": ("causal_attention", _attn_variant(lambda kp, qp: kp >= qp),
                                         [P.test_attention_zero_queries_give_prefix_means]),
    "attention forgets the scale": ("causal_attention", _attn_variant(lambda kp, qp: kp <= qp, scaled=False),
                                    [P.test_attention_brute_force, P.test_attention_matches_torch_sdpa]),
    "bias added inside the #sum": ("mlp_block", _mlp_bias_inside, [G.test_mlp_bias_of_sum_loop_is_added_once]),
    "gelu derivative drops x phi(x)": ("activation_grad", _gelu_grad_cdf_only,
                                       [BW.test_gelu_grad_closed_forms, BW.test_mlp_backward_matches_torch_autograd]),
    "gelu derivative subtracts x phi(x)": ("activation_grad", _gelu_grad_minus,
                                           [BW.test_gelu_grad_matches_central_differences_and_torch,
                                            BW.test_mlp_backward_central_differences_of_the_forward]),
    "all_gather concatenates in reverse": ("all_gather", _gather_reversed,
                                           [SP.test_all_gather_concatenates_in_axis_order,
                                            SP.test_z3_mlp_integer_exact_equals_unpartitioned]),
    "reduce_scatter hands out the wrong chunk": ("reduce_scatter", _scatter_wrong_chunk,
                                                 [SP.test_reduce_scatter_is_all_reduce_fused_with_all_slice,
                                                  SP.test_z3_mlp_integer_exact_equals_unpartitioned]),
    "attention backward drops the rowsum term": ("attention_backward", _attn_bwd_without_rowsum,
                                                 [BW.test_attention_backward_matches_torch_autograd,
                                                  BW.test_attention_backward_central_differences]),
    "keys projected with Wq": ("_attend_shard", _attend_k_from_q, [G.test_attn_block_brute_force]),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_planted_mistake_is_caught(case, golden, monkeypatch):
    name, wrong, pins = CASES[case]
    monkeypatch.setattr(O, name, wrong)
    assert _run(pins, golden) >= 1, f"no pin caught: {case}"


def test_unmodified_oracle_passes_the_same_pins(golden):
    pins = {p for _, _, ps in CASES.values() for p in ps}
    assert _run(sorted(pins, key=lambda p: p.__name__), golden) == 0

"""Pins for the oracle's PartIR:Core constructs and the partitioned matmul.

Every check compares the oracle against something other than itself: the
shapes the paper prints (tests/golden/paper_shapes.json), pure-Python brute
force, integer-exact equality with the unpartitioned product, and the
definition of contiguous equal chunks.
"""
import itertools

import numpy as np
import pytest

from oracle import partir_oracle as O

pytestmark = pytest.mark.filterwarnings("ignore")


def brute_matmul(a, b):
    n, k = len(a), len(a[0])
    m = len(b[0])
    return [[sum(a[i][t] * b[t][j] for t in range(k)) for j in range(m)] for i in range(n)]


def int_matrix(rng, shape, lo=-3, hi=3):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float64)


# ---------------------------------------------------------------------------
# slice / loop constructs
# ---------------------------------------------------------------------------
def test_slice_is_rth_contiguous_chunk():
    x = np.arange(24.0).reshape(4, 6)
    for r in range(3):
        assert O.slice_(x, 1, r, 3).tolist() == [[row[c] for c in range(2 * r, 2 * r + 2)] for row in x.tolist()]
    for r in range(2):
        assert O.slice_(x, 0, r, 2).tolist() == x.tolist()[2 * r:2 * r + 2]


def test_slice_rejects_indivisible_and_out_of_range():
    x = np.zeros((6, 4))
    with pytest.raises(ValueError):
        O.slice_(x, 0, 0, 4)
    with pytest.raises(ValueError):
        O.slice_(x, 1, 2, 2)


def test_value_tiling_shapes(golden):
    g = golden["value_tiling"]
    x = np.arange(np.prod(g["x"]), dtype=np.float64).reshape(g["x"])
    n = g["axis_size"]
    assert list(O.slice_(x, g["dim"], 0, n).shape) == g["slice"]
    t = O.loop_tile(n, g["dim"], lambda r: O.slice_(x, g["dim"], r, n))
    assert list(t.shape) == g["loop"]
    # value tiling is semantics preserving: the loop rebuilds x exactly
    assert np.array_equal(t, x)


def test_loop_tile_is_concatenation_in_r_order():
    parts = {r: np.full((2, 3), float(r)) for r in range(4)}
    t0 = O.loop_tile(4, 0, lambda r: parts[r])
    assert t0.shape == (8, 3) and [t0[2 * r, 0] for r in range(4)] == [0, 1, 2, 3]
    t1 = O.loop_tile(4, 1, lambda r: parts[r])
    assert t1.shape == (2, 12) and [t1[0, 3 * r] for r in range(4)] == [0, 1, 2, 3]


def test_loop_sum_sums_every_iteration_once():
    seen = []

    def body(r):
        seen.append(r)
        return np.array([10.0 ** r])

    assert O.loop_sum(5, body)[0] == 11111.0
    assert seen == [0, 1, 2, 3, 4]


def test_loop_sum_does_not_alias_first_body_value():
    base = np.ones(3)
    out = O.loop_sum(3, lambda r: base)
    assert out.tolist() == [3.0, 3.0, 3.0] and base.tolist() == [1.0, 1.0, 1.0]


# ---------------------------------------------------------------------------
# The three matmul equivalences (figure matmul-examples)
# ---------------------------------------------------------------------------
def test_matmul_equivalences_shapes_and_values(golden):
    g = golden["matmul_equivalences"]
    rng = np.random.default_rng(1)
    x, y, n = int_matrix(rng, g["x"]), int_matrix(rng, g["y"]), g["axis_size"]
    ref = brute_matmul(x.tolist(), y.tolist())
    assert list(O.slice_(x, 0, 1, n).shape) == g["tile0"]["slice_x"]
    assert list(O.matmul(O.slice_(x, 0, 1, n), y).shape) == g["tile0"]["body"]
    assert list(O.slice_(y, 1, 1, n).shape) == g["tile1"]["slice_y"]
    assert list(O.matmul(x, O.slice_(y, 1, 1, n)).shape) == g["tile1"]["body"]
    assert list(O.slice_(x, 1, 1, n).shape) == g["sum"]["slice_x"]
    assert list(O.slice_(y, 0, 1, n).shape) == g["sum"]["slice_y"]
    for name, (t, s) in {"tile0": (O.AXIS_M, O.AXIS_NONE), "tile1": (O.AXIS_N, O.AXIS_NONE),
                         "sum": (O.AXIS_NONE, O.AXIS_K)}.items():
        c = O.loop_matmul(x, y, t, s, n)
        assert list(c.shape) == g[name]["loop"]
        assert c.tolist() == ref, name


@pytest.mark.parametrize("tile,summ", [(O.AXIS_NONE, O.AXIS_NONE), (O.AXIS_M, O.AXIS_NONE),
                                       (O.AXIS_N, O.AXIS_NONE), (O.AXIS_NONE, O.AXIS_K),
                                       (O.AXIS_M, O.AXIS_K), (O.AXIS_N, O.AXIS_K)])
@pytest.mark.parametrize("R", [1, 2, 4])
def test_loop_matmul_brute_force(tile, summ, R):
    rng = np.random.default_rng(7 + R)
    M, N, K = 8, 12, 16
    a = rng.standard_normal((M, K))
    b = rng.standard_normal((K, N))
    ref = np.array(brute_matmul(a.tolist(), b.tolist()))
    got = O.loop_matmul(a, b, tile, summ, R)
    assert got.shape == (M, N)
    assert np.max(np.abs(got - ref) / O.abs_product(a, b)) < 1e-14


@pytest.mark.parametrize("R", [1, 2, 4, 8])
def test_loop_matmul_integer_exact_bitwise(R):
    rng = np.random.default_rng(R)
    a, b = int_matrix(rng, (16, 64)), int_matrix(rng, (64, 24))
    plain = O.matmul(a, b)
    for t, s in [(O.AXIS_M, O.AXIS_NONE), (O.AXIS_N, O.AXIS_NONE), (O.AXIS_NONE, O.AXIS_K),
                 (O.AXIS_M, O.AXIS_K)]:
        assert np.array_equal(O.loop_matmul(a, b, t, s, R), plain)


def test_loop_matmul_R1_is_plain_product():
    rng = np.random.default_rng(3)
    a, b = rng.standard_normal((5, 7)), rng.standard_normal((7, 3))
    ref = np.array(brute_matmul(a.tolist(), b.tolist()))
    for t, s in [(O.AXIS_M, O.AXIS_NONE), (O.AXIS_N, O.AXIS_NONE), (O.AXIS_NONE, O.AXIS_K)]:
        assert np.allclose(O.loop_matmul(a, b, t, s, 1), ref, rtol=0, atol=1e-13)


def test_loop_matmul_rejects_bad_axes():
    a, b = np.zeros((4, 4)), np.zeros((4, 4))
    with pytest.raises(ValueError):
        O.loop_matmul(a, b, O.AXIS_K, O.AXIS_NONE, 2)
    with pytest.raises(ValueError):
        O.loop_matmul(a, b, O.AXIS_NONE, O.AXIS_M, 2)
    with pytest.raises(ValueError):
        O.loop_matmul(np.zeros((6, 4)), b, O.AXIS_M, O.AXIS_NONE, 4)


def test_abs_product_brute_force():
    rng = np.random.default_rng(11)
    a, b = rng.standard_normal((3, 5)), rng.standard_normal((5, 4))
    ref = brute_matmul(np.abs(a).tolist(), np.abs(b).tolist())
    assert np.allclose(O.abs_product(a, b), ref, rtol=1e-15, atol=0)


# ---------------------------------------------------------------------------
# Nests and multi-axis slicing
# ---------------------------------------------------------------------------
def test_megatron_nest_shapes_and_values(golden):
    g = golden["megatron_nest"]
    nB, nM = g["mesh"]["B"], g["mesh"]["M"]
    rng = np.random.default_rng(5)
    x, w1, w2 = int_matrix(rng, g["x"]), int_matrix(rng, g["w1"]), int_matrix(rng, g["w2"])
    shapes = {}

    def body_b(rb):
        def body_m(rm):
            xs = O.slice_(x, 0, rb, nB)
            w1s = O.slice_(w1, 1, rm, nM)
            x1ss = O.matmul(xs, w1s)
            w2s = O.slice_(w2, 0, rm, nM)
            x2ss = O.matmul(x1ss, w2s)
            shapes.update(xs=xs.shape, w1s=w1s.shape, x1ss=x1ss.shape, w2s=w2s.shape, x2ss=x2ss.shape)
            return x2ss
        return O.loop_sum(nM, body_m)

    r = O.loop_tile(nB, 0, body_b)
    for k in ("xs", "w1s", "x1ss", "w2s", "x2ss"):
        assert list(shapes[k]) == g[k], k
    assert list(r.shape) == g["result"]
    # the nest is the unpartitioned chain (no activation), bitwise on integers
    ref = brute_matmul(brute_matmul(x.tolist(), w1.tolist()), w2.tolist())
    assert r.tolist() == ref
    assert np.array_equal(O.mlp_block(x, w1, w2, act="none", R_batch=nB, R_model=nM), r)


def test_distributed_type_local_shapes(golden):
    g = golden["distributed_types"]
    na, nb = g["mesh"]["a"], g["mesh"]["b"]
    x = np.arange(256 * 8, dtype=np.float64).reshape(g["x"])
    assert list(O.slice_(x, 0, 0, na).shape) == g["rows_a"]
    assert list(O.slice_(x, 1, 0, nb).shape) == g["cols_b"]
    assert list(O.slice_(O.slice_(x, 0, 0, na), 1, 0, nb).shape) == g["rows_a_cols_b"]
    assert list(O.slice_(O.slice_(x, 1, 0, na), 1, 0, nb).shape) == g["cols_ab"]
    assert list(O.slice_(O.slice_(x, 1, 0, nb), 1, 0, na).shape) == g["cols_ba"]


def test_deep_tiling_assignment_orders_are_transposed():
    """slice 1 (slice 1 x[ra])[rb] holds column 2*ra + rb (outer axis major);
    nesting the other way round transposes the device assignment (App. B.2,
    App. C.2 on [256,{a,b}8] vs [256,{b,a}8])."""
    x = np.tile(np.arange(8.0), (3, 1))
    ab = {(ra, rb): O.slice_(O.slice_(x, 1, ra, 4), 1, rb, 2)[0, 0] for ra, rb in itertools.product(range(4), range(2))}
    ba = {(ra, rb): O.slice_(O.slice_(x, 1, rb, 2), 1, ra, 4)[0, 0] for ra, rb in itertools.product(range(4), range(2))}
    assert all(ab[(ra, rb)] == 2 * ra + rb for ra, rb in ab)
    assert all(ba[(ra, rb)] == 4 * rb + ra for ra, rb in ba)
    # deep-tiled loop rebuilds x
    xtt = O.loop_tile(4, 1, lambda ra: O.loop_tile(2, 1, lambda rb: O.slice_(O.slice_(x, 1, ra, 4), 1, rb, 2)))
    assert np.array_equal(xtt, x)


def test_tile_reduce_stacked_views(golden):
    g = golden["tile_reduce"]
    na, nb = g["mesh"]["a"], g["mesh"]["b"]
    local = {(a, b): np.full(g["local"], 10.0 * a + b) for a in range(na) for b in range(nb)}
    t01 = O.loop_tile(na, 0, lambda a: O.loop_tile(nb, 1, lambda b: local[(a, b)]))
    assert list(t01.shape) == g["tile_a0_b1"]
    assert t01[64 * 3, 4 * 1] == 31.0
    t10 = O.loop_tile(nb, 0, lambda b: O.loop_tile(na, 1, lambda a: local[(a, b)]))
    assert list(t10.shape) == g["tile_a1_b0"]
    assert t10[64 * 1, 4 * 2] == 21.0
    s = O.loop_sum(na, lambda a: O.loop_sum(nb, lambda b: local[(a, b)]))
    assert list(s.shape) == g["sum_a_sum_b"]
    assert s[0, 0] == sum(10.0 * a + b for a in range(na) for b in range(nb))


def test_lowered_megatron_has_one_sum_per_block(golden):
    """The device-local form keeps exactly one all_reduce (the #sum over M) on a
    64x8 partial: counting the oracle's #sum loops in the nest gives one."""
    g = golden["lowered_megatron"]
    count = {"sum": 0}
    real = O.loop_sum

    def counting(n, body):
        count["sum"] += 1
        out = real(n, body)
        assert list(out.shape) == g["all_reduce"]
        return out

    rng = np.random.default_rng(2)
    x, w1, w2 = int_matrix(rng, (256, 8)), int_matrix(rng, (8, 16)), int_matrix(rng, (16, 8))
    O.loop_sum = counting
    try:
        O.mlp_block(x, w1, w2, act="none", R_batch=4, R_model=2)
    finally:
        O.loop_sum = real
    assert count["sum"] == 4 * g["n_all_reduce"]  # one per batch shard


def test_normalised_error_definition():
    ref = np.array([1.0, 2.0, 0.0])
    norm = np.array([2.0, 4.0, 0.0])
    assert O.normalised_error(np.array([1.5, 2.0, 0.0]), ref, norm) == 0.25
    assert O.normalised_error(np.array([1.0, 2.0, 1e-30]), ref, norm) == np.inf


# ---------------------------------------------------------------------------
# empty operands: TSlice with n_d = 0, and the empty sum
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("tile,summ,R", [(O.AXIS_NONE, O.AXIS_K, 4), (O.AXIS_M, O.AXIS_NONE, 4),
                                         (O.AXIS_N, O.AXIS_K, 2), (O.AXIS_NONE, O.AXIS_NONE, 1)])
def test_empty_contraction_is_the_empty_sum(tile, summ, R):
    """K = 0: each shard's partial is an [M, N] block of empty dot products,
    and a sum over no terms is 0 (pure-Python brute force agrees)."""
    A, B = np.zeros((8, 0)), np.zeros((0, 12))
    C = O.loop_matmul(A, B, tile, summ, R)
    assert C.shape == (8, 12)
    brute = [[sum(()) for _ in range(12)] for _ in range(8)]   # sum of an empty sequence
    assert C.tolist() == brute


@pytest.mark.parametrize("tile,R", [(O.AXIS_M, 4), (O.AXIS_N, 4)])
def test_tiling_an_empty_dim_gives_empty_shards(tile, R):
    """slice d x[r] of a zero-size dim: R empty chunks whose concatenation is
    the empty result of the right shape."""
    rng = np.random.default_rng(5)
    if tile == O.AXIS_M:
        A, B = rng.standard_normal((0, 16)), rng.standard_normal((16, 12))
        assert O.slice_(A, 0, R - 1, R).shape == (0, 16)
    else:
        A, B = rng.standard_normal((8, 16)), rng.standard_normal((16, 0))
        assert O.slice_(B, 1, R - 1, R).shape == (16, 0)
    C = O.loop_matmul(A, B, tile, O.AXIS_NONE, R)
    assert C.shape == (A.shape[0], B.shape[1]) and C.size == 0

"""Pins for the oracle's PartIR:SPMD collectives and the lowered MLP under
BP + MP + Z3 (device-local arrays on a mesh).

The collectives are checked against their definitions in Sec. 6 (all_gather
dual to all_slice; reduce_scatter is the fusion of all_reduce with
all_slice), against the shapes of the paper's collectives listing, and with
integer values that expose ordering and double counting.  The lowered MLP
program is checked against the unpartitioned MLP and the shard interpreter
(the lowering preserves semantics, App. C), and its local shapes against the
Sec. 3 fully sharded chain listing.
"""
import math

import numpy as np
import pytest

from oracle import partir_oracle as O

MESH = [("B", 4), ("M", 2)]


def local_ints(mesh, shape, seed):
    rng = np.random.default_rng(seed)
    return {d: rng.integers(-5, 6, size=shape).astype(np.float64) for d in O.mesh_devices(mesh)}


def test_mesh_devices_row_major():
    assert O.mesh_devices(MESH) == [(b, m) for b in range(4) for m in range(2)]


@pytest.mark.parametrize("dim,axis", [(0, "B"), (1, "B"), (0, "M"), (1, "M")])
def test_all_gather_of_all_slice_is_identity(dim, axis):
    x = np.arange(8 * 16, dtype=np.float64).reshape(8, 16)
    rep = O.replicated(x, MESH)
    back = O.all_gather(O.all_slice(rep, MESH, dim, axis), MESH, dim, axis)
    assert all(np.array_equal(v, x) for v in back.values())


def test_all_slice_of_all_gather_is_identity_on_local_arrays():
    loc = local_ints(MESH, (3, 5), 0)
    back = O.all_slice(O.all_gather(loc, MESH, 1, "B"), MESH, 1, "B")
    assert all(np.array_equal(back[d], loc[d]) for d in loc)


def test_all_gather_concatenates_in_axis_order():
    loc = {d: np.full((2, 1), 10.0 * d[0] + d[1]) for d in O.mesh_devices(MESH)}
    g = O.all_gather(loc, MESH, 0, "B")
    assert np.array_equal(g[(2, 1)][:, 0], [1, 1, 11, 11, 21, 21, 31, 31])
    g = O.all_gather(loc, MESH, 1, "M")
    assert np.array_equal(g[(3, 0)], [[30, 31], [30, 31]])


def test_all_reduce_counts_every_device_once():
    loc = {d: np.array([10.0 ** d[0] + 100.0 * d[1]]) for d in O.mesh_devices(MESH)}
    r = O.all_reduce(loc, MESH, "B")
    assert r[(0, 1)][0] == 1 + 10 + 100 + 1000 + 400 and r[(2, 0)][0] == 1111
    r = O.all_reduce(loc, MESH, "M")
    assert r[(3, 0)][0] == r[(3, 1)][0] == 2 * 1000 + 100


@pytest.mark.parametrize("dim,axis", [(0, "M"), (1, "B"), (0, "B")])
def test_reduce_scatter_is_all_reduce_fused_with_all_slice(dim, axis):
    loc = local_ints(MESH, (8, 8), 1)
    rs = O.reduce_scatter(loc, MESH, dim, axis)
    fused = O.all_slice(O.all_reduce(loc, MESH, axis), MESH, dim, axis)
    assert all(np.array_equal(rs[d], fused[d]) for d in loc)


def test_collectives_listing_shapes(golden):
    g = golden["spmd_collectives"]
    mesh = list(g["mesh"].items())
    x = np.zeros(g["all_slice"]["in"])

    def apply(fn, local, spec):
        for dim, axes in enumerate(spec):
            for a in axes:
                local = fn(local, mesh, dim, a)
        return local

    rep = O.replicated(x, mesh)
    for key in ("all_slice", "all_slice_two_axes"):
        out = apply(O.all_slice, rep, g[key]["axes"])
        assert all(list(v.shape) == g[key]["out"] for v in out.values()), key
    loc = O.replicated(np.zeros(g["all_gather"]["in"]), mesh)
    out = apply(O.all_gather, loc, g["all_gather"]["axes"])
    assert all(list(v.shape) == g["all_gather"]["out"] for v in out.values())
    out = apply(O.reduce_scatter, rep, g["reduce_scatter"]["axes"])
    assert all(list(v.shape) == g["reduce_scatter"]["out"] for v in out.values())


def test_fsdp_chain_listing_shapes(golden):
    g = golden["fsdp_chain"]
    RB, RM = g["mesh"]["B"], g["mesh"]["M"]
    X, W1, W2 = np.zeros(g["x"]), np.zeros(g["w1"]), np.zeros(g["w2"])
    x, w1, w2 = O.z3_local_operands(X, W1, W2, RB, RM, sequence_sharded=False)
    mesh = [("B", RB), ("M", RM)]
    d = (1, 1)
    assert list(x[d].shape) == g["x_local"] and list(w1[d].shape) == g["w1_local"]
    assert list(w2[d].shape) == g["w2_local"]
    w1g = O.all_gather(w1, mesh, 0, "B")[d]
    w2g = O.all_gather(w2, mesh, 1, "B")[d]
    assert list(w1g.shape) == g["w1g"] and list(w2g.shape) == g["w2g"]
    x1 = O.matmul(x[d], w1g)
    x2 = O.matmul(x1, w2g)
    assert list(x1.shape) == g["x1"] and list(x2.shape) == g["x2"]
    y = O.mlp_block_z3(x, w1, w2, act="none", R_batch=RB, R_model=RM, sequence_sharded=False)
    assert list(y[d].shape) == g["x3"]


def gather_rows(y, RB, RM):
    return np.concatenate([y[(b, m)] for b in range(RB) for m in range(RM)], axis=0)


@pytest.mark.parametrize("RB,RM", [(1, 1), (4, 2), (2, 4), (1, 8), (8, 1)])
@pytest.mark.parametrize("seq", [True, False])
def test_z3_mlp_integer_exact_equals_unpartitioned(RB, RM, seq):
    rng = np.random.default_rng(RB * 10 + RM)
    T, D, F = 64, 16, 32
    X = rng.integers(-2, 3, (T, D)).astype(float)
    W1 = rng.integers(-2, 3, (D, F)).astype(float)
    W2 = rng.integers(-2, 3, (F, D)).astype(float)
    b1, b2 = rng.integers(-2, 3, F).astype(float), rng.integers(-2, 3, D).astype(float)
    x, w1, w2 = O.z3_local_operands(X, W1, W2, RB, RM, seq)
    y = O.mlp_block_z3(x, w1, w2, b1, b2, "none", RB, RM, seq)
    want = (X @ W1 + b1) @ W2 + b2
    if seq:
        assert np.array_equal(gather_rows(y, RB, RM), want)
    else:   # replicated over M: every model device holds its batch block
        for (b, m), v in y.items():
            assert np.array_equal(v, want[b * T // RB:(b + 1) * T // RB])


def test_z3_mlp_gelu_equals_mlp_ref_and_shard_interpreter():
    rng = np.random.default_rng(3)
    T, D, F, RB, RM = 128, 16, 64, 2, 4
    X = rng.standard_normal((T, D))
    W1, W2 = rng.standard_normal((D, F)) / math.sqrt(D), rng.standard_normal((F, D)) / math.sqrt(F)
    b1, b2 = rng.standard_normal(F), rng.standard_normal(D)
    y = gather_rows(O.mlp_block_z3(*O.z3_local_operands(X, W1, W2, RB, RM), b1, b2, "gelu", RB, RM), RB, RM)
    assert np.max(np.abs(y - O.mlp_ref(X, W1, W2, b1, b2, "gelu"))) < 1e-12
    assert np.max(np.abs(y - O.mlp_block(X, W1, W2, b1, b2, "gelu", RB, RM))) < 1e-12


def test_z3_local_operand_blocks():
    """W1 block (b, m) is rows block b (over B) and columns block m (over M);
    W2 block (b, m) is rows block m and columns block b."""
    X = np.arange(24 * 8.0).reshape(24, 8)
    W1, W2 = np.arange(8 * 12.0).reshape(8, 12), np.arange(12 * 8.0).reshape(12, 8)
    x, w1, w2 = O.z3_local_operands(X, W1, W2, 2, 3)
    assert np.array_equal(w1[(1, 2)], W1[4:8, 8:12])
    assert np.array_equal(w2[(1, 2)], W2[8:12, 4:8])
    assert np.array_equal(x[(1, 2)], X[20:24])       # token block b * R_model + m = 5 of 6


@pytest.mark.parametrize("RB,RM", [(1, 1), (2, 2), (1, 4), (2, 1)])
def test_decoder_z3_equals_shard_interpreter_and_reference(RB, RM):
    """Sequence-parallel norms: the norms run on each device's tokens; the
    layer still equals the unpartitioned decoder and the shard interpreter."""
    rng = np.random.default_rng(RB * 7 + RM)
    B, S, H, dh, F = 2, 8, 4, 2, 16
    D = H * dh
    x = rng.standard_normal((B * S, D))
    p = {"g1": 1 + 0.1 * rng.standard_normal(D), "g2": 1 + 0.1 * rng.standard_normal(D)}
    for k in ("Wq", "Wk", "Wv", "Wo"):
        p[k] = rng.standard_normal((D, D)) / math.sqrt(D)
    p["W1"], p["W2"] = rng.standard_normal((D, F)) / math.sqrt(D), rng.standard_normal((F, D)) / math.sqrt(F)
    x_loc, p_loc = O.z3_local_decoder(x, p, RB, RM)
    y = O.decoder_layer_z3(x_loc, p_loc, p["g1"], p["g2"], B, S, H, dh, 1e-6, RB, RM)
    got = gather_rows(y, RB, RM)
    assert np.max(np.abs(got - O.decoder_ref(x, [p], B, S, H, dh, 1e-6))) < 1e-12
    assert np.max(np.abs(got - O.decoder_layer(x, p, B, S, H, dh, 1e-6, RB, RM))) < 1e-12


def test_decoder_z3_norm_is_local():
    """Scaling one device's tokens scales nothing else: the norm of a token
    row depends on that row only (no communication for the norms)."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((8, 4))
    mesh = [("B", 2), ("M", 2)]
    loc = O.all_slice(O.all_slice(O.replicated(x, mesh), mesh, 0, "B"), mesh, 0, "M")
    g = np.ones(4)
    before = {d: O.rmsnorm(v, g, 1e-6) for d, v in loc.items()}
    loc[(1, 0)] = loc[(1, 0)] * 3.0
    after = {d: O.rmsnorm(v, g, 1e-6) for d, v in loc.items()}
    for d in loc:
        if d != (1, 0):
            assert np.array_equal(after[d], before[d])
    # and the scaled device's rows are normalised to the same values (up to eps)
    assert np.max(np.abs(after[(1, 0)] - before[(1, 0)])) < 1e-5

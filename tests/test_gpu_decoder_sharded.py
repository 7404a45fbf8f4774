"""GPU parity of partir_decoder_layer_sharded: a decoder layer on
device-local arrays under BP + MP + Z3 with sequence-parallel norms.

Small shapes: every residual part against the oracle's lowered SPMD program
(decoder_layer_z3).  The two-layer decoder workload's layer shapes (4 x 2048
tokens, d_model 5120, 40 heads, FFN 13824, mesh {B: 2, M: 4}): bit for bit
equal to partir_decoder_layer on the concatenated residual (same tiles and
K order), and seeded rows against the oracle.
"""
import numpy as np
import pytest
import torch

from oracle import partir_oracle as O
from paper_2401_11202_amd import inputs as I
from paper_2401_11202_amd import partir as P
from tests.gpu_common import TOL_BF16, TOL_REL_FRO, host, rel_fro, say

pytestmark = pytest.mark.gpu


def make(seed, B, S, D, F):
    x = I.gaussian(seed, 0, (B * S, D), 1.0, "f32")
    p = {k: I.gaussian(seed, 1 + i, (D, D), D ** -0.5) for i, k in enumerate(("Wq", "Wk", "Wv", "Wo"))}
    p["W1"] = I.gaussian(seed, 5, (D, F), D ** -0.5)
    p["W2"] = I.gaussian(seed, 6, (F, D), F ** -0.5)
    g1 = I.gaussian(seed, 7, (D,), 0.1, "f32")
    g2 = I.gaussian(seed, 8, (D,), 0.1, "f32")
    return x, p, g1, g2


def gains(g):
    """RMSNorm gains 1 + N(0, 0.01), as float32 on both sides."""
    return (1.0 + g.values).astype(np.float32)


def run_sharded(x, p, g1, g2, B, S, H, RB, RM):
    Wd = {k: v.to_device() for k, v in p.items()}
    xs, parts = P.z3_decoder_arrays(x.to_device(), Wd, RB, RM)
    G1, G2 = torch.from_numpy(gains(g1)).cuda(), torch.from_numpy(gains(g2)).cuda()
    P.decoder_layer_sharded(xs, G1, G2, parts, B=B, S=S, n_heads=H, R_batch=RB, R_model=RM)
    torch.cuda.synchronize()
    return np.concatenate([host(t) for t in xs], axis=0)


def oracle_params(p, g1, g2):
    q = {k: v.f64() for k, v in p.items()}
    q["g1"], q["g2"] = gains(g1).astype(np.float64), gains(g2).astype(np.float64)
    return q


@pytest.mark.parametrize("RB,RM", [(2, 4), (1, 2), (1, 1), (2, 2), (2, 8)])
def test_decoder_sharded_small_every_part(RB, RM):
    B, S, H, F = 2, 256, 8, 2048
    D = H * 128
    x, p, g1, g2 = make(140, B, S, D, F)
    say(f"decoder sharded B={B} S={S} D={D} F={F} mesh B={RB} M={RM}")
    got = run_sharded(x, p, g1, g2, B, S, H, RB, RM)
    q = oracle_params(p, g1, g2)
    x_loc, p_loc = O.z3_local_decoder(x.f64(), q, RB, RM)
    y = O.decoder_layer_z3(x_loc, p_loc, q["g1"], q["g2"], B, S, H, 128, 1e-6, RB, RM)
    ref = np.concatenate([y[(b, m)] for b in range(RB) for m in range(RM)], axis=0)
    _, norm = O.decoder_layer(x.f64(), q, B, S, H, 128, 1e-6, RB, RM, return_norm=True)
    err, fro = O.normalised_error(got, ref, norm), rel_fro(got - x.f64(), ref - x.f64())
    say(f"    max normalised error {err:.3e}, relative Frobenius of the update {fro:.3e}")
    assert err <= TOL_BF16 and fro <= TOL_REL_FRO


def test_decoder_sharded_largest_mesh_every_part():
    """The largest mesh the boundary admits, {B: 3, M: 7} (21 devices, three
    weight groups in the 64-slot part table): every residual part against the
    oracle's lowered SPMD program.  Shapes are the smallest that divide over
    it (tokens over 21 parts, heads and FFN over 7, d_model over 3)."""
    RB, RM = 3, 7
    B, S, H, F = 3, 896, 21, 2688
    D = H * 128
    x, p, g1, g2 = make(141, B, S, D, F)
    say(f"decoder sharded B={B} S={S} D={D} F={F} mesh B={RB} M={RM}")
    got = run_sharded(x, p, g1, g2, B, S, H, RB, RM)
    q = oracle_params(p, g1, g2)
    x_loc, p_loc = O.z3_local_decoder(x.f64(), q, RB, RM)
    y = O.decoder_layer_z3(x_loc, p_loc, q["g1"], q["g2"], B, S, H, 128, 1e-6, RB, RM)
    ref = np.concatenate([y[(b, m)] for b in range(RB) for m in range(RM)], axis=0)
    _, norm = O.decoder_layer(x.f64(), q, B, S, H, 128, 1e-6, RB, RM, return_norm=True)
    err, fro = O.normalised_error(got, ref, norm), rel_fro(got - x.f64(), ref - x.f64())
    say(f"    max normalised error {err:.3e}, relative Frobenius of the update {fro:.3e}")
    assert err <= TOL_BF16 and fro <= TOL_REL_FRO


def test_decoder_sharded_full_size_equals_whole_layer():
    B, S, H, F, RB, RM = 4, 2048, 40, 13824, 2, 4
    D = H * 128
    x, p, g1, g2 = make(141, B, S, D, F)
    say(f"decoder sharded B={B} S={S} D={D} F={F} mesh B={RB} M={RM}")
    got = run_sharded(x, p, g1, g2, B, S, H, RB, RM)
    xw = x.to_device()
    Wd = [p[k].to_device() for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2")]
    G1, G2 = torch.from_numpy(gains(g1)).cuda(), torch.from_numpy(gains(g2)).cuda()
    P.decoder_layer(xw, G1, G2, *Wd, B=B, S=S, n_heads=H, R_batch=RB, R_model=RM)
    torch.cuda.synchronize()
    assert np.array_equal(got, host(xw))
    rows = [0, 1, 200, S - 1]
    q = oracle_params(p, g1, g2)
    ref, norm = O.decoder_layer(x.f64(), q, B, S, H, 128, 1e-6, RB, RM, rows=rows, return_norm=True)
    err = O.normalised_error(got[rows], ref, norm)
    say(f"    rows {rows}: max normalised error {err:.3e}")
    assert err <= TOL_BF16

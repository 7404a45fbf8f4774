"""GPU parity of the attention block's training step: partir_attn_block_train
(forward that keeps Q, K, V, A and lse) and partir_attn_block_backward.

The small twin is compared on every element of every gradient against the
oracle's shard interpreter (attn_block_backward), for two partitions; the
attention-block workload (4 x 2048 tokens, d_model 4096, 32 heads, R = 8)
on dX rows of one sequence and the weight gradients of seeded heads, each
evaluated by the oracle through its owning shards.
"""
import numpy as np
import pytest
import torch

from oracle import partir_oracle as O
from paper_2401_11202_amd import inputs as I
from paper_2401_11202_amd import partir as P
from paper_2401_11202_amd import workloads as W
from tests.gpu_common import TOL_BF16, TOL_REL_FRO, host, rel_fro, say

pytestmark = pytest.mark.gpu
KEYS = ("dX", "dWq", "dWk", "dWv", "dWo")


def run(w, x, dY, Rb, Rm):
    B, S, D, H = w["B"], w["S"], w["D"], w["H"]
    Xd = x["X"].to_device()
    Ws = [x[k].to_device() for k in ("Wq", "Wk", "Wv", "Wo")]
    Y, saved = P.attn_block_train(Xd, *Ws, B=B, S=S, n_heads=H, R_batch=Rb, R_model=Rm)
    Y0 = P.attn_block(Xd, *Ws, B=B, S=S, n_heads=H, R_batch=Rb, R_model=Rm)
    g = P.attn_block_backward(Xd, *Ws, saved, dY.to_device(), B=B, S=S, n_heads=H, R_batch=Rb, R_model=Rm)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y0)          # the training forward computes the same Y
    out = {"dX": host(g[0])}
    for k, t in zip(KEYS[1:], g[1:]):
        out[k] = host(t)               # [fan_in, fan_out], as the weights
    return out


@pytest.mark.parametrize("Rb,Rm", [(1, 8), (2, 4), (1, 1), (2, 8)])
def test_attn_block_backward_small_every_element(Rb, Rm):
    w = W.WORKLOADS["attn_block_small"]
    x = W.make_inputs(w)
    dY = I.gaussian(w.wid, 20, (w["B"] * w["S"], w["D"]), 1.0)
    say(f"attn block backward {w.dims} R_batch={Rb} R_model={Rm}")
    got = run(w, x, dY, Rb, Rm)
    ref, nrm = O.attn_block_backward(x["X"].f64(), x["Wq"].f64(), x["Wk"].f64(), x["Wv"].f64(), x["Wo"].f64(),
                                     dY.f64(), w["B"], w["S"], w["H"], w["dh"], True, None, Rb, Rm,
                                     return_norm=True)
    for k in KEYS:
        err = O.normalised_error(got[k], ref[k], nrm[k])
        fro = rel_fro(got[k], ref[k])
        say(f"    {k}: max normalised error {err:.3e}, relative Frobenius {fro:.3e}")
        assert err <= TOL_BF16 and fro <= TOL_REL_FRO, k


def test_attn_block_backward_one_sequence_one_head_per_shard():
    """Three sequences of the minimum length (128, one query block), three
    heads, mesh 3 x 3: every shard holds one sequence and one head, and the
    model #sum folds three single-head partials; every element."""
    B, S, H, dh = 3, 128, 3, 128
    D = H * dh
    w = {"B": B, "S": S, "D": D, "H": H}
    x = {"X": I.gaussian(133, 0, (B * S, D), 1.0)}
    for i, k in enumerate(("Wq", "Wk", "Wv", "Wo")):
        x[k] = I.gaussian(133, 1 + i, (D, D), D ** -0.5)
    dY = I.gaussian(133, 9, (B * S, D), 1.0)
    say(f"attn block backward B={B} S={S} H={H} R_batch=3 R_model=3")
    got = run(w, x, dY, 3, 3)
    ref, nrm = O.attn_block_backward(x["X"].f64(), x["Wq"].f64(), x["Wk"].f64(), x["Wv"].f64(), x["Wo"].f64(),
                                     dY.f64(), B, S, H, dh, True, None, 3, 3, return_norm=True)
    for k in KEYS:
        err = O.normalised_error(got[k], ref[k], nrm[k])
        fro = rel_fro(got[k], ref[k])
        say(f"    {k}: max normalised error {err:.3e}, relative Frobenius {fro:.3e}")
        assert err <= TOL_BF16 and fro <= TOL_REL_FRO, k


def test_attn_block_backward_full_size_sampled():
    w = W.WORKLOADS["attn_block"]
    x = W.make_inputs(w)
    B, S, D, H, dh = w["B"], w["S"], w["D"], w["H"], w["dh"]
    dY = I.gaussian(w.wid, 20, (B * S, D), 1.0)
    say(f"attn block backward {w.dims}")
    got = run(w, x, dY, w["R_batch"], w["R_model"])
    rng = np.random.default_rng(w.wid)
    seq = B - 1
    rows = sorted({0, S - 1} | set(rng.choice(S, 6, replace=False).tolist()))
    for head in (0, int(rng.integers(1, H))):
        ref, nrm = O.attn_block_backward_sampled(
            x["X"].f64(), x["Wq"].f64(), x["Wk"].f64(), x["Wv"].f64(), x["Wo"].f64(), dY.f64(), B, S, H, dh,
            True, None, w["R_batch"], w["R_model"], seq, rows, head)
        cs = slice(head * dh, (head + 1) * dh)
        picked = {"dX": got["dX"][seq * S + np.array(rows)], "dWq": got["dWq"][:, cs], "dWk": got["dWk"][:, cs],
                  "dWv": got["dWv"][:, cs], "dWo": got["dWo"][cs]}
        for k in KEYS:
            err = O.normalised_error(picked[k], ref[k], nrm[k])
            fro = rel_fro(picked[k], ref[k])
            say(f"    head {head} {k}: max normalised error {err:.3e}, relative Frobenius {fro:.3e}")
            assert err <= TOL_BF16 and fro <= TOL_REL_FRO, k


def test_attn_block_backward_deterministic():
    w = W.WORKLOADS["attn_block_small"]
    x = W.make_inputs(w)
    dY = I.gaussian(w.wid, 20, (w["B"] * w["S"], w["D"]), 1.0)
    a = run(w, x, dY, 1, 8)
    b = run(w, x, dY, 1, 8)
    for k in KEYS:
        assert np.array_equal(a[k], b[k]), k

"""GPU parity of the MLP, attention and decoder entry points against the oracle.

Small twins (same structure and partition sizes, scaled down) are compared on
every output element; the full-size workloads, in the launch configuration
the benchmark times, on a seeded sample of output rows that the oracle
evaluates one by one (exact for the MLP; attention rows get every key they
need).  The error measure is normalised by |A|.|B| of the last contraction
(plus |residual| for the decoder).
"""
import numpy as np
import pytest
import torch

from oracle import partir_oracle as O
from paper_2401_11202_amd import inputs as I
from paper_2401_11202_amd import partir as P
from paper_2401_11202_amd import workloads as W
from tests.gpu_common import TOL_BF16, every_block_rows, host, sample_rows, say

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------------
# MLP
# ---------------------------------------------------------------------------
def run_mlp(w, x, b1=None, b2=None, act="gelu", out_dtype=torch.float32):
    return P.mlp_block(x["X"].to_device(), x["W1"].to_device(), x["W2"].to_device(),
                       b1=None if b1 is None else b1.to_device(), b2=None if b2 is None else b2.to_device(),
                       R_batch=w["R_batch"], R_model=w["R_model"], act=act, out_dtype=out_dtype)


@pytest.mark.parametrize("name", ["mlp_megatron_small", "mlp_batch_x_megatron_small"])
@pytest.mark.parametrize("out", [torch.float32, torch.bfloat16])
def test_mlp_small_full_output(name, out):
    w = W.WORKLOADS[name]
    x = W.make_inputs(w)
    say(f"{name} out={out}")
    Y = run_mlp(w, x, out_dtype=out)
    torch.cuda.synchronize()
    ref, norm = O.mlp_block(x["X"].f64(), x["W1"].f64(), x["W2"].f64(), act="gelu",
                            R_batch=w["R_batch"], R_model=w["R_model"], return_norm=True)
    err = O.normalised_error(host(Y), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16


def test_mlp_small_with_biases():
    w = W.WORKLOADS["mlp_megatron_small"]
    x = W.make_inputs(w)
    b1 = I.gaussian(w.wid, 10, (w["F"],), 0.5, "f32")
    b2 = I.gaussian(w.wid, 11, (w["D"],), 0.5, "f32")
    Y = run_mlp(w, x, b1, b2)
    torch.cuda.synchronize()
    ref, norm = O.mlp_block(x["X"].f64(), x["W1"].f64(), x["W2"].f64(), b1.f64(), b2.f64(), "gelu",
                            w["R_batch"], w["R_model"], return_norm=True)
    assert O.normalised_error(host(Y), ref, norm) <= TOL_BF16
    # b2 is added once after the #sum: removing it changes Y by exactly b2 (to rounding)
    Y0 = run_mlp(w, x, b1, None)
    torch.cuda.synchronize()
    assert np.max(np.abs(host(Y) - host(Y0) - b2.f64())) < 1e-5


def test_gelu_epilogue_values_across_the_range():
    """Y = gelu(X I) I with identity weights stores bf16(GELU(x)) for every
    bf16 value x with 2^-10 <= |x| < 8 (and 0, +-40): within the bf16 unit
    roundoff (2^-8 relative) of the exact GELU plus the epilogue's documented
    5.4e-7 |x|."""
    bits = np.arange(0x3A80, 0x4100, dtype=np.uint32)          # 2^-10 .. just below 8
    pos = (bits << 16).view(np.float32).astype(np.float64)
    xs = np.concatenate([pos, -pos, [0.0, 40.0, -40.0]])
    D = 256
    rows = -(-len(xs) // D)
    X = np.zeros(rows * D, np.float32)
    X[:len(xs)] = xs
    X = X.reshape(rows, D)
    Xd = torch.from_numpy(X).to(torch.bfloat16).cuda()
    assert np.array_equal(Xd.float().cpu().numpy(), X)      # every value exact in bf16
    eye = torch.eye(D, dtype=torch.bfloat16, device="cuda")
    Y = P.mlp_block(Xd, eye, eye, R_batch=1, R_model=1, act="gelu", out_dtype=torch.float32)
    torch.cuda.synchronize()
    got = host(Y).reshape(-1)[:len(xs)]
    ref = O.gelu_erf(xs)
    bound = 2.0 ** -8 * np.abs(ref) + 1e-6 * np.abs(xs) + 1e-30   # bf16 unit roundoff 2^-8
    assert np.all(np.abs(got - ref) <= bound), float(np.max(np.abs(got - ref) / bound))


@pytest.mark.parametrize("Rb,Rm", [(1, 1), (1, 8), (4, 8), (2, 2)])
def test_mlp_integer_exact(Rb, Rm):
    """act = none with entries in {-1, 0, 1}: H is an integer of magnitude <= D
    (exact in bf16 for D <= 256) and Y is exact in fp32, for every nest."""
    T, D, F = 512, 256, 1024
    X = I.small_ints(110, 0, (T, D), -1, 1)
    W1 = I.small_ints(110, 1, (D, F), -1, 1)
    W2 = I.small_ints(110, 2, (F, D), -1, 1)
    Y = P.mlp_block(X.to_device(), W1.to_device(), W2.to_device(), R_batch=Rb, R_model=Rm, act="none",
                    out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.mlp_block(X.f64(), W1.f64(), W2.f64(), act="none", R_batch=Rb, R_model=Rm)
    assert np.array_equal(host(Y), ref)


@pytest.mark.parametrize("Rb,Rm", [(3, 3), (3, 5), (1, 5)])
def test_mlp_integer_exact_odd_nests(Rb, Rm):
    """Odd loop sizes (batch shards of 256 rows, model shards of 320 / 192
    hidden units), act = none, entries in {-1, 0, 1}: exact for every nest."""
    T, D, F = 768, 256, 960
    X = I.small_ints(113, 0, (T, D), -1, 1)
    W1 = I.small_ints(113, 1, (D, F), -1, 1)
    W2 = I.small_ints(113, 2, (F, D), -1, 1)
    Y = P.mlp_block(X.to_device(), W1.to_device(), W2.to_device(), R_batch=Rb, R_model=Rm, act="none",
                    out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.mlp_block(X.f64(), W1.f64(), W2.f64(), act="none", R_batch=Rb, R_model=Rm)
    assert np.array_equal(host(Y), ref)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["mlp_megatron", "mlp_batch_x_megatron"])
def test_mlp_full_size_sampled_rows(name):
    w = W.WORKLOADS[name]
    say(f"{name}: generating inputs")
    x = W.make_inputs(w)
    Y = run_mlp(w, x)
    torch.cuda.synchronize()
    rows = sample_rows(w["T"], w["R_batch"], 64, seed=w.wid)
    say(f"{name}: oracle on {len(rows)} rows")
    ref, norm = O.mlp_block(x["X"].f64(), x["W1"].f64(), x["W2"].f64(), act="gelu",
                            R_batch=w["R_batch"], R_model=w["R_model"], rows=rows, return_norm=True)
    err = O.normalised_error(host(Y[rows]), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------
def run_attn(w, x, causal=True, out_dtype=torch.float32, Rb=None, Rm=None):
    return P.attn_block(x["X"].to_device(), *(x[k].to_device() for k in ("Wq", "Wk", "Wv", "Wo")),
                        B=w["B"], S=w["S"], n_heads=w["H"], d_head=w["dh"], causal=causal,
                        R_batch=w["R_batch"] if Rb is None else Rb, R_model=w["R_model"] if Rm is None else Rm,
                        out_dtype=out_dtype)


def oracle_attn(w, x, causal=True, rows=None, Rb=None, Rm=None):
    return O.attn_block(x["X"].f64(), x["Wq"].f64(), x["Wk"].f64(), x["Wv"].f64(), x["Wo"].f64(),
                        w["B"], w["S"], w["H"], w["dh"], causal, None,
                        w["R_batch"] if Rb is None else Rb, w["R_model"] if Rm is None else Rm,
                        rows=rows, return_norm=True)


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("Rb,Rm", [(1, 8), (2, 4), (1, 1)])
def test_attn_small_full_output(causal, Rb, Rm):
    w = W.WORKLOADS["attn_block_small"]
    x = W.make_inputs(w)
    say(f"attn small causal={causal} Rb={Rb} Rm={Rm}")
    Y = run_attn(w, x, causal, Rb=Rb, Rm=Rm)
    torch.cuda.synchronize()
    ref, norm = oracle_attn(w, x, causal, Rb=Rb, Rm=Rm)
    err = O.normalised_error(host(Y), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16


def test_attn_zero_queries_average_values():
    """Wq = 0 makes every score equal: causal attention returns the running
    mean of V, so Y = prefix_mean(X Wv) Wo; checked against the oracle."""
    w = W.WORKLOADS["attn_block_small"]
    x = W.make_inputs(w)
    x = dict(x)
    x["Wq"] = I.HostTensor(np.zeros_like(x["Wq"].values), "bf16", np.zeros_like(x["Wq"].bits))
    Y = run_attn(w, x)
    torch.cuda.synchronize()
    ref, norm = oracle_attn(w, x)
    V = O.matmul(x["X"].f64(), x["Wv"].f64())
    S = w["S"]
    pm = np.concatenate([np.cumsum(V[s * S:(s + 1) * S], 0) / np.arange(1, S + 1)[:, None]
                         for s in range(w["B"])])
    assert np.max(np.abs(O.matmul(pm, x["Wo"].f64()) - ref)) < 1e-10
    assert O.normalised_error(host(Y), ref, norm) <= TOL_BF16


@pytest.mark.slow
def test_attn_full_size_sampled_rows():
    w = W.WORKLOADS["attn_block"]
    say("attn_block: generating inputs")
    x = W.make_inputs(w)
    Y = run_attn(w, x)
    torch.cuda.synchronize()
    # a row in every 128-query block of the first and the last sequence
    rows = every_block_rows(w["B"], w["S"], (0, w["B"] - 1), seed=w.wid)
    say(f"attn_block: oracle on {len(rows)} rows")
    ref, norm = oracle_attn(w, x, rows=rows)
    err = O.normalised_error(host(Y[rows]), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16


# ---------------------------------------------------------------------------
# decoder
# ---------------------------------------------------------------------------
def run_decoder(w, x):
    xd = x["x"].to_device()
    for p in x["layers"]:
        P.decoder_layer(xd, p["g1"].to_device(), p["g2"].to_device(), p["Wq"].to_device(), p["Wk"].to_device(),
                        p["Wv"].to_device(), p["Wo"].to_device(), p["W1"].to_device(), p["W2"].to_device(),
                        B=w["B"], S=w["S"], n_heads=w["H"], d_head=w["dh"], eps=1e-6,
                        R_batch=w["R_batch"], R_model=w["R_model"])
    torch.cuda.synchronize()
    return xd


def oracle_layers(x):
    return [{k: v.f64() for k, v in p.items()} for p in x["layers"]]


def test_decoder_small_full_output():
    w = W.WORKLOADS["decoder_2layer_small"]
    x = W.make_inputs(w)
    out = run_decoder(w, x)
    ref, norm = O.decoder(x["x"].f64(), oracle_layers(x), w["B"], w["S"], w["H"], w["dh"], 1e-6,
                          w["R_batch"], w["R_model"], return_norm=True)
    err = O.normalised_error(host(out), ref, norm)
    say(f"decoder small: max normalised error {err:.3e}")
    assert err <= TOL_BF16


@pytest.mark.parametrize("Rb,Rm", [(1, 1), (1, 8), (2, 2)])
def test_decoder_small_other_partitions(Rb, Rm):
    """The small decoder under other nests of batch #tile and model #tile /
    #sum (unpartitioned; one head per model shard with F/R = 216; 2 x 2),
    every element against the oracle's shard interpreter for that nest."""
    w = W.WORKLOADS["decoder_2layer_small"]
    x = W.make_inputs(w)
    nest = dict(w.dims, R_batch=Rb, R_model=Rm)
    say(f"decoder small R_batch={Rb} R_model={Rm}")
    out = run_decoder(nest, x)
    ref, norm = O.decoder(x["x"].f64(), oracle_layers(x), w["B"], w["S"], w["H"], w["dh"], 1e-6, Rb, Rm,
                          return_norm=True)
    err = O.normalised_error(host(out), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16


def test_decoder_small_random_gains():
    w = W.WORKLOADS["decoder_2layer_small"]
    x = W.make_inputs(w)
    for li, p in enumerate(x["layers"]):
        p["g1"] = I.gaussian(w.wid, 100 + li, (w["D"],), 1.0, "f32")
        p["g2"] = I.gaussian(w.wid, 200 + li, (w["D"],), 1.0, "f32")
    out = run_decoder(w, x)
    ref, norm = O.decoder(x["x"].f64(), oracle_layers(x), w["B"], w["S"], w["H"], w["dh"], 1e-6,
                          w["R_batch"], w["R_model"], return_norm=True)
    assert O.normalised_error(host(out), ref, norm) <= TOL_BF16


@pytest.mark.slow
def test_decoder_full_size_sampled_rows():
    w = W.WORKLOADS["decoder_2layer"]
    say("decoder_2layer: generating inputs")
    x = W.make_inputs(w)
    out = run_decoder(w, x)
    # a row in every 128-query block of the first and the last sequence (one
    # per batch shard)
    rows = every_block_rows(w["B"], w["S"], (0, w["B"] - 1), seed=w.wid)
    say(f"decoder_2layer: oracle on {len(rows)} rows")
    ref, norm = O.decoder(x["x"].f64(), oracle_layers(x), w["B"], w["S"], w["H"], w["dh"], 1e-6,
                          w["R_batch"], w["R_model"], rows=rows, return_norm=True)
    err = O.normalised_error(host(out[rows]), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16


# ---------------------------------------------------------------------------
# empty operands
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("out", [torch.float32, torch.bfloat16])
def test_mlp_with_empty_ffn_is_the_output_bias(out):
    """F = 0: each model shard is empty, the #sum adds nothing, Y = b2."""
    T, D = 256, 512
    X = I.gaussian(108, 0, (T, D), 1.0, "bf16").to_device()
    b2 = I.gaussian(108, 1, (D,), 1.0, "f32")
    W1 = torch.empty((D, 0), dtype=torch.bfloat16, device="cuda")
    W2 = torch.empty((0, D), dtype=torch.bfloat16, device="cuda")
    say(f"mlp F=0 out={out}")
    Y = P.mlp_block(X, W1, W2, b2=b2.to_device(), R_model=4, out_dtype=out)
    torch.cuda.synchronize()
    ref = O.mlp_block(np.zeros((T, D)), np.zeros((D, 0)), np.zeros((0, D)), None, b2.f64(), "gelu", 1, 4)
    if out == torch.bfloat16:
        ref = I.bf16_to_f32(I.bf16_bits(ref.astype(np.float32))).astype(np.float64)
    assert np.array_equal(host(Y), ref)


def test_decoder_with_empty_ffn_matches_oracle():
    """F = 0: the FFN half adds the empty sum, so only attention updates x."""
    w = W.WORKLOADS["decoder_2layer_small"]
    x = W.make_inputs(w)
    D = w["D"]
    for p in x["layers"]:
        p["W1"] = I.gaussian(w.wid, 300, (D, 0), 1.0, "bf16")
        p["W2"] = I.gaussian(w.wid, 301, (0, D), 1.0, "bf16")
    out = run_decoder(w, x)
    ref, norm = O.decoder(x["x"].f64(), oracle_layers(x), w["B"], w["S"], w["H"], w["dh"], 1e-6,
                          w["R_batch"], w["R_model"], return_norm=True)
    err = O.normalised_error(host(out), ref, norm)
    say(f"decoder F=0: max normalised error {err:.3e}")
    assert err <= TOL_BF16


def test_attention_with_no_tokens_is_a_no_op():
    X = torch.empty((0, 1024), dtype=torch.bfloat16, device="cuda")
    W_ = I.gaussian(109, 0, (1024, 1024), 1.0 / 32, "bf16")
    Wd = W_.to_device()
    Y = P.attn_block(X, Wd, Wd, Wd, Wd, B=0, S=256, n_heads=8, R_model=8)
    torch.cuda.synchronize()
    assert tuple(Y.shape) == (0, 1024)


# ---------------------------------------------------------------------------
# the planner's emitted entry point, executed
# ---------------------------------------------------------------------------
def test_planner_emitted_mlp_call_runs_and_matches_oracle():
    """BP + MP tactics on the MLP program: the planner names partir_mlp_block
    with the loop sizes of its nest; running that call reproduces the oracle."""
    w = W.WORKLOADS["mlp_megatron_small"]
    x = W.make_inputs(w)
    T, D, F = w["T"], w["D"], w["F"]
    prog = (f"mesh B=2 M=8\narg x {T}x{D}\narg w1 {D}x{F}\narg w2 {F}x{D}\n"
            "h = matmul x w1\ng = gelu h\ny = matmul g w2\nret y")
    r = P.propagate(prog, [("B", {"x": 0}), ("M", {"w1": 1})])
    (call,) = r["calls"]
    name, out, *fields = call.split()
    assert name == "partir_mlp_block" and out == "y"
    f = dict(kv.split("=") for kv in fields)
    Rb, Rm = int(f["R_batch"]), int(f["R_model"])
    assert (Rb, Rm) == (2, 8)
    say(f"planner call: {call}")
    Y = P.mlp_block(x["X"].to_device(), x["W1"].to_device(), x["W2"].to_device(), R_batch=Rb, R_model=Rm, act="gelu",
                    out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref, norm = O.mlp_block(x["X"].f64(), x["W1"].f64(), x["W2"].f64(), act="gelu", R_batch=Rb, R_model=Rm,
                            return_norm=True)
    err = O.normalised_error(host(Y), ref, norm)
    say(f"    max normalised error {err:.3e}")
    assert err <= TOL_BF16

"""Workload definitions: shapes, partition sizes and seeded input recipes.

Each workload is a partitioned program of the kinds in the paper (a single
partitioned matmul, the Megatron MLP nest of Sec. 5.2.2, an attention block
with heads tiled and the output projection summed, a batch-tiled nest over
those, and a pre-norm decoder).  Sizes follow the transformer widths of the
paper's evaluation (Sec. 7.1: d_model 4096 with 32 heads, and 8192); the
paper gives no sequence length, S = 2048 is used.  Inputs are synthetic
Gaussian (weights scaled by 1/sqrt(fan_in)); no dataset is involved.

Weight tensors are generated in their logical [fan_in, fan_out] orientation
and stored for the library "output-major" ([fan_out, fan_in], the transpose),
which is the layout the HIP library takes.  Counting FLOPs and bytes is
bookkeeping for the benchmark, not part of the computation.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict

from . import inputs as I


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str                 # matmul | mlp | attn | decoder | attn_core | mlp_train | mlp_z3 | attn_train
                              # | decoder_z3
    wid: int                  # seed id
    dims: Dict[str, int] = field(default_factory=dict)
    dtype: str = "bf16"

    def __getitem__(self, k):
        return self.dims[k]


def _mlp(name, wid, T, D, F, Rb, Rm):
    return Workload(name, "mlp", wid, dict(T=T, D=D, F=F, R_batch=Rb, R_model=Rm))


def _mlp_train(name, wid, T, D, F, Rb, Rm):
    return Workload(name, "mlp_train", wid, dict(T=T, D=D, F=F, R_batch=Rb, R_model=Rm))


def _attn(name, wid, B, S, D, H, dh, Rb, Rm):
    return Workload(name, "attn", wid, dict(B=B, S=S, D=D, H=H, dh=dh, R_batch=Rb, R_model=Rm))


def _dec(name, wid, B, S, D, H, dh, F, L, Rb, Rm):
    return Workload(name, "decoder", wid, dict(B=B, S=S, D=D, H=H, dh=dh, F=F, L=L,
                                               R_batch=Rb, R_model=Rm))


WORKLOADS = {
    # fp32 matmul C[256,256] = A[256,512] B[512,256], #sum over K, R = 4
    "matmul_f32_sumK": Workload("matmul_f32_sumK", "matmul", 1,
                                dict(M=256, N=256, K=512, tile=-1, sum=2, R=4), "f32"),
    # Megatron MLP: W1 #tile over columns, W2 #sum over rows, R = 8
    "mlp_megatron": _mlp("mlp_megatron", 2, 8192, 4096, 16384, 1, 8),
    # attention block: heads #tile (4 heads per shard), W_o #sum, R = 8
    "attn_block": _attn("attn_block", 3, 4, 2048, 4096, 32, 128, 1, 8),
    # batch #tile R1 = 4 outside a Megatron MLP R2 = 8: 32 virtual shards
    "mlp_batch_x_megatron": _mlp("mlp_batch_x_megatron", 4, 16384, 8192, 32768, 4, 8),
    # two-layer pre-norm decoder, batch R = 2 x model R = 4
    "decoder_2layer": _dec("decoder_2layer", 5, 4, 2048, 5120, 40, 128, 13824, 2, 2, 4),
    # attention core alone over one 8192-token sequence with 2 heads (a device's
    # share after head tiling): 128 workgroups leave most of the GPU idle unless
    # the key axis is also a loop, here of R_kv = 4 shards
    "attn_core_long": Workload("attn_core_long", "attn_core", 6, dict(B=1, S=8192, H=2, dh=128, R_kv=4)),
    "attn_core_long_R1": Workload("attn_core_long_R1", "attn_core", 6, dict(B=1, S=8192, H=2, dh=128, R_kv=1)),
    # training step of the Megatron MLP (forward, then the backward nests of
    # the same partition): the model #sum of dX and the batch #sum of the
    # weight gradients
    "mlp_megatron_train": _mlp_train("mlp_megatron_train", 7, 8192, 4096, 16384, 1, 8),
    "mlp_batch_x_megatron_train": _mlp_train("mlp_batch_x_megatron_train", 8, 8192, 4096, 16384, 2, 4),
    # training step of the attention block (forward keeping Q, K, V, A, lse,
    # then every gradient of the same nest)
    "attn_block_train": Workload("attn_block_train", "attn_train", 10,
                                 dict(B=4, S=2048, D=4096, H=32, dh=128, R_batch=1, R_model=8)),
    # the MLP on device-local arrays under BP + MP + Z3 with the activations
    # also sharded over the model axis: mesh {B: 2, M: 4}, 8 devices
    "mlp_z3_sp": Workload("mlp_z3_sp", "mlp_z3", 9, dict(T=8192, D=4096, F=16384, R_batch=2, R_model=4)),
    # the two-layer decoder on device-local arrays (BP + MP + Z3, the residual
    # stream and its norms sharded over the model axis too)
    "decoder_z3_sp": Workload("decoder_z3_sp", "decoder_z3", 5, dict(B=4, S=2048, D=5120, H=40, dh=128, F=13824,
                                                                     L=2, R_batch=2, R_model=4)),
    # small twins: same structure and partition sizes, scaled down
    "mlp_megatron_small": _mlp("mlp_megatron_small", 12, 512, 256, 1024, 1, 8),
    "attn_block_small": _attn("attn_block_small", 13, 2, 256, 1024, 8, 128, 1, 8),
    "mlp_batch_x_megatron_small": _mlp("mlp_batch_x_megatron_small", 14, 1024, 512, 2048, 4, 8),
    "mlp_z3_sp_small": Workload("mlp_z3_sp_small", "mlp_z3", 17, dict(T=1024, D=256, F=1024, R_batch=2,
                                                                      R_model=4)),
    "mlp_train_small": _mlp_train("mlp_train_small", 16, 512, 256, 1024, 2, 4),
    "decoder_2layer_small": _dec("decoder_2layer_small", 15, 2, 256, 1024, 8, 128, 1728, 2, 2, 4),
}


# ---------------------------------------------------------------------------
# Seeded inputs per workload (tensor indices fixed in the order listed)
# ---------------------------------------------------------------------------
def matmul_inputs(w: Workload):
    M, N, K = w["M"], w["N"], w["K"]
    A = I.gaussian(w.wid, 0, (M, K), 1.0, w.dtype)
    B = I.gaussian(w.wid, 1, (K, N), 1.0, w.dtype)
    return dict(A=A, B=B)


def mlp_inputs(w: Workload):
    T, D, F = w["T"], w["D"], w["F"]
    X = I.gaussian(w.wid, 0, (T, D), 1.0)
    W1 = I.gaussian(w.wid, 1, (D, F), D ** -0.5)
    W2 = I.gaussian(w.wid, 2, (F, D), F ** -0.5)
    return dict(X=X, W1=W1, W2=W2)


def mlp_train_inputs(w: Workload):
    """The MLP's inputs plus the output cotangent dY ~ N(0, 1) and b1."""
    x = mlp_inputs(w)
    x["dY"] = I.gaussian(w.wid, 3, (w["T"], w["D"]), 1.0)
    x["b1"] = I.gaussian(w.wid, 4, (w["F"],), 0.5, "f32")
    return x


def mlp_z3_inputs(w: Workload):
    """The MLP's whole operands (the device-local arrays are their blocks)
    plus biases b1 ~ N(0, 1/4), b2 ~ N(0, 1/4)."""
    x = mlp_inputs(w)
    x["b1"] = I.gaussian(w.wid, 4, (w["F"],), 0.5, "f32")
    x["b2"] = I.gaussian(w.wid, 5, (w["D"],), 0.5, "f32")
    return x


def attn_inputs(w: Workload):
    B, S, D = w["B"], w["S"], w["D"]
    X = I.gaussian(w.wid, 0, (B * S, D), 1.0)
    Ws = {n: I.gaussian(w.wid, 1 + i, (D, D), D ** -0.5) for i, n in enumerate(("Wq", "Wk", "Wv", "Wo"))}
    out = dict(X=X, **Ws)
    if w.kind == "attn_train":   # the output cotangent dY ~ N(0, 1)
        out["dY"] = I.gaussian(w.wid, 20, (B * S, D), 1.0)
    return out


def decoder_inputs(w: Workload):
    B, S, D, F, L = w["B"], w["S"], w["D"], w["F"], w["L"]
    x = I.gaussian(w.wid, 0, (B * S, D), 1.0, "f32")
    layers = []
    for l in range(L):
        base = 1 + 10 * l
        p = {n: I.gaussian(w.wid, base + i, (D, D), D ** -0.5) for i, n in enumerate(("Wq", "Wk", "Wv", "Wo"))}
        p["W1"] = I.gaussian(w.wid, base + 4, (D, F), D ** -0.5)
        p["W2"] = I.gaussian(w.wid, base + 5, (F, D), F ** -0.5)
        p["g1"] = I.ones((D,), "f32")
        p["g2"] = I.ones((D,), "f32")
        layers.append(p)
    return dict(x=x, layers=layers)


def attn_core_inputs(w: Workload):
    T, D = w["B"] * w["S"], w["H"] * w["dh"]
    return {n: I.gaussian(w.wid, i, (T, D), 1.0) for i, n in enumerate(("Q", "K", "V"))}


def make_inputs(w: Workload):
    return {"matmul": matmul_inputs, "mlp": mlp_inputs, "attn": attn_inputs,
            "decoder": decoder_inputs, "attn_core": attn_core_inputs, "mlp_train": mlp_train_inputs,
            "mlp_z3": mlp_z3_inputs, "attn_train": attn_inputs, "decoder_z3": decoder_inputs}[w.kind](w)


# ---------------------------------------------------------------------------
# Algorithmic work (what the method must compute; causal attention counts
# only the unmasked key/query pairs)
# ---------------------------------------------------------------------------
def attn_core_flops(B, S, H, dh, causal=True):
    pairs = S * (S + 1) // 2 if causal else S * S
    return 4.0 * B * H * pairs * dh


def flops(w: Workload) -> float:
    if w.kind == "matmul":
        return 2.0 * w["M"] * w["N"] * w["K"]
    if w.kind in ("mlp", "mlp_z3"):
        return 4.0 * w["T"] * w["D"] * w["F"]
    if w.kind == "attn":
        T = w["B"] * w["S"]
        return 8.0 * T * w["D"] * w["D"] + attn_core_flops(w["B"], w["S"], w["H"], w["dh"])
    if w.kind in ("decoder", "decoder_z3"):
        T = w["B"] * w["S"]
        per = 8.0 * T * w["D"] * w["D"] + attn_core_flops(w["B"], w["S"], w["H"], w["dh"]) \
            + 4.0 * T * w["D"] * w["F"]
        return per * w["L"]
    if w.kind == "attn_core":
        return attn_core_flops(w["B"], w["S"], w["H"], w["dh"])
    if w.kind == "mlp_train":
        # forward 4TDF; backward dH, dW2, dW1, dX 8TDF (recomputing Z is not counted)
        return 12.0 * w["T"] * w["D"] * w["F"]
    if w.kind == "attn_train":
        # forward 8TD^2 + core; backward dA, dX, dW{q,k,v}, dWo 16TD^2 + 2.5 x core
        T = w["B"] * w["S"]
        return 24.0 * T * w["D"] * w["D"] + 3.5 * attn_core_flops(w["B"], w["S"], w["H"], w["dh"])
    raise ValueError(w.kind)

"""Host-side tests of the Python binding's argument checks (no GPU needed).

Every tensor handed to the C ABI must match the sizes and dtype codes passed
with it, or the library would read or write past its end.  These calls use
CPU tensors: each bad argument is refused before any pointer reaches the
library, and correct shapes on the CPU are refused for not being on a GPU.
"""
import pytest
import torch

from paper_2401_11202_amd import partir as P

bf, f32 = torch.bfloat16, torch.float32


def t(*shape, dtype=bf):
    return torch.zeros(shape, dtype=dtype)


def status(fn):
    with pytest.raises(P.PartirError) as e:
        fn()
    return P.STATUS[e.value.status]


T, D, F = 64, 32, 48


@pytest.mark.parametrize("args,kw,want", [
    ((t(T, D), t(F, D), t(D, F)), {}, "PARTIR_E_SHAPE"),             # weights given transposed
    ((t(T, D), t(D, F), t(D, F)), {}, "PARTIR_E_SHAPE"),             # W2 not [F, D]
    ((t(T, D, dtype=f32), t(D, F), t(F, D)), {}, "PARTIR_E_DTYPE"),
    ((t(T, D), t(D, F, dtype=f32), t(F, D)), {}, "PARTIR_E_DTYPE"),
    ((t(T, D), t(F, D).t(), t(F, D)), {}, "PARTIR_E_LAYOUT"),         # right shape, not row-major
    ((t(T, D), t(D, F), t(F, D)), {"b1": t(D, dtype=f32)}, "PARTIR_E_SHAPE"),
    ((t(T, D), t(D, F), t(F, D)), {"b2": t(D)}, "PARTIR_E_DTYPE"),
    ((t(T, D), t(D, F), t(F, D)), {"out": t(T, D)}, "PARTIR_E_DTYPE"),     # f32 output by default
    ((t(T, D), t(D, F), t(F, D)), {"out": t(T, D + 8, dtype=f32)}, "PARTIR_E_SHAPE"),
    ((t(T, D), t(D, F), t(F, D)), {}, "PARTIR_E_LAYOUT"),             # all correct, but on the CPU
])
def test_mlp_block_checks(args, kw, want):
    assert status(lambda: P.mlp_block(*args, **kw)) == want


def test_mlp_block_error_names_the_tensor():
    with pytest.raises(P.PartirError, match="W1 has shape"):
        P.mlp_block(t(T, D), t(F, D), t(F, D))
    with pytest.raises(P.PartirError, match="must be on a GPU"):
        P.mlp_block(t(T, D), t(D, F), t(F, D))


def test_mlp_block_train_and_backward_checks():
    X, W1, W2 = t(T, D), t(D, F), t(F, D)
    assert status(lambda: P.mlp_block_train(X, W1, W2, Z=t(T, D))) == "PARTIR_E_SHAPE"
    assert status(lambda: P.mlp_block_backward(X, W1, W2, t(T, F))) == "PARTIR_E_SHAPE"
    assert status(lambda: P.mlp_block_backward(X, W1, W2, t(T, D, dtype=f32))) == "PARTIR_E_DTYPE"
    assert status(lambda: P.mlp_block_backward(X, W1, W2, t(T, D), Z=t(T, F, dtype=f32))) == "PARTIR_E_DTYPE"
    assert status(lambda: P.mlp_block_backward(X, W1, W2, t(T, D))) == "PARTIR_E_LAYOUT"   # CPU


@pytest.mark.parametrize("A,B,kw,want", [
    (t(64, 32), t(48, 16), {}, "PARTIR_E_SHAPE"),                     # B holds K = 48, A K = 32
    (t(64, 32), t(32, 16, dtype=f32), {}, "PARTIR_E_DTYPE"),
    # f32 operands with a bf16 output buffer of the right shape: the fp32
    # epilogue would write twice its size
    (t(64, 32, dtype=f32), t(32, 16, dtype=f32), {"out": t(64, 16)}, "PARTIR_E_LAYOUT"),
    (t(64, 32), t(32, 16), {"out": t(64, 24)}, "PARTIR_E_LAYOUT"),
    (t(64, 32), t(16, 32), {"b_layout": "nk", "out": t(16, 64)}, "PARTIR_E_LAYOUT"),
    (t(64, 32), t(32, 16), {}, "PARTIR_E_LAYOUT"),                    # CPU
])
def test_loop_matmul_checks(A, B, kw, want):
    assert status(lambda: P.loop_matmul(A, B, **kw)) == want


def test_loop_matmul_wrong_output_names_shape_and_dtype():
    """The output check comes before the device check, so the message names
    what is wrong with the buffer."""
    with pytest.raises(P.PartirError, match=r"out is \(64, 16\) torch.bfloat16, expected \[64, 16\] torch.float32"):
        P.loop_matmul(t(64, 32, dtype=f32), t(32, 16, dtype=f32), out=t(64, 16))


def test_attention_entry_point_checks():
    B, S, H = 2, 128, 2
    Dm = H * 128
    X, W = t(B * S, Dm), t(Dm, Dm)
    assert status(lambda: P.attn_block(t(B * S + 8, Dm), W, W, W, W, B=B, S=S, n_heads=H)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.attn_block(X, W, W, W, t(Dm, Dm + 8), B=B, S=S, n_heads=H)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.attn_block(X, W, W, t(Dm, Dm, dtype=f32), W, B=B, S=S, n_heads=H)) == "PARTIR_E_DTYPE"
    assert status(lambda: P.attn_block(X, W, W, W, W, B=B, S=S, n_heads=H)) == "PARTIR_E_LAYOUT"
    Q = t(B * S, Dm)
    assert status(lambda: P.attention(Q, Q, t(B * S, Dm + 8), B=B, S=S, n_heads=H)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.attention_backward(Q, Q, Q, Q, Q, t(B * S, H + 1, dtype=f32), B=B, S=S,
                                               n_heads=H)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.attention_train(Q, Q, Q, lse=t(B * S, H), B=B, S=S, n_heads=H)) == "PARTIR_E_DTYPE"
    assert status(lambda: P.attention_train(Q, Q, Q, lse=t(B * S, H, dtype=f32), B=B, S=S,
                                            n_heads=H)) == "PARTIR_E_LAYOUT"   # CPU


def test_decoder_layer_checks():
    B, S, H = 2, 128, 2
    Dm, Fm = H * 128, 512
    x, g, W = t(B * S, Dm, dtype=f32), t(Dm, dtype=f32), t(Dm, Dm)
    assert status(lambda: P.decoder_layer(x, g, g, W, W, W, W, t(Fm, Dm), t(Fm, Dm), B=B, S=S,
                                          n_heads=H)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.decoder_layer(t(B * S, Dm), g, g, W, W, W, W, t(Dm, Fm), t(Fm, Dm), B=B, S=S,
                                          n_heads=H)) == "PARTIR_E_DTYPE"
    assert status(lambda: P.decoder_layer(x, t(Dm + 1, dtype=f32), g, W, W, W, W, t(Dm, Fm), t(Fm, Dm), B=B,
                                          S=S, n_heads=H)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.decoder_layer(x, g, g, W, W, W, W, t(Dm, Fm), t(Fm, Dm), B=B, S=S,
                                          n_heads=H)) == "PARTIR_E_LAYOUT"


def test_sharded_parts_are_checked():
    xs = [t(16, 64) for _ in range(4)]
    w1 = [t(32, 32) for _ in range(4)]
    w2 = [t(32, 32) for _ in range(4)]
    assert status(lambda: P.mlp_block_sharded(xs, w1, w2[:3], R_batch=2, R_model=2)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.mlp_block_sharded(xs[:3], w1, w2, R_batch=2, R_model=2)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.mlp_block_sharded(xs, w1, [t(32, 16)] * 4, R_batch=2, R_model=2)) == "PARTIR_E_SHAPE"
    assert status(lambda: P.mlp_block_sharded(xs, w1, w2, R_batch=2, R_model=2)) == "PARTIR_E_LAYOUT"   # CPU

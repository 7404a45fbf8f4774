"""Python binding of libpartir (ctypes).

Argument marshalling only: every step of the computation runs in the HIP
library.  PyTorch supplies device memory (outputs and workspaces are
allocated with ``torch.empty``) and the current HIP stream.  If the built
library is missing, every call raises ``PartirError`` -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpartir.so")

F32, BF16 = 0, 1
AXIS_NONE, AXIS_M, AXIS_N, AXIS_K = -1, 0, 1, 2
B_KN, B_NK = 0, 1
SUM_AUTO, SUM_FUSED, SUM_SPLITK = 0, 1, 2
ACT_NONE, ACT_GELU = 0, 1

STATUS = {0: "PARTIR_OK", 1: "PARTIR_E_NULL", 2: "PARTIR_E_SHAPE", 3: "PARTIR_E_DIVISIBILITY",
          4: "PARTIR_E_AXIS", 5: "PARTIR_E_DTYPE", 6: "PARTIR_E_LAYOUT", 7: "PARTIR_E_WORKSPACE",
          8: "PARTIR_E_HIP", 9: "PARTIR_E_UNSUPPORTED"}
ERR = {v: k for k, v in STATUS.items()}

EXPORTS = ("partir_loop_matmul", "partir_loop_matmul_workspace", "partir_mlp_block",
           "partir_mlp_block_workspace", "partir_attn_block", "partir_attn_block_workspace",
           "partir_decoder_layer", "partir_decoder_layer_workspace", "partir_plan_loop_matmul",
           "partir_plan_mlp_block", "partir_plan_attn_block", "partir_plan_decoder_layer",
           "partir_last_plan_text", "partir_trace_enable", "partir_trace_read", "partir_trace_reset",
           "partir_status_string", "partir_last_error", "partir_version", "partir_propagate",
           "partir_attention", "partir_attention_workspace", "partir_plan_attention",
           "partir_mlp_block_backward", "partir_mlp_block_backward_workspace", "partir_plan_mlp_block_backward",
           "partir_mlp_block_train", "partir_mlp_block_sharded", "partir_mlp_block_sharded_workspace",
           "partir_plan_mlp_block_sharded", "partir_attention_train", "partir_attention_backward",
           "partir_attention_backward_workspace", "partir_plan_attention_backward", "partir_attn_block_train",
           "partir_attn_block_saved_bytes", "partir_attn_block_backward", "partir_attn_block_backward_workspace",
           "partir_plan_attn_block_backward", "partir_decoder_layer_sharded",
           "partir_decoder_layer_sharded_workspace", "partir_plan_decoder_layer_sharded")


class PartirError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class PlanInfo(ctypes.Structure):
    _fields_ = [("n_virtual_shards", ctypes.c_int), ("n_tile_loops", ctypes.c_int),
                ("n_sum_loops", ctypes.c_int), ("n_sum_splitk", ctypes.c_int),
                ("n_launches", ctypes.c_int), ("reserved", ctypes.c_int),
                ("workspace_bytes", ctypes.c_size_t), ("flops", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "reserved"}


class TraceEntry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


_lib = None
I64, I32, P, SZ, F = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_float
PP = ctypes.POINTER(ctypes.c_void_p)   # a host array of device pointers


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PartirError(-1, f"{LIB_PATH} is not built; run `python -m paper_2401_11202_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    sig = {
        "partir_loop_matmul": (I32, [P, P, P, I64, I64, I64, I64, I64, I64, I32, I32, I32, I32, I32, I32, I32, P, SZ, P]),
        "partir_loop_matmul_workspace": (SZ, [I64, I64, I64, I32, I32, I32, I32, I32, I32, I32]),
        "partir_mlp_block": (I32, [P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, I32, I32, P, SZ, P]),
        "partir_mlp_block_workspace": (SZ, [I64, I64, I64, I32, I32, I32]),
        "partir_attn_block": (I32, [P, P, P, P, P, P, I64, I64, I64, I64, I64, I32, F, I32, I32, I32, I32, P, SZ, P]),
        "partir_attn_block_workspace": (SZ, [I64, I64, I64, I64, I64, I32, I32]),
        "partir_decoder_layer": (I32, [P, P, P, F, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I32, I32, P, SZ, P]),
        "partir_decoder_layer_workspace": (SZ, [I64, I64, I64, I64, I64, I64, I32, I32]),
        "partir_plan_loop_matmul": (I32, [I64, I64, I64, I32, I32, I32, I32, I32, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_plan_mlp_block": (I32, [I64, I64, I64, I32, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_plan_attn_block": (I32, [I64, I64, I64, I64, I64, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_plan_decoder_layer": (I32, [I64, I64, I64, I64, I64, I64, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_last_plan_text": (ctypes.c_char_p, []),
        "partir_trace_enable": (I32, [I32]),
        "partir_trace_read": (I32, [ctypes.POINTER(TraceEntry), I32]),
        "partir_trace_reset": (None, []),
        "partir_status_string": (ctypes.c_char_p, [I32]),
        "partir_last_error": (ctypes.c_char_p, []),
        "partir_version": (ctypes.c_char_p, []),
        "partir_propagate": (I32, [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_char_p, SZ, ctypes.POINTER(SZ)]),
        "partir_attention": (I32, [P, P, P, P, I64, I64, I64, I64, I32, F, I32, P, SZ, P]),
        "partir_attention_workspace": (SZ, [I64, I64, I64, I64, I32]),
        "partir_plan_attention": (I32, [I64, I64, I64, I64, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_mlp_block_backward": (I32, [P, P, P, P, P, P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, P, SZ, P]),
        "partir_mlp_block_train": (I32, [P, P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, I32, I32, P, SZ, P]),
        "partir_mlp_block_backward_workspace": (SZ, [I64, I64, I64, I32, I32, I32, I32]),
        "partir_plan_mlp_block_backward": (I32, [I64, I64, I64, I32, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_mlp_block_sharded": (I32, [PP, PP, P, PP, P, PP, I64, I64, I64, I32, I32, I32, I32, P, SZ, P]),
        "partir_mlp_block_sharded_workspace": (SZ, [I64, I64, I64, I32, I32]),
        "partir_plan_mlp_block_sharded": (I32, [I64, I64, I64, I32, I32, I32, ctypes.POINTER(PlanInfo)]),
        "partir_decoder_layer_sharded": (I32, [PP, P, P, F, PP, PP, PP, PP, PP, PP, I64, I64, I64, I64, I64, I64, I32,
                                               I32, P, SZ, P]),
        "partir_decoder_layer_sharded_workspace": (SZ, [I64, I64, I64, I64, I64, I64, I32, I32]),
        "partir_plan_decoder_layer_sharded": (I32, [I64, I64, I64, I64, I64, I64, I32, I32,
                                                    ctypes.POINTER(PlanInfo)]),
        "partir_attention_train": (I32, [P, P, P, P, P, I64, I64, I64, I64, I32, F, I32, P, SZ, P]),
        "partir_attention_backward": (I32, [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, I32, F, P, SZ, P]),
        "partir_attention_backward_workspace": (SZ, [I64, I64, I64, I64]),
        "partir_plan_attention_backward": (I32, [I64, I64, I64, I64, I32, ctypes.POINTER(PlanInfo)]),
        "partir_attn_block_train": (I32, [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I32, F, I32, I32, I32, I32,
                                          P, SZ, P]),
        "partir_attn_block_saved_bytes": (SZ, [I64, I64, I64, I64]),
        "partir_attn_block_backward": (I32, [P, P, P, P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I32, F,
                                             I32, I32, P, SZ, P]),
        "partir_attn_block_backward_workspace": (SZ, [I64, I64, I64, I64, I64, I32, I32]),
        "partir_plan_attn_block_backward": (I32, [I64, I64, I64, I64, I64, I32, I32, I32,
                                                  ctypes.POINTER(PlanInfo)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise PartirError(status, lib().partir_last_error().decode())


def _stream(stream):
    import torch
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _dt(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise PartirError(ERR["PARTIR_E_DTYPE"], f"unsupported tensor dtype {t.dtype}")


def _tdt(code: int):
    import torch
    return torch.bfloat16 if code == BF16 else torch.float32


def _rowmajor(t, name):
    if t.dim() != 2:
        raise PartirError(ERR["PARTIR_E_LAYOUT"], f"{name} must be a 2-D row-major tensor")
    if t.numel() == 0:
        return t.shape[1]          # holds no elements: its strides are never used
    if t.stride(1) != 1:
        raise PartirError(ERR["PARTIR_E_LAYOUT"], f"{name} must be a 2-D row-major tensor")
    return t.stride(0)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _workspace(nbytes: int, device, ws):
    import torch
    if nbytes == ctypes.c_size_t(-1).value:
        # invalid arguments: the entry point itself reports the precise status
        return None, 0
    if nbytes == 0:
        return None, 0
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws, ws.numel() * ws.element_size()


def _axis(name):
    return {None: AXIS_NONE, "M": AXIS_M, "N": AXIS_N, "K": AXIS_K}[name]


# ---------------------------------------------------------------------------
def loop_matmul(A, B, *, tile: Optional[str] = None, sum: Optional[str] = None, R: int = 1,
                b_layout: str = "kn", out_dtype=None, sum_impl: str = "auto", out=None,
                workspace=None, stream=None):
    """C = A @ B as a loop over R virtual shards.  tile in {None, 'M', 'N'},
    sum in {None, 'K'}.  b_layout 'kn': B is [K, N]; 'nk': B is given as B^T
    [N, K]."""
    import torch
    M, K = A.shape
    bl = B_KN if b_layout == "kn" else B_NK
    N = B.shape[1] if bl == B_KN else B.shape[0]
    ab = _dt(A)
    cd = ab if out_dtype is None else (BF16 if out_dtype == torch.bfloat16 else F32)
    if ab == F32:
        cd = F32 if out_dtype is None else cd
    si = {"auto": SUM_AUTO, "fused": SUM_FUSED, "splitk": SUM_SPLITK}[sum_impl]
    if out is None:
        out = torch.empty((M, N), dtype=_tdt(cd), device=A.device)
    nbytes = lib().partir_loop_matmul_workspace(M, N, K, ab, cd, bl, _axis(tile), _axis(sum), R, si)
    ws, wsb = _workspace(nbytes, A.device, workspace)
    _check(lib().partir_loop_matmul(_ptr(A), _ptr(B), _ptr(out), M, N, K, _rowmajor(A, "A"), _rowmajor(B, "B"),
                                    _rowmajor(out, "C"), ab, cd, bl, _axis(tile), _axis(sum), R, si,
                                    _ptr(ws), wsb, _stream(stream)))
    return out


def mlp_block_workspace(T, D, F, out_dtype=F32, R_batch=1, R_model=1) -> int:
    return lib().partir_mlp_block_workspace(T, D, F, out_dtype, R_batch, R_model)


def mlp_block(X, W1t, W2t, *, b1=None, b2=None, R_batch: int = 1, R_model: int = 1, act: str = "gelu",
              out_dtype=None, out=None, workspace=None, stream=None):
    """Y = loop b[#tile<0>](R_batch){ loop m[#sum](R_model){ act(X_b W1[:, m] + b1_m) W2[m, :] } + b2 }.
    W1t = W1^T [F, D], W2t = W2^T [D, F], all bf16."""
    import torch
    T, D = X.shape
    F = W1t.shape[0]
    od = F32 if out_dtype in (None, torch.float32) else BF16
    if out is None:
        out = torch.empty((T, D), dtype=_tdt(od), device=X.device)
    ws, wsb = _workspace(mlp_block_workspace(T, D, F, od, R_batch, R_model), X.device, workspace)
    _check(lib().partir_mlp_block(_ptr(X), _ptr(W1t), _ptr(b1), _ptr(W2t), _ptr(b2), _ptr(out), T, D, F,
                                  _dt(X), od, ACT_GELU if act == "gelu" else ACT_NONE, R_batch, R_model,
                                  _ptr(ws), wsb, _stream(stream)))
    return out


def mlp_block_train(X, W1t, W2t, *, b1=None, b2=None, R_batch: int = 1, R_model: int = 1, act: str = "gelu",
                    out_dtype=None, out=None, Z=None, workspace=None, stream=None):
    """mlp_block that also keeps the pre-activation Z = X W1 + b1 [T, F] bf16
    for mlp_block_backward.  Returns (Y, Z)."""
    import torch
    T, D = X.shape
    F = W1t.shape[0]
    od = F32 if out_dtype in (None, torch.float32) else BF16
    if out is None:
        out = torch.empty((T, D), dtype=_tdt(od), device=X.device)
    if Z is None:
        Z = torch.empty((T, F), dtype=torch.bfloat16, device=X.device)
    ws, wsb = _workspace(mlp_block_workspace(T, D, F, od, R_batch, R_model), X.device, workspace)
    _check(lib().partir_mlp_block_train(_ptr(X), _ptr(W1t), _ptr(b1), _ptr(W2t), _ptr(b2), _ptr(out), _ptr(Z),
                                        T, D, F, _dt(X), od, ACT_GELU if act == "gelu" else ACT_NONE, R_batch,
                                        R_model, _ptr(ws), wsb, _stream(stream)))
    return out, Z


def mlp_block_backward(X, W1t, W2t, dY, *, b1=None, Z=None, R_batch: int = 1, R_model: int = 1,
                       act: str = "gelu", bias_grads: bool = False, out=None, workspace=None, stream=None):
    """Gradients of mlp_block w.r.t. X, W1, W2 (and b1, b2 with bias_grads).
    Returns dX [T, D], dW1t [F, D], dW2t [D, F] (fp32; weight gradients in the
    weights' stored layout) and, with bias_grads, db1 [F] and db2 [D].
    ``Z``: the pre-activation kept by mlp_block_train (else recomputed);
    ``out``: a tuple of the result tensors to write into."""
    import torch
    T, D = X.shape
    F = W1t.shape[0]
    a = ACT_GELU if act == "gelu" else ACT_NONE
    f32 = dict(dtype=torch.float32, device=X.device)
    if out is None:
        out = (torch.empty((T, D), **f32), torch.empty((F, D), **f32), torch.empty((D, F), **f32)) + \
            ((torch.empty((F,), **f32), torch.empty((D,), **f32)) if bias_grads else ())
    dX, dW1t, dW2t = out[:3]
    db1, db2 = out[3:5] if bias_grads else (None, None)
    nbytes = lib().partir_mlp_block_backward_workspace(T, D, F, a, int(bias_grads), R_batch, R_model)
    ws, wsb = _workspace(nbytes, X.device, workspace)
    _check(lib().partir_mlp_block_backward(_ptr(X), _ptr(W1t), _ptr(b1), _ptr(W2t), _ptr(dY), _ptr(Z), _ptr(dX),
                                           _ptr(dW1t), _ptr(db1), _ptr(dW2t), _ptr(db2), T, D, F, a, R_batch,
                                           R_model, _ptr(ws), wsb, _stream(stream)))
    return (dX, dW1t, dW2t, db1, db2) if bias_grads else (dX, dW1t, dW2t)


def _ptr_array(ts):
    """Host array of the tensors' device pointers (None for an absent list)."""
    if ts is None:
        return None
    arr = (ctypes.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = None if t is None else t.data_ptr()
    return arr


def mlp_block_sharded(X_parts, W1t_parts, W2t_parts, *, R_batch: int, R_model: int, b1=None, b2=None,
                      act: str = "gelu", out_dtype=None, out_parts=None, workspace=None, stream=None):
    """The MLP block on device-local arrays (BP + MP + Z3, activations sharded
    over the model axis).  Part p = b * R_model + m of the mesh {B, M}:
    X_parts[p] [T/(R_batch R_model), D]; W1t_parts[p] = W1t[F/R_model rows m,
    D/R_batch cols b]; W2t_parts[p] = W2t[D/R_batch rows b, F/R_model cols m].
    Returns the list of Y parts (token rows p of Y)."""
    import torch
    nd = R_batch * R_model
    rows, D = X_parts[0].shape
    T = rows * nd
    F = W1t_parts[0].shape[0] * R_model
    od = F32 if out_dtype in (None, torch.float32) else BF16
    if out_parts is None:
        out_parts = [torch.empty((rows, D), dtype=_tdt(od), device=X_parts[0].device) for _ in range(nd)]
    ws, wsb = _workspace(lib().partir_mlp_block_sharded_workspace(T, D, F, R_batch, R_model), X_parts[0].device,
                         workspace)
    xs, w1s, w2s, ys = (_ptr_array(v) for v in (X_parts, W1t_parts, W2t_parts, out_parts))
    _check(lib().partir_mlp_block_sharded(xs, w1s, _ptr(b1), w2s, _ptr(b2), ys, T, D, F, od,
                                          ACT_GELU if act == "gelu" else ACT_NONE, R_batch, R_model,
                                          _ptr(ws), wsb, _stream(stream)))
    return out_parts


def z3_device_arrays(X, W1t, W2t, R_batch: int, R_model: int):
    """Copies whole operands into the device-local arrays mlp_block_sharded
    takes (each part its own allocation): X by token blocks p = b * R_model +
    m; W1t block (rows m, cols b); W2t block (rows b, cols m)."""
    nd = R_batch * R_model
    T, D = X.shape
    F = W1t.shape[0]
    tr, dr, fr = T // nd, D // R_batch, F // R_model
    xs = [X[p * tr:(p + 1) * tr].clone() for p in range(nd)]
    w1 = [W1t[m * fr:(m + 1) * fr, b * dr:(b + 1) * dr].contiguous() for b in range(R_batch) for m in range(R_model)]
    w2 = [W2t[b * dr:(b + 1) * dr, m * fr:(m + 1) * fr].contiguous() for b in range(R_batch) for m in range(R_model)]
    return xs, w1, w2


def z3_decoder_arrays(x, W, R_batch: int, R_model: int):
    """Device-local arrays of a decoder layer (each its own allocation): x
    (fp32 [T, D]) by token blocks; W = {name: stored W^T} with Wq, Wk, Wv, W1
    split as (rows block m, cols block b) and Wo, W2 as (rows block b, cols
    block m), part p = b * R_model + m.  Returns (x_parts, {name: parts})."""
    nd = R_batch * R_model
    T = x.shape[0]
    xs = [x[p * (T // nd):(p + 1) * (T // nd)].clone() for p in range(nd)]
    parts = {}
    for k, w in W.items():
        rows, cols = w.shape
        col_par = k in ("Wq", "Wk", "Wv", "W1")
        rr, cc = (rows // R_model, cols // R_batch) if col_par else (rows // R_batch, cols // R_model)
        out = []
        for b in range(R_batch):
            for m in range(R_model):
                i, j = (m, b) if col_par else (b, m)
                out.append(w[i * rr:(i + 1) * rr, j * cc:(j + 1) * cc].contiguous())
        parts[k] = out
    return xs, parts


def decoder_layer_sharded(x_parts, g1, g2, W_parts, *, B: int, S: int, n_heads: int, d_head: int = 128,
                          R_batch: int = 1, R_model: int = 1, eps: float = 1e-6, workspace=None, stream=None):
    """One decoder layer on device-local arrays, x_parts updated in place
    (see z3_decoder_arrays for the layout)."""
    D = x_parts[0].shape[1]
    F = W_parts["W1"][0].shape[0] * R_model
    nbytes = lib().partir_decoder_layer_sharded_workspace(B, S, D, n_heads, d_head, F, R_batch, R_model)
    ws, wsb = _workspace(nbytes, x_parts[0].device, workspace)
    ws_ = [_ptr_array(W_parts[k]) for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2")]
    _check(lib().partir_decoder_layer_sharded(_ptr_array(x_parts), _ptr(g1), _ptr(g2), eps, *ws_, B, S, D, n_heads,
                                              d_head, F, R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return x_parts


def plan_decoder_layer_sharded(B, S, D, n_heads, d_head=128, F=0, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_decoder_layer_sharded, B, S, D, n_heads, d_head, F, R_batch, R_model)


def plan_mlp_block_sharded(T, D, F, act=ACT_GELU, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_mlp_block_sharded, T, D, F, act, R_batch, R_model)


def plan_mlp_block_backward(T, D, F, act=ACT_GELU, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_mlp_block_backward, T, D, F, act, R_batch, R_model)


def attn_block_workspace(B, S, D, n_heads, d_head=128, R_batch=1, R_model=1) -> int:
    return lib().partir_attn_block_workspace(B, S, D, n_heads, d_head, R_batch, R_model)


def attn_block(X, Wq_t, Wk_t, Wv_t, Wo_t, *, B: int, S: int, n_heads: int, d_head: int = 128,
               causal: bool = True, scale: float = 0.0, R_batch: int = 1, R_model: int = 1,
               out_dtype=None, out=None, workspace=None, stream=None):
    import torch
    T, D = X.shape
    od = F32 if out_dtype in (None, torch.float32) else BF16
    if out is None:
        out = torch.empty((T, D), dtype=_tdt(od), device=X.device)
    ws, wsb = _workspace(attn_block_workspace(B, S, D, n_heads, d_head, R_batch, R_model), X.device, workspace)
    _check(lib().partir_attn_block(_ptr(X), _ptr(Wq_t), _ptr(Wk_t), _ptr(Wv_t), _ptr(Wo_t), _ptr(out),
                                   B, S, D, n_heads, d_head, int(causal), float(scale), _dt(X), od,
                                   R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return out


def attention(Q, K, V, *, B: int, S: int, n_heads: int, d_head: int = 128, causal: bool = True,
              scale: float = 0.0, R_kv: int = 1, out=None, workspace=None, stream=None):
    """O = softmax attention per (sequence, head), the key axis a loop of R_kv
    shards reduced with the (max, sum, output) combiner.  Q, K, V, O: [B*S, n_heads*d_head] bf16."""
    import torch
    T, D = Q.shape
    if out is None:
        out = torch.empty((T, D), dtype=torch.bfloat16, device=Q.device)
    nbytes = lib().partir_attention_workspace(B, S, n_heads, d_head, R_kv)
    ws, wsb = _workspace(nbytes, Q.device, workspace)
    _check(lib().partir_attention(_ptr(Q), _ptr(K), _ptr(V), _ptr(out), B, S, n_heads, d_head, int(causal),
                                  float(scale), R_kv, _ptr(ws), wsb, _stream(stream)))
    return out


def attention_train(Q, K, V, *, B: int, S: int, n_heads: int, d_head: int = 128, causal: bool = True,
                    scale: float = 0.0, R_kv: int = 1, out=None, lse=None, workspace=None, stream=None):
    """attention that also returns the per-row base-2 log-sum-exp [B*S, n_heads]
    fp32 for attention_backward.  Returns (O, lse)."""
    import torch
    if out is None:
        out = torch.empty_like(Q)
    if lse is None:
        lse = torch.empty((B * S, n_heads), dtype=torch.float32, device=Q.device)
    ws, wsb = _workspace(lib().partir_attention_workspace(B, S, n_heads, d_head, R_kv), Q.device, workspace)
    _check(lib().partir_attention_train(_ptr(Q), _ptr(K), _ptr(V), _ptr(out), _ptr(lse), B, S, n_heads, d_head,
                                        int(causal), scale, R_kv, _ptr(ws), wsb, _stream(stream)))
    return out, lse


def attention_backward(Q, K, V, O, dO, lse, *, B: int, S: int, n_heads: int, d_head: int = 128,
                       causal: bool = True, scale: float = 0.0, out=None, workspace=None, stream=None):
    """Gradients (dQ, dK, dV) of attention for the output cotangent dO (bf16,
    the layout of Q, K, V), from the forward's O and lse."""
    import torch
    if out is None:
        out = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V))
    ws, wsb = _workspace(lib().partir_attention_backward_workspace(B, S, n_heads, d_head), Q.device, workspace)
    _check(lib().partir_attention_backward(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(lse), _ptr(out[0]),
                                           _ptr(out[1]), _ptr(out[2]), B, S, n_heads, d_head, int(causal), scale,
                                           _ptr(ws), wsb, _stream(stream)))
    return out


def attn_block_train(X, Wq_t, Wk_t, Wv_t, Wo_t, *, B: int, S: int, n_heads: int, d_head: int = 128,
                     causal: bool = True, scale: float = 0.0, R_batch: int = 1, R_model: int = 1, out=None,
                     saved=None, workspace=None, stream=None):
    """attn_block that also keeps Q, K, V, A and lse in `saved` (a uint8
    tensor) for attn_block_backward.  Returns (Y, saved)."""
    import torch
    T, D = X.shape
    if out is None:
        out = torch.empty((T, D), dtype=torch.float32, device=X.device)
    if saved is None:
        saved = torch.empty(max(1, lib().partir_attn_block_saved_bytes(B, S, D, n_heads)), dtype=torch.uint8,
                            device=X.device)
    ws, wsb = _workspace(attn_block_workspace(B, S, D, n_heads, d_head, R_batch, R_model), X.device, workspace)
    _check(lib().partir_attn_block_train(_ptr(X), _ptr(Wq_t), _ptr(Wk_t), _ptr(Wv_t), _ptr(Wo_t), _ptr(out),
                                         _ptr(saved), B, S, D, n_heads, d_head, int(causal), scale, _dt(X),
                                         _dt(out), R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return out, saved


def attn_block_backward(X, Wq_t, Wk_t, Wv_t, Wo_t, saved, dY, *, B: int, S: int, n_heads: int,
                        d_head: int = 128, causal: bool = True, scale: float = 0.0, R_batch: int = 1,
                        R_model: int = 1, out=None, workspace=None, stream=None):
    """Gradients (dX, dWq_t, dWk_t, dWv_t, dWo_t), fp32, weights' stored layout."""
    import torch
    T, D = X.shape
    f32 = dict(dtype=torch.float32, device=X.device)
    if out is None:
        out = (torch.empty((T, D), **f32),) + tuple(torch.empty((D, D), **f32) for _ in range(4))
    ws, wsb = _workspace(lib().partir_attn_block_backward_workspace(B, S, D, n_heads, d_head, R_batch, R_model),
                         X.device, workspace)
    _check(lib().partir_attn_block_backward(_ptr(X), _ptr(Wq_t), _ptr(Wk_t), _ptr(Wv_t), _ptr(Wo_t), _ptr(saved),
                                            _ptr(dY), *(_ptr(o) for o in out), B, S, D, n_heads, d_head,
                                            int(causal), scale, R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return out


def plan_attn_block_backward(B, S, D, n_heads, d_head=128, causal=True, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_attn_block_backward, B, S, D, n_heads, d_head, int(causal), R_batch, R_model)


def plan_attention_backward(B, S, n_heads, d_head=128, causal=True):
    return _plan(lib().partir_plan_attention_backward, B, S, n_heads, d_head, int(causal))


def plan_attention(B, S, n_heads, d_head=128, causal=True, R_kv=1):
    return _plan(lib().partir_plan_attention, B, S, n_heads, d_head, int(causal), R_kv)


def decoder_layer_workspace(B, S, D, n_heads, d_head, F, R_batch=1, R_model=1) -> int:
    return lib().partir_decoder_layer_workspace(B, S, D, n_heads, d_head, F, R_batch, R_model)


def decoder_layer(x, g1, g2, Wq_t, Wk_t, Wv_t, Wo_t, W1t, W2t, *, B: int, S: int, n_heads: int,
                  d_head: int = 128, eps: float = 1e-6, R_batch: int = 1, R_model: int = 1,
                  workspace=None, stream=None):
    """In place on the fp32 residual stream x [B*S, D]."""
    T, D = x.shape
    F = W1t.shape[0]
    ws, wsb = _workspace(decoder_layer_workspace(B, S, D, n_heads, d_head, F, R_batch, R_model), x.device, workspace)
    _check(lib().partir_decoder_layer(_ptr(x), _ptr(g1), _ptr(g2), float(eps), _ptr(Wq_t), _ptr(Wk_t), _ptr(Wv_t),
                                      _ptr(Wo_t), _ptr(W1t), _ptr(W2t), B, S, D, n_heads, d_head, F,
                                      R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return x


# ---------------------------------------------------------------------------
def _plan(fn, *args):
    info = PlanInfo()
    _check(fn(*args, ctypes.byref(info)))
    d = info.as_dict()
    d["text"] = lib().partir_last_plan_text().decode()
    return d


def plan_loop_matmul(M, N, K, ab=BF16, c=F32, b_layout=B_NK, tile=None, sum=None, R=1, sum_impl=SUM_AUTO):
    return _plan(lib().partir_plan_loop_matmul, M, N, K, ab, c, b_layout, _axis(tile), _axis(sum), R, sum_impl)


def plan_mlp_block(T, D, F, out_dtype=F32, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_mlp_block, T, D, F, out_dtype, R_batch, R_model)


def plan_attn_block(B, S, D, n_heads, d_head=128, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_attn_block, B, S, D, n_heads, d_head, R_batch, R_model)


def plan_decoder_layer(B, S, D, n_heads, d_head, F, R_batch=1, R_model=1):
    return _plan(lib().partir_plan_decoder_layer, B, S, D, n_heads, d_head, F, R_batch, R_model)


def trace_enable(on: bool = True):
    _check(lib().partir_trace_enable(int(on)))


def trace_reset():
    lib().partir_trace_reset()


def trace_read():
    """{kernel name: (launches, total_ms)} since the last reset."""
    n = lib().partir_trace_read(None, 0)
    if n < 0:
        raise PartirError(-n, lib().partir_last_error().decode())
    buf = (TraceEntry * max(n, 1))()
    n = lib().partir_trace_read(buf, n)
    return {buf[i].name.decode(): (buf[i].launches, buf[i].total_ms) for i in range(n)}


# ---------------------------------------------------------------------------
# planner (host only)
# ---------------------------------------------------------------------------
def schedule_text(schedule) -> str:
    """[(axis, {name: dim, ...}), ...] -> the planner's schedule text: one
    ManualPartition tactic per line."""
    return "\n".join("partition " + axis + " " + " ".join(f"{n}:{d}" for n, d in parts.items())
                     for axis, parts in schedule)


def propagate_text(program: str, schedule: str) -> str:
    """Run partir_propagate and return its report text."""
    need = SZ(0)
    buf = ctypes.create_string_buffer(1 << 16)
    st = lib().partir_propagate(program.encode(), schedule.encode(), buf, len(buf), ctypes.byref(need))
    if st == ERR["PARTIR_E_WORKSPACE"] and need.value > len(buf):
        buf = ctypes.create_string_buffer(need.value)
        st = lib().partir_propagate(program.encode(), schedule.encode(), buf, len(buf), ctypes.byref(need))
    _check(st)
    return buf.value.decode()


def parse_report(text: str) -> dict:
    """Report text -> {'actions': [...], 'loops': {op: [(axis, action)]},
    'operands': {(op, i): {axis: dim}}, 'values': {name: {axis: dim}},
    'gathers': [(op, value, axis)], 'reshards': [...], 'conflicts': [(op, axis)],
    'calls': [str], 'nests': [op]}."""
    r = {"actions": [], "loops": {}, "kinds": {}, "operands": {}, "operand_names": {}, "values": {},
         "gathers": [], "reshards": [], "conflicts": [], "calls": [], "nests": []}
    for line in text.splitlines():
        t = line.split()
        if not t:
            continue
        if t[0] == "action":
            r["actions"].append(" ".join(t[1:]))
            if t[1] == "conflict":
                r["conflicts"].append((t[2], t[3]))
        elif t[0] == "loop":
            r["kinds"][t[1]] = t[2]
            r["loops"][t[1]] = [] if t[3:] == ["none"] else [tuple(x.split(":")) for x in t[3:]]
        elif t[0] == "operand":
            r["operands"][(t[1], int(t[2]))] = {a: int(d) for a, d in (x.split(":") for x in t[4:])}
            r["operand_names"][(t[1], int(t[2]))] = t[3]
        elif t[0] in ("gather", "reshard"):
            r[t[0] + "s"].append((t[1], t[2], t[3]))
        elif t[0] == "value":
            r["values"][t[1]] = {} if t[2:] == ["replicated"] else {a: int(d) for a, d in (x.split(":") for x in t[2:])}
        elif t[0] == "call":
            r["calls"].append(" ".join(t[1:]))
        elif t[0] == "nest":
            r["nests"].append(t[1])
    return r


def propagate(program: str, schedule) -> dict:
    """Partition `program` with a schedule of ManualPartition tactics
    [(axis, {name: dim})] (or schedule text) and return the parsed report."""
    text = schedule if isinstance(schedule, str) else schedule_text(schedule)
    return parse_report(propagate_text(program, text))

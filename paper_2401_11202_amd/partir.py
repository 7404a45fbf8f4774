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
           "partir_decoder_layer_sharded_workspace", "partir_plan_decoder_layer_sharded",
           "partir_loop_matmul_noalloc")


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
        "partir_loop_matmul_noalloc": (I32, [P, P, P, I64, I64, I64, I64, I64, I64, I32, I32, I32, I32, I32, I32, I32,
                                             P]),
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


# ---------------------------------------------------------------------------
# argument checks: every tensor handed to the C ABI must match the sizes and
# dtype codes passed with it (the library trusts them)
# ---------------------------------------------------------------------------
def _bad(status: str, msg: str):
    raise PartirError(ERR[status], msg)


def _req(t, name: str, shape, dtype, device=None):
    """A dense row-major tensor of exactly `shape` and `dtype` (on `device`)."""
    import torch
    if not isinstance(t, torch.Tensor):
        _bad("PARTIR_E_NULL", f"{name} must be a tensor")
    if t.dtype != dtype:
        _bad("PARTIR_E_DTYPE", f"{name} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(int(v) for v in shape):
        _bad("PARTIR_E_SHAPE", f"{name} has shape {tuple(t.shape)}, expected {tuple(int(v) for v in shape)}")
    if t.numel() > 0 and not t.is_contiguous():
        _bad("PARTIR_E_LAYOUT", f"{name} must be contiguous (row-major)")
    if device is not None and t.device != device:
        _bad("PARTIR_E_LAYOUT", f"{name} is on {t.device}, expected {device}")
    return t


def _opt(t, name, shape, dtype, device=None):
    return None if t is None else _req(t, name, shape, dtype, device)


def _gpu(t, name: str):
    """The device every operand of the call lives on (a GPU)."""
    if t.device.type != "cuda":
        _bad("PARTIR_E_LAYOUT", f"{name} must be on a GPU (got {t.device})")
    return t.device


def _gpu_all(**named):
    """Every operand on one GPU, the first one's (checked after shapes and
    dtypes, so that those errors are reported for CPU tensors too)."""
    dev = None
    for name, t in named.items():
        ts = t if isinstance(t, (list, tuple)) else [t]
        for i, u in enumerate(ts):
            if u is None:
                continue
            nm = name if len(ts) == 1 and not isinstance(t, (list, tuple)) else f"{name}[{i}]"
            if dev is None:
                dev = _gpu(u, nm)
            elif u.device != dev:
                _bad("PARTIR_E_LAYOUT", f"{nm} is on {u.device}, expected {dev}")
    return dev


def _on_stream(stream, *tensors):
    """Kernels run on `stream`: tensors allocated here on the current stream
    are marked as used there, so the caching allocator does not hand their
    memory out again before those kernels finish."""
    import torch
    if isinstance(stream, torch.cuda.Stream) and stream != torch.cuda.current_stream(stream.device):
        for t in tensors:
            if t is not None and t.numel() > 0:
                t.record_stream(stream)


def _workspace(nbytes: int, device, ws):
    import torch
    if nbytes == ctypes.c_size_t(-1).value:
        # invalid arguments: the entry point itself reports the precise status
        return None, 0
    if nbytes == 0:
        return None, 0
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    elif ws.device != device or not ws.is_contiguous():
        _bad("PARTIR_E_WORKSPACE", f"workspace must be a contiguous buffer on {device}")
    return ws, ws.numel() * ws.element_size()


def _axis(name):
    return {None: AXIS_NONE, "M": AXIS_M, "N": AXIS_N, "K": AXIS_K}[name]


def _bf16():
    import torch
    return torch.bfloat16


def _f32():
    import torch
    return torch.float32


# ---------------------------------------------------------------------------
# Each wrapper checks shapes and dtypes of every tensor first, then that all
# of them live on one GPU, then allocates what the caller did not pass.
def loop_matmul(A, B, *, tile: Optional[str] = None, sum: Optional[str] = None, R: int = 1,
                b_layout: str = "kn", out_dtype=None, sum_impl: str = "auto", out=None,
                workspace=None, stream=None):
    """C = A @ B as a loop over R virtual shards.  tile in {None, 'M', 'N'},
    sum in {None, 'K'}.  b_layout 'kn': B is [K, N]; 'nk': B is given as B^T
    [N, K].  A, B and C may be row-major views with a leading dim."""
    import torch
    lda, ldb = _rowmajor(A, "A"), _rowmajor(B, "B")
    M, K = A.shape
    bl = B_KN if b_layout == "kn" else B_NK
    Kb, N = (B.shape[0], B.shape[1]) if bl == B_KN else (B.shape[1], B.shape[0])
    if Kb != K:
        _bad("PARTIR_E_SHAPE", f"B holds K = {Kb}, A holds K = {K}")
    ab = _dt(A)
    if B.dtype != A.dtype:
        _bad("PARTIR_E_DTYPE", f"A is {A.dtype}, B is {B.dtype}")
    cd = ab if out_dtype is None else (BF16 if out_dtype == torch.bfloat16 else F32)
    if ab == F32:
        cd = F32 if out_dtype is None else cd
    si = {"auto": SUM_AUTO, "fused": SUM_FUSED, "splitk": SUM_SPLITK}[sum_impl]
    if out is not None:
        _rowmajor(out, "C")
        if tuple(out.shape) != (M, N) or out.dtype != _tdt(cd):
            _bad("PARTIR_E_LAYOUT", f"out is {tuple(out.shape)} {out.dtype}, expected [{M}, {N}] {_tdt(cd)}")
    dev = _gpu_all(A=A, B=B, out=out)
    fresh = out is None
    if fresh:
        out = torch.empty((M, N), dtype=_tdt(cd), device=dev)
    nbytes = lib().partir_loop_matmul_workspace(M, N, K, ab, cd, bl, _axis(tile), _axis(sum), R, si)
    ws, wsb = _workspace(nbytes, dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh else None)
    _check(lib().partir_loop_matmul(_ptr(A), _ptr(B), _ptr(out), M, N, K, lda, ldb,
                                    _rowmajor(out, "C"), ab, cd, bl, _axis(tile), _axis(sum), R, si,
                                    _ptr(ws), wsb, _stream(stream)))
    return out


def loop_matmul_noalloc(A, B, *, tile: Optional[str] = None, sum: Optional[str] = None, R: int = 1,
                        b_layout: str = "kn", out_dtype=None, sum_impl: str = "auto", out, stream=None):
    """loop_matmul without a workspace: the library's per-GPU scratch array
    holds the #sum partials (see partir_loop_matmul_noalloc).  `out` must be
    given (this call allocates nothing)."""
    import torch
    lda, ldb = _rowmajor(A, "A"), _rowmajor(B, "B")
    M, K = A.shape
    bl = B_KN if b_layout == "kn" else B_NK
    Kb, N = (B.shape[0], B.shape[1]) if bl == B_KN else (B.shape[1], B.shape[0])
    if Kb != K:
        _bad("PARTIR_E_SHAPE", f"B holds K = {Kb}, A holds K = {K}")
    ab = _dt(A)
    if B.dtype != A.dtype:
        _bad("PARTIR_E_DTYPE", f"A is {A.dtype}, B is {B.dtype}")
    cd = ab if out_dtype is None else (BF16 if out_dtype == torch.bfloat16 else F32)
    ldc = _rowmajor(out, "C")
    if tuple(out.shape) != (M, N) or out.dtype != _tdt(cd):
        _bad("PARTIR_E_LAYOUT", f"out is {tuple(out.shape)} {out.dtype}, expected [{M}, {N}] {_tdt(cd)}")
    _gpu_all(A=A, B=B, out=out)
    si = {"auto": SUM_AUTO, "fused": SUM_FUSED, "splitk": SUM_SPLITK}[sum_impl]
    _check(lib().partir_loop_matmul_noalloc(_ptr(A), _ptr(B), _ptr(out), M, N, K, lda, ldb, ldc, ab, cd, bl,
                                            _axis(tile), _axis(sum), R, si, _stream(stream)))
    return out


def mlp_block_workspace(T, D, F, out_dtype=F32, R_batch=1, R_model=1) -> int:
    return lib().partir_mlp_block_workspace(T, D, F, out_dtype, R_batch, R_model)


def _mlp_shapes(X, W1, W2, b1, b2):
    bf = _bf16()
    if X.dim() != 2 or W1.dim() != 2:
        _bad("PARTIR_E_SHAPE", "X and W1 must be 2-D")
    T, D = X.shape
    F = W1.shape[1]
    _req(X, "X", (T, D), bf)
    _req(W1, "W1", (D, F), bf)
    _req(W2, "W2", (F, D), bf)
    _opt(b1, "b1", (F,), _f32())
    _opt(b2, "b2", (D,), _f32())
    return T, D, F


def _out_dtype(out_dtype):
    import torch
    return F32 if out_dtype in (None, torch.float32) else BF16


def mlp_block(X, W1, W2, *, b1=None, b2=None, R_batch: int = 1, R_model: int = 1, act: str = "gelu",
              out_dtype=None, out=None, workspace=None, stream=None):
    """Y = loop b[#tile<0>](R_batch){ loop m[#sum](R_model){ act(X_b W1[:, m] + b1_m) W2[m, :] } + b2 }.
    X [T, D], W1 [D, F], W2 [F, D] bf16 ([fan_in, fan_out]); b1 [F], b2 [D] fp32."""
    import torch
    T, D, F = _mlp_shapes(X, W1, W2, b1, b2)
    od = _out_dtype(out_dtype)
    _opt(out, "out", (T, D), _tdt(od))
    dev = _gpu_all(X=X, W1=W1, W2=W2, b1=b1, b2=b2, out=out)
    fresh = out is None
    if fresh:
        out = torch.empty((T, D), dtype=_tdt(od), device=dev)
    ws, wsb = _workspace(mlp_block_workspace(T, D, F, od, R_batch, R_model), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh else None)
    _check(lib().partir_mlp_block(_ptr(X), _ptr(W1), _ptr(b1), _ptr(W2), _ptr(b2), _ptr(out), T, D, F,
                                  BF16, od, ACT_GELU if act == "gelu" else ACT_NONE, R_batch, R_model,
                                  _ptr(ws), wsb, _stream(stream)))
    return out


def mlp_block_train(X, W1, W2, *, b1=None, b2=None, R_batch: int = 1, R_model: int = 1, act: str = "gelu",
                    out_dtype=None, out=None, Z=None, workspace=None, stream=None):
    """mlp_block that also keeps the pre-activation Z = X W1 + b1 [T, F] bf16
    for mlp_block_backward.  Returns (Y, Z)."""
    import torch
    T, D, F = _mlp_shapes(X, W1, W2, b1, b2)
    od = _out_dtype(out_dtype)
    _opt(out, "out", (T, D), _tdt(od))
    _opt(Z, "Z", (T, F), _bf16())
    dev = _gpu_all(X=X, W1=W1, W2=W2, b1=b1, b2=b2, out=out, Z=Z)
    fresh_y, fresh_z = out is None, Z is None
    if fresh_y:
        out = torch.empty((T, D), dtype=_tdt(od), device=dev)
    if fresh_z:
        Z = torch.empty((T, F), dtype=torch.bfloat16, device=dev)
    ws, wsb = _workspace(mlp_block_workspace(T, D, F, od, R_batch, R_model), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh_y else None, Z if fresh_z else None)
    _check(lib().partir_mlp_block_train(_ptr(X), _ptr(W1), _ptr(b1), _ptr(W2), _ptr(b2), _ptr(out), _ptr(Z),
                                        T, D, F, BF16, od, ACT_GELU if act == "gelu" else ACT_NONE, R_batch,
                                        R_model, _ptr(ws), wsb, _stream(stream)))
    return out, Z


def mlp_block_backward(X, W1, W2, dY, *, b1=None, Z=None, R_batch: int = 1, R_model: int = 1,
                       act: str = "gelu", bias_grads: bool = False, out=None, workspace=None, stream=None):
    """Gradients of mlp_block w.r.t. X, W1, W2 (and b1, b2 with bias_grads).
    Returns dX [T, D], dW1 [D, F], dW2 [F, D] (fp32, the weights' layout) and,
    with bias_grads, db1 [F] and db2 [D].  ``Z``: the pre-activation kept by
    mlp_block_train (else recomputed); ``out``: a tuple of the result tensors
    to write into."""
    import torch
    T, D, F = _mlp_shapes(X, W1, W2, b1, None)
    _req(dY, "dY", (T, D), _bf16())
    _opt(Z, "Z", (T, F), _bf16())
    a = ACT_GELU if act == "gelu" else ACT_NONE
    shapes = [(T, D), (D, F), (F, D)] + ([(F,), (D,)] if bias_grads else [])
    if out is not None:
        if len(out) != len(shapes):
            _bad("PARTIR_E_SHAPE", f"out must hold {len(shapes)} tensors")
        for u, sh, nm in zip(out, shapes, ("dX", "dW1", "dW2", "db1", "db2")):
            _req(u, nm, sh, torch.float32)
    dev = _gpu_all(X=X, W1=W1, W2=W2, b1=b1, dY=dY, Z=Z, out=out)
    fresh = out is None
    if fresh:
        out = tuple(torch.empty(sh, dtype=torch.float32, device=dev) for sh in shapes)
    dX, dW1, dW2 = out[:3]
    db1, db2 = out[3:5] if bias_grads else (None, None)
    nbytes = lib().partir_mlp_block_backward_workspace(T, D, F, a, int(bias_grads), R_batch, R_model)
    ws, wsb = _workspace(nbytes, dev, workspace)
    _on_stream(stream, ws if workspace is None else None, *(out if fresh else ()))
    _check(lib().partir_mlp_block_backward(_ptr(X), _ptr(W1), _ptr(b1), _ptr(W2), _ptr(dY), _ptr(Z), _ptr(dX),
                                           _ptr(dW1), _ptr(db1), _ptr(dW2), _ptr(db2), T, D, F, a, R_batch,
                                           R_model, _ptr(ws), wsb, _stream(stream)))
    return (dX, dW1, dW2, db1, db2) if bias_grads else (dX, dW1, dW2)


def _ptr_array(ts):
    """Host array of the tensors' device pointers (None for an absent list)."""
    if ts is None:
        return None
    arr = (ctypes.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = None if t is None else t.data_ptr()
    return arr


def _parts(ts, name, n, shape, dtype):
    if ts is None or len(ts) != n:
        _bad("PARTIR_E_SHAPE", f"{name} must be a list of {n} device-local arrays")
    for i, t in enumerate(ts):
        _req(t, f"{name}[{i}]", shape, dtype)


def mlp_block_sharded(X_parts, W1t_parts, W2t_parts, *, R_batch: int, R_model: int, b1=None, b2=None,
                      act: str = "gelu", out_dtype=None, out_parts=None, workspace=None, stream=None):
    """The MLP block on device-local arrays (BP + MP + Z3, activations sharded
    over the model axis).  Part p = b * R_model + m of the mesh {B, M}:
    X_parts[p] [T/(R_batch R_model), D]; W1t_parts[p] = W1^T[F/R_model rows m,
    D/R_batch cols b]; W2t_parts[p] = W2^T[D/R_batch rows b, F/R_model cols m]
    (the transposed blocks: device-local arrays are read K-contiguous).
    Returns the list of Y parts (token rows p of Y)."""
    import torch
    nd = R_batch * R_model
    if not X_parts or not W1t_parts or len(X_parts) != nd or len(W1t_parts) != nd:
        _bad("PARTIR_E_SHAPE", f"{nd} X and W1t parts expected")
    rows, D = X_parts[0].shape
    T = rows * nd
    F = W1t_parts[0].shape[0] * R_model
    bf = _bf16()
    _parts(X_parts, "X_parts", nd, (rows, D), bf)
    _parts(W1t_parts, "W1t_parts", nd, (F // R_model, D // R_batch), bf)
    _parts(W2t_parts, "W2t_parts", nd, (D // R_batch, F // R_model), bf)
    _opt(b1, "b1", (F,), _f32())
    _opt(b2, "b2", (D,), _f32())
    od = _out_dtype(out_dtype)
    if out_parts is not None:
        _parts(out_parts, "out_parts", nd, (rows, D), _tdt(od))
    dev = _gpu_all(X_parts=X_parts, W1t_parts=W1t_parts, W2t_parts=W2t_parts, b1=b1, b2=b2, out_parts=out_parts)
    fresh = out_parts is None
    if fresh:
        out_parts = [torch.empty((rows, D), dtype=_tdt(od), device=dev) for _ in range(nd)]
    ws, wsb = _workspace(lib().partir_mlp_block_sharded_workspace(T, D, F, R_batch, R_model), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, *(out_parts if fresh else ()))
    xs, w1s, w2s, ys = (_ptr_array(v) for v in (X_parts, W1t_parts, W2t_parts, out_parts))
    _check(lib().partir_mlp_block_sharded(xs, w1s, _ptr(b1), w2s, _ptr(b2), ys, T, D, F, od,
                                          ACT_GELU if act == "gelu" else ACT_NONE, R_batch, R_model,
                                          _ptr(ws), wsb, _stream(stream)))
    return out_parts


def z3_device_arrays(X, W1, W2, R_batch: int, R_model: int):
    """Copies whole operands into the device-local arrays mlp_block_sharded
    takes (each part its own allocation): X by token blocks p = b * R_model +
    m; the transposed weight blocks W1^T (rows m, cols b) and W2^T (rows b,
    cols m).  W1 [D, F], W2 [F, D] as mlp_block takes them."""
    nd = R_batch * R_model
    T, D = X.shape
    F = W1.shape[1]
    tr, dr, fr = T // nd, D // R_batch, F // R_model
    W1t, W2t = W1.t(), W2.t()
    xs = [X[p * tr:(p + 1) * tr].clone() for p in range(nd)]
    w1 = [W1t[m * fr:(m + 1) * fr, b * dr:(b + 1) * dr].contiguous() for b in range(R_batch) for m in range(R_model)]
    w2 = [W2t[b * dr:(b + 1) * dr, m * fr:(m + 1) * fr].contiguous() for b in range(R_batch) for m in range(R_model)]
    return xs, w1, w2


def z3_decoder_arrays(x, W, R_batch: int, R_model: int):
    """Device-local arrays of a decoder layer (each its own allocation): x
    (fp32 [T, D]) by token blocks; W = {name: weight [fan_in, fan_out]} as
    decoder_layer takes them, stored per part transposed: W^T of Wq, Wk, Wv,
    W1 split as (rows block m, cols block b) and of Wo, W2 as (rows block b,
    cols block m), part p = b * R_model + m.  Returns (x_parts, {name: parts})."""
    nd = R_batch * R_model
    T = x.shape[0]
    xs = [x[p * (T // nd):(p + 1) * (T // nd)].clone() for p in range(nd)]
    parts = {}
    for k, w in W.items():
        wt = w.t()
        rows, cols = wt.shape
        col_par = k in ("Wq", "Wk", "Wv", "W1")
        rr, cc = (rows // R_model, cols // R_batch) if col_par else (rows // R_batch, cols // R_model)
        out = []
        for b in range(R_batch):
            for m in range(R_model):
                i, j = (m, b) if col_par else (b, m)
                out.append(wt[i * rr:(i + 1) * rr, j * cc:(j + 1) * cc].contiguous())
        parts[k] = out
    return xs, parts


def decoder_layer_sharded(x_parts, g1, g2, W_parts, *, B: int, S: int, n_heads: int, d_head: int = 128,
                          R_batch: int = 1, R_model: int = 1, eps: float = 1e-6, workspace=None, stream=None):
    """One decoder layer on device-local arrays, x_parts updated in place
    (see z3_decoder_arrays for the layout)."""
    nd = R_batch * R_model
    if not x_parts or len(x_parts) != nd:
        _bad("PARTIR_E_SHAPE", f"{nd} x parts expected")
    D = x_parts[0].shape[1]
    F = W_parts["W1"][0].shape[0] * R_model
    bf = _bf16()
    _parts(x_parts, "x_parts", nd, (B * S // nd, D), _f32())
    _req(g1, "g1", (D,), _f32())
    _opt(g2, "g2", (D,), _f32())
    for k in ("Wq", "Wk", "Wv"):
        _parts(W_parts[k], k, nd, (D // R_model, D // R_batch), bf)
    _parts(W_parts["Wo"], "Wo", nd, (D // R_batch, D // R_model), bf)
    _parts(W_parts["W1"], "W1", nd, (F // R_model, D // R_batch), bf)
    _parts(W_parts["W2"], "W2", nd, (D // R_batch, F // R_model), bf)
    dev = _gpu_all(x_parts=x_parts, g1=g1, g2=g2, **{k: W_parts[k] for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2")})
    nbytes = lib().partir_decoder_layer_sharded_workspace(B, S, D, n_heads, d_head, F, R_batch, R_model)
    ws, wsb = _workspace(nbytes, dev, workspace)
    _on_stream(stream, ws if workspace is None else None)
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


def _attn_shapes(X, Ws, B, S):
    bf = _bf16()
    if X.dim() != 2:
        _bad("PARTIR_E_SHAPE", "X must be 2-D")
    T, D = X.shape
    if T != B * S:
        _bad("PARTIR_E_SHAPE", f"X has {T} rows, B*S = {B * S}")
    _req(X, "X", (T, D), bf)
    for nm, w in zip(("Wq", "Wk", "Wv", "Wo"), Ws):
        _req(w, nm, (D, D), bf)
    return T, D


def attn_block(X, Wq, Wk, Wv, Wo, *, B: int, S: int, n_heads: int, d_head: int = 128,
               causal: bool = True, scale: float = 0.0, R_batch: int = 1, R_model: int = 1,
               out_dtype=None, out=None, workspace=None, stream=None):
    """Y = loop b [#tile<0>] loop m [#sum] (heads #tile attention) . Wo[m]:
    X [B*S, D] bf16; Wq, Wk, Wv, Wo [D, D] bf16 ([fan_in, fan_out])."""
    import torch
    T, D = _attn_shapes(X, (Wq, Wk, Wv, Wo), B, S)
    od = _out_dtype(out_dtype)
    _opt(out, "out", (T, D), _tdt(od))
    dev = _gpu_all(X=X, Wq=Wq, Wk=Wk, Wv=Wv, Wo=Wo, out=out)
    fresh = out is None
    if fresh:
        out = torch.empty((T, D), dtype=_tdt(od), device=dev)
    ws, wsb = _workspace(attn_block_workspace(B, S, D, n_heads, d_head, R_batch, R_model), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh else None)
    _check(lib().partir_attn_block(_ptr(X), _ptr(Wq), _ptr(Wk), _ptr(Wv), _ptr(Wo), _ptr(out),
                                   B, S, D, n_heads, d_head, int(causal), float(scale), BF16, od,
                                   R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return out


def _qkv_shapes(ts, names, B, S, n_heads, d_head):
    T, D = B * S, n_heads * d_head
    for t, nm in zip(ts, names):
        _req(t, nm, (T, D), _bf16())
    return T, D


def attention(Q, K, V, *, B: int, S: int, n_heads: int, d_head: int = 128, causal: bool = True,
              scale: float = 0.0, R_kv: int = 1, out=None, workspace=None, stream=None):
    """O = softmax attention per (sequence, head), the key axis a loop of R_kv
    shards reduced with the (max, sum, output) combiner.  Q, K, V, O: [B*S, n_heads*d_head] bf16."""
    import torch
    T, D = _qkv_shapes((Q, K, V), ("Q", "K", "V"), B, S, n_heads, d_head)
    _opt(out, "out", (T, D), _bf16())
    dev = _gpu_all(Q=Q, K=K, V=V, out=out)
    fresh = out is None
    if fresh:
        out = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
    nbytes = lib().partir_attention_workspace(B, S, n_heads, d_head, R_kv)
    ws, wsb = _workspace(nbytes, dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh else None)
    _check(lib().partir_attention(_ptr(Q), _ptr(K), _ptr(V), _ptr(out), B, S, n_heads, d_head, int(causal),
                                  float(scale), R_kv, _ptr(ws), wsb, _stream(stream)))
    return out


def attention_train(Q, K, V, *, B: int, S: int, n_heads: int, d_head: int = 128, causal: bool = True,
                    scale: float = 0.0, R_kv: int = 1, out=None, lse=None, workspace=None, stream=None):
    """attention that also returns the per-row base-2 log-sum-exp [B*S, n_heads]
    fp32 for attention_backward.  Returns (O, lse)."""
    import torch
    T, D = _qkv_shapes((Q, K, V), ("Q", "K", "V"), B, S, n_heads, d_head)
    _opt(out, "out", (T, D), _bf16())
    _opt(lse, "lse", (T, n_heads), _f32())
    dev = _gpu_all(Q=Q, K=K, V=V, out=out, lse=lse)
    fresh_o, fresh_l = out is None, lse is None
    if fresh_o:
        out = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
    if fresh_l:
        lse = torch.empty((T, n_heads), dtype=torch.float32, device=dev)
    ws, wsb = _workspace(lib().partir_attention_workspace(B, S, n_heads, d_head, R_kv), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh_o else None, lse if fresh_l else None)
    _check(lib().partir_attention_train(_ptr(Q), _ptr(K), _ptr(V), _ptr(out), _ptr(lse), B, S, n_heads, d_head,
                                        int(causal), scale, R_kv, _ptr(ws), wsb, _stream(stream)))
    return out, lse


def attention_backward(Q, K, V, O, dO, lse, *, B: int, S: int, n_heads: int, d_head: int = 128,
                       causal: bool = True, scale: float = 0.0, out=None, workspace=None, stream=None):
    """Gradients (dQ, dK, dV) of attention for the output cotangent dO (bf16,
    the layout of Q, K, V), from the forward's O and lse."""
    import torch
    T, D = _qkv_shapes((Q, K, V, O, dO), ("Q", "K", "V", "O", "dO"), B, S, n_heads, d_head)
    _req(lse, "lse", (T, n_heads), _f32())
    if out is not None:
        if len(out) != 3:
            _bad("PARTIR_E_SHAPE", "out must hold (dQ, dK, dV)")
        _qkv_shapes(out, ("dQ", "dK", "dV"), B, S, n_heads, d_head)
    dev = _gpu_all(Q=Q, K=K, V=V, O=O, dO=dO, lse=lse, out=out)
    fresh = out is None
    if fresh:
        out = tuple(torch.empty((T, D), dtype=torch.bfloat16, device=dev) for _ in range(3))
    ws, wsb = _workspace(lib().partir_attention_backward_workspace(B, S, n_heads, d_head), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, *(out if fresh else ()))
    _check(lib().partir_attention_backward(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(lse), _ptr(out[0]),
                                           _ptr(out[1]), _ptr(out[2]), B, S, n_heads, d_head, int(causal), scale,
                                           _ptr(ws), wsb, _stream(stream)))
    return out


def attn_block_train(X, Wq, Wk, Wv, Wo, *, B: int, S: int, n_heads: int, d_head: int = 128,
                     causal: bool = True, scale: float = 0.0, R_batch: int = 1, R_model: int = 1, out=None,
                     saved=None, workspace=None, stream=None):
    """attn_block that also keeps Q, K, V, A and lse in `saved` (a uint8
    tensor) for attn_block_backward.  Returns (Y, saved)."""
    import torch
    T, D = _attn_shapes(X, (Wq, Wk, Wv, Wo), B, S)
    need = lib().partir_attn_block_saved_bytes(B, S, D, n_heads)
    if out is not None:
        if out.dtype not in (torch.float32, torch.bfloat16):
            _bad("PARTIR_E_DTYPE", "out must be float32 or bfloat16")
        _req(out, "out", (T, D), out.dtype)
    if saved is not None and (saved.dtype != torch.uint8 or saved.numel() < need or not saved.is_contiguous()):
        _bad("PARTIR_E_WORKSPACE", f"saved must be a contiguous uint8 buffer of >= {need} bytes")
    dev = _gpu_all(X=X, Wq=Wq, Wk=Wk, Wv=Wv, Wo=Wo, out=out, saved=saved)
    fresh_y, fresh_s = out is None, saved is None
    if fresh_y:
        out = torch.empty((T, D), dtype=torch.float32, device=dev)
    if fresh_s:
        saved = torch.empty(max(1, need), dtype=torch.uint8, device=dev)
    ws, wsb = _workspace(attn_block_workspace(B, S, D, n_heads, d_head, R_batch, R_model), dev, workspace)
    _on_stream(stream, ws if workspace is None else None, out if fresh_y else None, saved if fresh_s else None)
    _check(lib().partir_attn_block_train(_ptr(X), _ptr(Wq), _ptr(Wk), _ptr(Wv), _ptr(Wo), _ptr(out),
                                         _ptr(saved), B, S, D, n_heads, d_head, int(causal), scale, BF16,
                                         _dt(out), R_batch, R_model, _ptr(ws), wsb, _stream(stream)))
    return out, saved


def attn_block_backward(X, Wq, Wk, Wv, Wo, saved, dY, *, B: int, S: int, n_heads: int,
                        d_head: int = 128, causal: bool = True, scale: float = 0.0, R_batch: int = 1,
                        R_model: int = 1, out=None, workspace=None, stream=None):
    """Gradients (dX, dWq, dWk, dWv, dWo), fp32, the weights' [fan_in, fan_out] layout."""
    import torch
    T, D = _attn_shapes(X, (Wq, Wk, Wv, Wo), B, S)
    need = lib().partir_attn_block_saved_bytes(B, S, D, n_heads)
    if saved.dtype != torch.uint8 or saved.numel() < need:
        _bad("PARTIR_E_SHAPE", f"saved must be the >= {need}-byte uint8 buffer of attn_block_train")
    _req(dY, "dY", (T, D), _bf16())
    shapes = [(T, D)] + [(D, D)] * 4
    if out is not None:
        if len(out) != 5:
            _bad("PARTIR_E_SHAPE", "out must hold 5 tensors")
        for u, sh, nm in zip(out, shapes, ("dX", "dWq", "dWk", "dWv", "dWo")):
            _req(u, nm, sh, torch.float32)
    dev = _gpu_all(X=X, Wq=Wq, Wk=Wk, Wv=Wv, Wo=Wo, saved=saved, dY=dY, out=out)
    fresh = out is None
    if fresh:
        out = tuple(torch.empty(sh, dtype=torch.float32, device=dev) for sh in shapes)
    ws, wsb = _workspace(lib().partir_attn_block_backward_workspace(B, S, D, n_heads, d_head, R_batch, R_model),
                         dev, workspace)
    _on_stream(stream, ws if workspace is None else None, *(out if fresh else ()))
    _check(lib().partir_attn_block_backward(_ptr(X), _ptr(Wq), _ptr(Wk), _ptr(Wv), _ptr(Wo), _ptr(saved),
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


def decoder_layer(x, g1, g2, Wq, Wk, Wv, Wo, W1, W2, *, B: int, S: int, n_heads: int,
                  d_head: int = 128, eps: float = 1e-6, R_batch: int = 1, R_model: int = 1,
                  workspace=None, stream=None):
    """In place on the fp32 residual stream x [B*S, D].  Wq..Wo [D, D],
    W1 [D, F], W2 [F, D], bf16 ([fan_in, fan_out]); g1, g2 [D] fp32."""
    if x.dim() != 2 or W1.dim() != 2:
        _bad("PARTIR_E_SHAPE", "x and W1 must be 2-D")
    T, D = x.shape
    F = W1.shape[1]
    if T != B * S:
        _bad("PARTIR_E_SHAPE", f"x has {T} rows, B*S = {B * S}")
    bf = _bf16()
    _req(x, "x", (T, D), _f32())
    _req(g1, "g1", (D,), _f32())
    _opt(g2, "g2", (D,), _f32())
    for nm, w in zip(("Wq", "Wk", "Wv", "Wo"), (Wq, Wk, Wv, Wo)):
        _req(w, nm, (D, D), bf)
    _req(W1, "W1", (D, F), bf)
    _req(W2, "W2", (F, D), bf)
    dev = _gpu_all(x=x, g1=g1, g2=g2, Wq=Wq, Wk=Wk, Wv=Wv, Wo=Wo, W1=W1, W2=W2)
    ws, wsb = _workspace(decoder_layer_workspace(B, S, D, n_heads, d_head, F, R_batch, R_model), dev, workspace)
    _on_stream(stream, ws if workspace is None else None)
    _check(lib().partir_decoder_layer(_ptr(x), _ptr(g1), _ptr(g2), float(eps), _ptr(Wq), _ptr(Wk), _ptr(Wv),
                                      _ptr(Wo), _ptr(W1), _ptr(W2), B, S, D, n_heads, d_head, F,
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

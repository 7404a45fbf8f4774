"""GPU test of partir_loop_matmul_noalloc (the entry point for callers that
cannot allocate): through the C ABI, its output equals partir_loop_matmul's
(same plan, same kernels, so bit for bit) and the oracle's within the
tolerance, on two calls in a row, the second with a smaller input, so the
second call runs on scratch the first one left behind."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import partir_oracle as O
from paper_2401_11202_amd import inputs as I
from paper_2401_11202_amd import partir as P
from tests.gpu_common import TOL_BF16, TOL_F32, host, say

pytestmark = pytest.mark.gpu


def call(fn_name, A, B, C, M, N, K, ab, c, R, impl, ws=None):
    L = P.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    args = [ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(B.data_ptr()), ctypes.c_void_p(C.data_ptr()),
            M, N, K, K, K, N, ab, c, P.B_NK, P.AXIS_NONE, P.AXIS_K, R, impl]
    if fn_name == "partir_loop_matmul":
        args += [ctypes.c_void_p(ws.data_ptr()) if ws is not None else None, 0 if ws is None else ws.numel()]
    st = getattr(L, fn_name)(*args, stream)
    assert st == 0, L.partir_last_error().decode()


# (M, N, K, R, ab dtype, out dtype, sum realisation): each #sum runs as
# split-K, so the scratch holds R fp32 partials [M, N]
CASES = [
    (512, 512, 8192, 8, P.BF16, P.F32, P.SUM_SPLITK),     # 8 MiB of partials
    (256, 384, 1024, 4, P.BF16, P.BF16, P.SUM_SPLITK),    # 1.5 MiB, smaller: the second call
    (256, 256, 512, 4, P.F32, P.F32, P.SUM_AUTO),         # the fp32 256x256x512 #sum, 1 MiB
]


@pytest.mark.parametrize("first,second", [(0, 1), (0, 2)])
def test_noalloc_equals_workspace_entry_point_on_two_calls(first, second):
    for i in (first, second):
        M, N, K, R, ab, c, impl = CASES[i]
        need = P.lib().partir_loop_matmul_workspace(M, N, K, ab, c, P.B_NK, P.AXIS_NONE, P.AXIS_K, R, impl)
        assert 0 < need <= 64 << 20
        kind = "bf16" if ab == P.BF16 else "f32"
        A = I.gaussian(151, 2 * i, (M, K), 1.0, kind)
        Bt = I.gaussian(151, 2 * i + 1, (N, K), K ** -0.5, kind)
        Ad, Bd = A.to_device(), Bt.to_device()
        odt = torch.bfloat16 if c == P.BF16 else torch.float32
        say(f"noalloc call {i}: {kind} {M}x{N}x{K} #sum K R={R} scratch {need} bytes")
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        C_ws = torch.full((M, N), float("nan"), dtype=odt, device="cuda")
        C_na = torch.full((M, N), float("nan"), dtype=odt, device="cuda")
        call("partir_loop_matmul", Ad, Bd, C_ws, M, N, K, ab, c, R, impl, ws)
        call("partir_loop_matmul_noalloc", Ad, Bd, C_na, M, N, K, ab, c, R, impl)
        torch.cuda.synchronize()
        assert torch.equal(C_ws, C_na)
        ref = O.loop_matmul(A.f64(), Bt.f64().T, O.AXIS_NONE, O.AXIS_K, R)
        err = O.normalised_error(host(C_na), ref, O.abs_product(A.f64(), Bt.f64().T))
        say(f"    equal to partir_loop_matmul; max normalised error vs the oracle {err:.3e}")
        assert err <= (TOL_BF16 if ab == P.BF16 else TOL_F32)
        del ws


def test_noalloc_refuses_more_scratch_than_it_holds():
    A = torch.zeros((2048, 8192), dtype=torch.bfloat16, device="cuda")
    C = torch.zeros((2048, 2048), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(P.PartirError, match="bytes of scratch"):
        P.loop_matmul_noalloc(A, A[:2048], sum="K", R=8, b_layout="nk", out=C)

"""Host-side tests of the C ABI: exports, validation, plans (no GPU needed).

No call here passes validation without PARTIR_FAIL_LAUNCH=1, which makes the
library return PARTIR_E_HIP before touching the GPU; pointers are dummies that
are never dereferenced.
"""
import ctypes
import os
import re

import pytest

from paper_2401_11202_amd import partir as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DUMMY = ctypes.c_void_p(0x10000)      # 16-byte aligned, never dereferenced
DUMMY_ODD = ctypes.c_void_p(0x10004)  # misaligned
NULL = None


@pytest.fixture(autouse=True)
def _never_launch(monkeypatch):
    """Should a case pass validation by mistake, it still stops before the GPU."""
    monkeypatch.setenv("PARTIR_FAIL_LAUNCH", "1")


def declared_functions():
    text = open(os.path.join(ROOT, "include", "partir.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(partir_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = P.lib()
    names = declared_functions()
    assert len(names) >= 19
    for n in names:
        assert hasattr(L, n), n
    assert set(P.EXPORTS) == set(names)


def test_status_strings():
    L = P.lib()
    for code, name in P.STATUS.items():
        assert L.partir_status_string(code).decode() == name
    assert P.lib().partir_version().decode().startswith("libpartir")


# ---------------------------------------------------------------------------
# loop_matmul validation
# ---------------------------------------------------------------------------
def mm(M=256, N=256, K=512, lda=None, ldb=None, ldc=None, ab=P.F32, c=P.F32, bl=P.B_KN,
       tile=P.AXIS_NONE, summ=P.AXIS_K, R=4, impl=P.SUM_AUTO, A=DUMMY, B=DUMMY, C=DUMMY,
       ws=DUMMY, ws_bytes=1 << 30):
    lda = K if lda is None else lda
    ldb = (N if bl == P.B_KN else K) if ldb is None else ldb
    ldc = N if ldc is None else ldc
    return P.lib().partir_loop_matmul(A, B, C, M, N, K, lda, ldb, ldc, ab, c, bl, tile, summ, R, impl,
                                      ws, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(A=NULL), "PARTIR_E_NULL"),
    (dict(C=NULL), "PARTIR_E_NULL"),
    (dict(M=-1), "PARTIR_E_SHAPE"),
    (dict(K=-4), "PARTIR_E_SHAPE"),
    (dict(M=256, N=256, K=0, A=NULL, lda=0), "PARTIR_E_HIP"),       # empty contraction: valid, reaches launch
    (dict(M=0, N=256, K=512, C=NULL), "PARTIR_E_HIP"),              # empty output: valid (no launch needed)
    (dict(R=0), "PARTIR_E_UNSUPPORTED"),
    (dict(R=3), "PARTIR_E_DIVISIBILITY"),                          # 3 does not divide K = 512
    (dict(tile=P.AXIS_M, summ=P.AXIS_NONE, M=250, R=4), "PARTIR_E_DIVISIBILITY"),
    (dict(tile=P.AXIS_N, summ=P.AXIS_NONE, N=100, R=8), "PARTIR_E_DIVISIBILITY"),
    (dict(tile=P.AXIS_K, summ=P.AXIS_NONE), "PARTIR_E_AXIS"),       # a contracted dim cannot be tiled
    (dict(tile=P.AXIS_M, summ=P.AXIS_M), "PARTIR_E_AXIS"),          # one axis tiled and summed
    (dict(summ=P.AXIS_N), "PARTIR_E_AXIS"),
    (dict(tile=7), "PARTIR_E_AXIS"),
    (dict(ab=5), "PARTIR_E_DTYPE"),
    (dict(ab=P.F32, c=P.BF16), "PARTIR_E_DTYPE"),
    (dict(lda=500), "PARTIR_E_LAYOUT"),                              # lda < K
    (dict(ldc=258), "PARTIR_E_LAYOUT"),                              # rows not 16-byte aligned
    (dict(A=DUMMY_ODD), "PARTIR_E_LAYOUT"),
    (dict(K=510, R=2, lda=512), "PARTIR_E_LAYOUT"),                  # K not a whole 16-byte run
    (dict(ab=P.BF16, c=P.BF16, bl=P.B_NK, K=520, R=4, lda=520), "PARTIR_E_LAYOUT"),  # K/R = 130
    (dict(ws_bytes=16), "PARTIR_E_WORKSPACE"),
    (dict(ws=NULL), "PARTIR_E_NULL"),
    (dict(impl=9), "PARTIR_E_UNSUPPORTED"),
    # bf16 B as [K, N]: its rows are read in 16-byte chunks
    (dict(ab=P.BF16, c=P.BF16, bl=P.B_KN, N=260, ldc=264, ldb=264, summ=P.AXIS_NONE, R=1), "PARTIR_E_LAYOUT"),
    (dict(ab=P.BF16, c=P.BF16, bl=P.B_KN, N=264, tile=P.AXIS_N, summ=P.AXIS_NONE, R=2), "PARTIR_E_LAYOUT"),
    (dict(ab=P.BF16, c=P.BF16, bl=P.B_KN, N=264, summ=P.AXIS_NONE, R=1, ws=NULL, ws_bytes=0), "PARTIR_E_HIP"),
])
def test_loop_matmul_validation(kwargs, status):
    st = mm(**kwargs)
    assert P.STATUS[st] == status, P.lib().partir_last_error().decode()
    assert P.lib().partir_last_error().decode().startswith(status)


@pytest.mark.parametrize("kwargs,status", [
    # a bf16 operand addresses a 64-row block through a 32-bit byte range: at
    # lda = 2^25 that range (64 * lda * 2 = 2^32) wraps, so it is refused
    (dict(M=64, N=8, K=2 ** 25), "PARTIR_E_SHAPE"),
    (dict(M=64, N=8, K=2 ** 26), "PARTIR_E_SHAPE"),
    (dict(M=64, N=8, K=2 ** 24 + 8), "PARTIR_E_SHAPE"),
    (dict(M=64, N=8, K=2 ** 24), "PARTIR_E_HIP"),                    # the largest addressable K
    (dict(M=64, N=8, K=64, lda=2 ** 24 + 8), "PARTIR_E_SHAPE"),      # a long leading dim alone
    (dict(M=64, N=2 ** 24 + 8, K=64, bl=P.B_KN, ldc=2 ** 24 + 8), "PARTIR_E_SHAPE"),   # B [K, N] rows
    (dict(M=2 ** 24 + 8, N=8, K=64, bl=P.B_NK, ldb=2 ** 24 + 8), "PARTIR_E_SHAPE"),    # B^T rows
    # 2^24 x 2^8 output tiles of 64 x 64: more than a grid indexes
    (dict(M=2 ** 30, N=2 ** 14, K=64), "PARTIR_E_SHAPE"),
    (dict(M=2 ** 30, N=2 ** 12, K=64), "PARTIR_E_HIP"),
])
def test_loop_matmul_bf16_addressing_limits(kwargs, status):
    args = dict(ab=P.BF16, c=P.BF16, bl=P.B_NK, summ=P.AXIS_NONE, R=1, ws=NULL, ws_bytes=0)
    args.update(kwargs)
    st = mm(**args)
    assert P.STATUS[st] == status, P.lib().partir_last_error().decode()
    if status == "PARTIR_E_SHAPE" and not {"lda", "ldb", "ldc"} & set(kwargs):
        # the size query (leading dims = row lengths) refuses the same shapes
        assert P.lib().partir_loop_matmul_workspace(args["M"], args["N"], args["K"], P.BF16, P.BF16, args["bl"],
                                                    args.get("tile", P.AXIS_NONE), P.AXIS_NONE, args["R"],
                                                    P.SUM_AUTO) == ctypes.c_size_t(-1).value


def mm_noalloc(M=256, N=256, K=512, ab=P.F32, c=P.F32, bl=P.B_KN, tile=P.AXIS_NONE, summ=P.AXIS_K, R=4,
               impl=P.SUM_AUTO, A=DUMMY, B=DUMMY, C=DUMMY):
    lda, ldb, ldc = K, (N if bl == P.B_KN else K), N
    return P.lib().partir_loop_matmul_noalloc(A, B, C, M, N, K, lda, ldb, ldc, ab, c, bl, tile, summ, R, impl, None)


@pytest.mark.parametrize("kwargs,status", [
    # split-K partials of 8 x [2048, 2048] fp32 = 128 MiB: beyond the 64 MiB scratch
    (dict(M=2048, N=2048, K=8192, ab=P.BF16, c=P.BF16, bl=P.B_NK, R=8), "PARTIR_E_WORKSPACE"),
    (dict(M=4096, N=4096, K=4096, ab=P.BF16, c=P.F32, bl=P.B_NK, R=2, impl=P.SUM_SPLITK), "PARTIR_E_WORKSPACE"),
    # invalid calls report partir_loop_matmul's own status
    (dict(R=3), "PARTIR_E_DIVISIBILITY"),
    (dict(A=NULL), "PARTIR_E_NULL"),
    (dict(ab=P.F32, c=P.BF16), "PARTIR_E_DTYPE"),
    # no scratch needed (no #sum): straight to the launch, which is forced to fail here
    (dict(summ=P.AXIS_NONE, R=1), "PARTIR_E_HIP"),
])
def test_loop_matmul_noalloc_validation(kwargs, status):
    st = mm_noalloc(**kwargs)
    assert P.STATUS[st] == status, P.lib().partir_last_error().decode()
    if status == "PARTIR_E_WORKSPACE":
        assert "bytes of scratch" in P.lib().partir_last_error().decode()


def test_valid_call_reaches_launch(monkeypatch):
    monkeypatch.setenv("PARTIR_FAIL_LAUNCH", "1")
    assert P.STATUS[mm()] == "PARTIR_E_HIP"
    assert "PARTIR_FAIL_LAUNCH" in P.lib().partir_last_error().decode()
    assert P.STATUS[mm(ab=P.BF16, c=P.BF16, bl=P.B_NK, tile=P.AXIS_N, summ=P.AXIS_NONE, R=8)] == "PARTIR_E_HIP"


def test_error_message_is_thread_local():
    import threading
    mm(R=3)
    msg = {}

    def other():
        mm(M=-1)
        msg["t"] = P.lib().partir_last_error().decode()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert msg["t"].startswith("PARTIR_E_SHAPE")
    assert P.lib().partir_last_error().decode().startswith("PARTIR_E_DIVISIBILITY")


# ---------------------------------------------------------------------------
# block validation
# ---------------------------------------------------------------------------
def mlp(T=512, D=256, F=1024, ind=P.BF16, out=P.F32, act=P.ACT_GELU, Rb=1, Rm=8, X=DUMMY, Y=DUMMY,
        ws=DUMMY, ws_bytes=1 << 30):
    return P.lib().partir_mlp_block(X, DUMMY, None, DUMMY, None, Y, T, D, F, ind, out, act, Rb, Rm,
                                    ws, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(X=NULL), "PARTIR_E_NULL"),
    (dict(T=-1), "PARTIR_E_SHAPE"),
    (dict(Rm=0), "PARTIR_E_UNSUPPORTED"),
    (dict(Rm=3), "PARTIR_E_DIVISIBILITY"),
    (dict(Rb=3), "PARTIR_E_DIVISIBILITY"),
    (dict(ind=P.F32), "PARTIR_E_DTYPE"),
    (dict(out=4), "PARTIR_E_DTYPE"),
    (dict(act=5), "PARTIR_E_UNSUPPORTED"),
    (dict(D=252), "PARTIR_E_LAYOUT"),
    (dict(F=1024 + 32, Rm=8), "PARTIR_E_LAYOUT"),   # F/R = 132 is not a multiple of 8
    (dict(ws_bytes=100), "PARTIR_E_WORKSPACE"),
])
def test_mlp_validation(kwargs, status):
    assert P.STATUS[mlp(**kwargs)] == status, P.lib().partir_last_error().decode()


def attn(B=2, S=256, D=1024, H=8, dh=128, Rb=1, Rm=8, out=P.F32, ws_bytes=1 << 30, X=DUMMY):
    return P.lib().partir_attn_block(X, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, B, S, D, H, dh, 1, 0.0,
                                     P.BF16, out, Rb, Rm, DUMMY, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(X=NULL), "PARTIR_E_NULL"),
    (dict(H=6), "PARTIR_E_SHAPE"),               # 6 * 128 != 1024
    (dict(D=512, H=8, dh=64), "PARTIR_E_SHAPE"),  # d_head must be 128
    (dict(S=200), "PARTIR_E_SHAPE"),
    (dict(S=-128), "PARTIR_E_SHAPE"),
    (dict(Rm=3), "PARTIR_E_DIVISIBILITY"),
    (dict(Rb=4, B=2), "PARTIR_E_DIVISIBILITY"),   # batch shards hold whole sequences
    (dict(ws_bytes=0), "PARTIR_E_WORKSPACE"),
])
def test_attn_validation(kwargs, status):
    assert P.STATUS[attn(**kwargs)] == status, P.lib().partir_last_error().decode()


def test_decoder_validation():
    L = P.lib()
    st = L.partir_decoder_layer(DUMMY, DUMMY, DUMMY, 1e-6, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                2, 256, 1024, 8, 128, 1002, 2, 4, DUMMY, 1 << 34, None)
    assert P.STATUS[st] == "PARTIR_E_DIVISIBILITY"   # 4 does not divide F = 1002
    st = L.partir_decoder_layer(DUMMY, DUMMY, DUMMY, 1e-6, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                2, 256, 1024, 8, 128, 1000, 2, 4, DUMMY, 1 << 34, None)
    assert P.STATUS[st] == "PARTIR_E_LAYOUT"         # F/R = 250 is not a whole 16-byte run
    st = L.partir_decoder_layer(DUMMY, DUMMY, DUMMY, -1.0, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                2, 256, 1024, 8, 128, 1728, 2, 4, DUMMY, 1 << 34, None)
    assert P.STATUS[st] == "PARTIR_E_SHAPE"
    st = L.partir_decoder_layer(None, DUMMY, DUMMY, 1e-6, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                2, 256, 1024, 8, 128, 1728, 2, 4, DUMMY, 1 << 34, None)
    assert P.STATUS[st] == "PARTIR_E_NULL"


def test_blocks_reach_launch(monkeypatch):
    monkeypatch.setenv("PARTIR_FAIL_LAUNCH", "1")
    assert P.STATUS[mlp()] == "PARTIR_E_HIP"
    assert P.STATUS[attn()] == "PARTIR_E_HIP"
    st = P.lib().partir_decoder_layer(DUMMY, DUMMY, DUMMY, 1e-6, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                      2, 256, 1024, 8, 128, 1728, 2, 4, DUMMY, 1 << 34, None)
    assert P.STATUS[st] == "PARTIR_E_HIP"


# ---------------------------------------------------------------------------
# plans: the in-device stand-ins of the lowering's collectives
# ---------------------------------------------------------------------------
def test_megatron_mlp_has_exactly_one_sum_per_block():
    """Megatron: one all_reduce per MLP block in the forward pass (Sec. 2.3;
    Sec. 6.1 lowered program) -> exactly one in-device #sum."""
    p = P.plan_mlp_block(8192, 4096, 16384, R_batch=1, R_model=8)
    assert p["n_sum_loops"] == 1 and p["n_virtual_shards"] == 8 and p["n_launches"] == 2
    assert p["n_sum_splitk"] == 0          # 512 output tiles: fused accumulation, no partials
    assert p["workspace_bytes"] == 8192 * 16384 * 2
    assert p["flops"] == 4.0 * 8192 * 4096 * 16384


def test_batch_only_mlp_has_no_reduction_across_shards():
    p = P.plan_mlp_block(16384, 8192, 32768, R_batch=4, R_model=1)
    assert p["n_sum_loops"] == 0 and p["n_virtual_shards"] == 4


def test_two_axis_nest_plans():
    p = P.plan_mlp_block(16384, 8192, 32768, R_batch=4, R_model=8)
    assert p["n_virtual_shards"] == 32 and p["n_sum_loops"] == 1 and p["n_tile_loops"] == 2
    assert "#tile M x4" in p["text"] and "#sum K x8" in p["text"]


def test_attention_and_decoder_sums():
    a = P.plan_attn_block(4, 2048, 4096, 32, 128, 1, 8)
    assert a["n_sum_loops"] == 1 and a["n_launches"] == 3 and a["n_virtual_shards"] == 8
    d = P.plan_decoder_layer(4, 2048, 5120, 40, 128, 13824, 2, 4)
    # two #sum loops per layer (attention out-projection and FFN down): Megatron's 2 all_reduces;
    # 7 launches plus the fixups of the three GEMMs whose last wave is split (1920 and 640 tiles)
    assert d["n_sum_loops"] == 2 and d["n_virtual_shards"] == 8 and d["n_launches"] == 10
    assert d["text"].count(".fixup:") == 3 and d["text"].count("the last 128 tiles as 2 K parts") == 3


def test_small_output_uses_split_partials():
    p = P.plan_loop_matmul(256, 256, 512, ab=P.F32, c=P.F32, b_layout=P.B_KN, sum="K", R=4)
    assert p["n_sum_splitk"] == 1 and p["n_launches"] == 2 and p["workspace_bytes"] == 4 * 256 * 256 * 4
    f = P.plan_loop_matmul(256, 256, 512, ab=P.F32, c=P.F32, b_layout=P.B_KN, sum="K", R=4,
                           sum_impl=P.SUM_FUSED)
    assert f["n_sum_splitk"] == 0 and f["n_launches"] == 1 and f["workspace_bytes"] == 0


def test_workspace_queries_match_plans():
    L = P.lib()
    assert L.partir_mlp_block_workspace(8192, 4096, 16384, P.F32, 1, 8) == \
        P.plan_mlp_block(8192, 4096, 16384, R_model=8)["workspace_bytes"]
    assert L.partir_attn_block_workspace(4, 2048, 4096, 32, 128, 1, 8) == \
        P.plan_attn_block(4, 2048, 4096, 32, 128, 1, 8)["workspace_bytes"]
    assert L.partir_mlp_block_workspace(8192, 4096, 16383, P.F32, 1, 8) == ctypes.c_size_t(-1).value


def test_plan_text_names_every_shard_loop():
    p = P.plan_decoder_layer(4, 2048, 5120, 40, 128, 13824, 2, 4)
    t = p["text"]
    assert t.count("rmsnorm") == 2 and "attention" in t and t.count("fused in accumulator") == 2
    assert "#tile N x4 (cols 3456/shard)" in t


# ---------------------------------------------------------------------------
# empty operands: a zero-size dim is a legal TSlice (n_d = 0); #sum over an
# empty contraction is the empty sum
# ---------------------------------------------------------------------------
def test_empty_shapes_plan():
    e = P.plan_loop_matmul(0, 256, 512, ab=P.BF16, c=P.BF16, b_layout=P.B_NK, tile="M", R=4)
    assert e["n_launches"] == 0 and e["workspace_bytes"] == 0 and e["flops"] == 0
    z = P.plan_loop_matmul(256, 256, 0, ab=P.BF16, c=P.F32, b_layout=P.B_NK, sum="K", R=4)
    assert z["n_launches"] == 1 and z["n_sum_loops"] == 1 and z["workspace_bytes"] == 0
    assert "empty_sum" in z["text"]
    m = P.plan_mlp_block(512, 256, 0, R_model=8)        # every model shard is empty: Y = b2
    assert m["n_launches"] == 1 and m["workspace_bytes"] == 0
    assert P.plan_mlp_block(0, 256, 1024, R_model=8)["n_launches"] == 0
    assert P.plan_attn_block(0, 2048, 4096, 32, 128, 1, 8)["n_launches"] == 0
    d = P.plan_decoder_layer(2, 256, 1024, 8, 128, 0, 2, 4)   # FFN of width 0: attention half only
    assert d["n_sum_loops"] == 1 and "ffn" not in d["text"] and d["text"].count("rmsnorm") == 1
    assert P.plan_decoder_layer(0, 256, 1024, 8, 128, 1728, 2, 4)["n_launches"] == 0


def test_empty_calls_validate(monkeypatch):
    monkeypatch.setenv("PARTIR_FAIL_LAUNCH", "1")
    L = P.lib()
    # NULL operands are fine when they hold no elements
    st = L.partir_mlp_block(NULL, NULL, None, NULL, None, NULL, 0, 256, 1024, P.BF16, P.F32, P.ACT_GELU, 1, 8,
                            NULL, 0, None)
    assert P.STATUS[st] == "PARTIR_E_HIP"
    st = L.partir_attn_block(NULL, NULL, NULL, NULL, NULL, NULL, 0, 256, 1024, 8, 128, 1, 0.0,
                             P.BF16, P.F32, 1, 8, NULL, 0, None)
    assert P.STATUS[st] == "PARTIR_E_HIP"


# ---------------------------------------------------------------------------
# attention core with the key axis as a loop
# ---------------------------------------------------------------------------
def test_attention_core_plans():
    one = P.plan_attention(2, 2048, 8, 128, True, 1)
    assert one["n_launches"] == 1 and one["workspace_bytes"] == 0 and one["n_sum_loops"] == 0
    four = P.plan_attention(2, 2048, 8, 128, True, 4)
    T, D = 2 * 2048, 8 * 128
    assert four["n_launches"] == 2 and four["n_sum_loops"] == 1 and four["n_virtual_shards"] == 4
    assert four["workspace_bytes"] == 4 * T * D * 4 + 2 * 4 * T * 8 * 4
    assert four["flops"] == one["flops"] == 4.0 * 2 * 8 * (2048 * 2049 / 2) * 128
    assert "#sum softmax" in four["text"]
    assert P.lib().partir_attention_workspace(2, 2048, 8, 128, 4) == four["workspace_bytes"]


def test_attention_core_causal_parts():
    """A causal grid too small to fill the device runs each shard of >= 2048
    keys as ordered parts of >= 1024 keys; full attention, R_kv = 1 and large
    grids keep one part per shard."""
    B, S, H, R = 1, 8192, 2, 4
    T, D = B * S, H * 128
    causal = P.plan_attention(B, S, H, 128, True, R)
    assert "each as 2 ordered parts of 1024" in causal["text"] and "4 key shards of 2048" in causal["text"]
    assert causal["workspace_bytes"] == 8 * T * D * 4 + 2 * 8 * T * H * 4
    assert causal["n_virtual_shards"] == 4 and causal["n_launches"] == 2
    full = P.plan_attention(B, S, H, 128, False, R)
    assert "ordered parts" not in full["text"] and full["workspace_bytes"] == 4 * T * D * 4 + 2 * 4 * T * H * 4
    assert P.lib().partir_attention_workspace(B, S, H, 128, R) == causal["workspace_bytes"]
    assert "ordered parts" not in P.plan_attention(B, S, H, 128, True, 1)["text"]
    assert "ordered parts" not in P.plan_attention(4, S, 32, 128, True, R)["text"]      # 8192 workgroups
    four = P.plan_attention(1, 32768, 1, 128, True, 4)       # 128 key blocks a shard, 1024 workgroups
    assert "each as 2 ordered parts of 4096" in four["text"]
    eight = P.plan_attention(1, 32768, 1, 128, True, 2)      # 256 key blocks a shard, 512 workgroups
    assert "each as 4 ordered parts of 4096" in eight["text"]


@pytest.mark.parametrize("kwargs,status", [
    (dict(R=3), "PARTIR_E_DIVISIBILITY"),     # 32 key blocks of 64
    (dict(R=0), "PARTIR_E_UNSUPPORTED"),
    (dict(S=200), "PARTIR_E_SHAPE"),
    (dict(dh=64), "PARTIR_E_SHAPE"),
    (dict(S=1 << 20, H=16), "PARTIR_E_SHAPE"),  # one sequence's K: 2^20 x 2048 bf16 = 4 GiB
    (dict(B=256, S=1 << 16, H=8, R=1024), "PARTIR_E_SHAPE"),  # 2^30 workgroups
    (dict(Q=NULL), "PARTIR_E_NULL"),
    (dict(Q=DUMMY_ODD), "PARTIR_E_LAYOUT"),
    (dict(ws_bytes=0), "PARTIR_E_WORKSPACE"),
    (dict(), "PARTIR_E_HIP"),                  # valid: stops at the forced launch failure
])
def test_attention_core_validation(kwargs, status):
    a = dict(Q=DUMMY, B=2, S=2048, H=8, dh=128, R=4, ws_bytes=1 << 30)
    a.update(kwargs)
    st = P.lib().partir_attention(a["Q"], DUMMY, DUMMY, DUMMY, a["B"], a["S"], a["H"], a["dh"], 1, 0.0, a["R"],
                                  DUMMY, a["ws_bytes"], None)
    assert P.STATUS[st] == status, P.lib().partir_last_error().decode()


# ---------------------------------------------------------------------------
# MLP backward: the gradient reductions of batch (dW) and model (dX) loops
# ---------------------------------------------------------------------------
def mlp_bwd(T=512, D=256, F=1024, act=P.ACT_GELU, Rb=2, Rm=4, X=DUMMY, dX=DUMMY, dW=DUMMY, db=None,
            ws=DUMMY, ws_bytes=1 << 30):
    return P.lib().partir_mlp_block_backward(X, DUMMY, None, DUMMY, DUMMY, None, dX, dW, db, dW, db,
                                             T, D, F, act, Rb, Rm, ws, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(X=NULL), "PARTIR_E_NULL"),
    (dict(dW=NULL), "PARTIR_E_NULL"),
    (dict(T=0, dX=NULL, dW=NULL), "PARTIR_E_NULL"),    # the weight gradients still hold elements
    (dict(T=-1), "PARTIR_E_SHAPE"),
    (dict(T=1 << 28, F=1 << 12, D=1 << 10), "PARTIR_E_SHAPE"),
    (dict(Rm=0), "PARTIR_E_UNSUPPORTED"),
    (dict(act=7), "PARTIR_E_UNSUPPORTED"),
    (dict(Rm=3), "PARTIR_E_DIVISIBILITY"),
    (dict(Rb=3), "PARTIR_E_DIVISIBILITY"),
    (dict(D=252), "PARTIR_E_LAYOUT"),
    (dict(T=520, Rb=5), "PARTIR_E_HIP"),               # 104 tokens per shard: whole 16-byte runs
    (dict(T=500, Rb=5), "PARTIR_E_LAYOUT"),            # 100 tokens per shard are not
    (dict(F=1056, Rm=4), "PARTIR_E_HIP"),              # F/R = 264
    (dict(F=1040, Rm=4), "PARTIR_E_LAYOUT"),           # F/R = 260
    (dict(dX=DUMMY_ODD), "PARTIR_E_LAYOUT"),
    (dict(ws_bytes=100), "PARTIR_E_WORKSPACE"),
    (dict(), "PARTIR_E_HIP"),
    (dict(T=0, dX=NULL), "PARTIR_E_HIP"),              # no tokens: dX holds nothing
    (dict(F=0, dW=NULL), "PARTIR_E_HIP"),              # no hidden units: no weight gradients
])
def test_mlp_backward_validation(kwargs, status):
    assert P.STATUS[mlp_bwd(**kwargs)] == status, P.lib().partir_last_error().decode()


def test_mlp_backward_plans():
    T, D, F = 8192, 4096, 16384
    p = P.plan_mlp_block_backward(T, D, F, R_batch=2, R_model=8)
    t = p["text"]
    assert p["n_virtual_shards"] == 16 and p["n_tile_loops"] == 2 and p["n_sum_loops"] == 3
    assert p["flops"] == 10.0 * T * D * F
    # no transposed copies: W1 (as [K, N] for the recomputed Z) and the
    # activations are read in place; W1 and W2 are the K-contiguous
    # transposed operands of dX and dH
    assert "transpose" not in t and "act_backward" in t and t.count("read in place") == 3
    assert t.count("A as [K, M] B as [K, N]") == 2 and t.count("read in place: B as [K, N]") == 1
    # the batch #sum of the weight gradients runs over K = tokens, 2 shards
    assert "dW2 = sum_b" in t and "dW1 = sum_b" in t and "#sum K x2 (4096/shard)" in t
    # the model #sum of dX runs over K = F, 8 shards
    assert "dX = sum_m" in t and "#sum K x8 (2048/shard)" in t
    assert P.lib().partir_mlp_block_backward_workspace(T, D, F, P.ACT_GELU, 0, 2, 8) == p["workspace_bytes"]
    with_b = P.lib().partir_mlp_block_backward_workspace(T, D, F, P.ACT_GELU, 1, 2, 8)
    assert with_b == p["workspace_bytes"] + T // 64 * F * 4


def test_mlp_backward_empty_plans():
    e = P.plan_mlp_block_backward(0, 256, 1024, R_batch=2, R_model=4)
    assert e["n_launches"] == 2 and e["workspace_bytes"] == 0 and "empty_sum" in e["text"]
    f = P.plan_mlp_block_backward(512, 256, 0, R_batch=2, R_model=4)
    assert f["n_launches"] == 1 and f["workspace_bytes"] == 0          # dX = the empty #sum over m
    assert P.plan_mlp_block_backward(0, 0, 0)["n_launches"] == 0


def test_training_forward_validation(monkeypatch):
    monkeypatch.setenv("PARTIR_FAIL_LAUNCH", "1")
    L = P.lib()
    args = lambda Z, T=512: (DUMMY, DUMMY, None, DUMMY, None, DUMMY, Z, T, 256, 1024, P.BF16, P.F32, P.ACT_GELU,
                             1, 8, DUMMY, 1 << 30, None)
    assert P.STATUS[L.partir_mlp_block_train(*args(None))] == "PARTIR_E_NULL"
    assert P.STATUS[L.partir_mlp_block_train(*args(DUMMY_ODD))] == "PARTIR_E_LAYOUT"
    assert P.STATUS[L.partir_mlp_block_train(*args(DUMMY))] == "PARTIR_E_HIP"
    assert L.partir_last_plan_text().decode().startswith("mlp_block_train:")
    assert P.STATUS[L.partir_mlp_block_train(*args(None, T=0))] == "PARTIR_E_HIP"   # nothing to keep


# ---------------------------------------------------------------------------
# MLP on device-local arrays (BP + MP + Z3, activations sharded on M)
# ---------------------------------------------------------------------------
def sharded(T=1024, D=256, F=1024, Rb=2, Rm=4, parts=DUMMY, ws_bytes=1 << 30, out=P.F32):
    arr = (ctypes.c_void_p * (Rb * Rm))(*([parts] * (Rb * Rm)))
    return P.lib().partir_mlp_block_sharded(arr, arr, None, arr, None, arr, T, D, F, out, P.ACT_GELU, Rb, Rm,
                                            DUMMY, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(parts=NULL), "PARTIR_E_NULL"),
    (dict(parts=DUMMY_ODD), "PARTIR_E_LAYOUT"),
    (dict(T=1028), "PARTIR_E_DIVISIBILITY"),
    (dict(D=255), "PARTIR_E_DIVISIBILITY"),
    (dict(F=1022), "PARTIR_E_DIVISIBILITY"),
    (dict(T=512), "PARTIR_E_HIP"),                   # 64 rows per device is fine ...
    (dict(T=256), "PARTIR_E_LAYOUT"),                # ... 32 is not a whole load block
    (dict(D=64), "PARTIR_E_LAYOUT"),                 # D/R_batch = 32
    (dict(Rb=8, Rm=16, T=8192 * 16, D=512, F=1024), "PARTIR_E_UNSUPPORTED"),   # 128 devices
    (dict(out=7), "PARTIR_E_DTYPE"),
    (dict(ws_bytes=10), "PARTIR_E_WORKSPACE"),
    (dict(), "PARTIR_E_HIP"),
])
def test_sharded_validation(kwargs, status):
    assert P.STATUS[sharded(**kwargs)] == status, P.lib().partir_last_error().decode()


def test_sharded_plan():
    p = P.plan_mlp_block_sharded(8192, 4096, 16384, R_batch=2, R_model=4)
    assert p["n_launches"] == 2 and p["n_sum_loops"] == 1 and p["n_sum_splitk"] == 0
    assert p["n_virtual_shards"] == 8 and p["workspace_bytes"] == 8192 * 16384 * 2
    assert "fused all_gathers" in p["text"] and "fused reduce_scatter" in p["text"]
    assert P.lib().partir_mlp_block_sharded_workspace(8192, 4096, 16384, 2, 4) == p["workspace_bytes"]
    # a small grid still accumulates the whole #sum in the tile: the owner writes its rows
    s = P.plan_mlp_block_sharded(1024, 256, 1024, R_batch=2, R_model=4)
    assert s["n_sum_splitk"] == 0 and s["n_launches"] == 2
    e = P.plan_mlp_block_sharded(1024, 256, 0, R_batch=2, R_model=4)
    assert e["n_launches"] == 8 and e["workspace_bytes"] == 0        # b2 into each device's part


# ---------------------------------------------------------------------------
# attention core backward
# ---------------------------------------------------------------------------
def attn_bwd(B=2, S=2048, H=8, dh=128, ptr=DUMMY, lse=DUMMY, ws_bytes=1 << 30):
    return P.lib().partir_attention_backward(ptr, DUMMY, DUMMY, DUMMY, DUMMY, lse, DUMMY, DUMMY, DUMMY,
                                             B, S, H, dh, 1, 0.0, DUMMY, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(ptr=NULL), "PARTIR_E_NULL"),
    (dict(lse=NULL), "PARTIR_E_NULL"),
    (dict(ptr=DUMMY_ODD), "PARTIR_E_LAYOUT"),
    (dict(lse=ctypes.c_void_p(0x10002)), "PARTIR_E_LAYOUT"),
    (dict(S=200), "PARTIR_E_SHAPE"),
    (dict(dh=64), "PARTIR_E_SHAPE"),
    (dict(ws_bytes=0), "PARTIR_E_WORKSPACE"),
    (dict(), "PARTIR_E_HIP"),
    (dict(B=0, ptr=NULL, lse=NULL, ws_bytes=0), "PARTIR_E_HIP"),   # no tokens: valid, nothing launched
])
def test_attention_backward_validation(kwargs, status):
    assert P.STATUS[attn_bwd(**kwargs)] == status, P.lib().partir_last_error().decode()


def test_attention_backward_plan():
    p = P.plan_attention_backward(4, 2048, 32, 128, True)
    assert p["n_launches"] == 1 and p["workspace_bytes"] == 4 * 2048 * 32 * 4
    assert p["flops"] == 2.5 * 4.0 * 4 * 32 * (2048 * 2049 / 2) * 128
    assert "dq pass" in p["text"]
    assert P.lib().partir_attention_backward_workspace(4, 2048, 32, 128) == p["workspace_bytes"]


def test_attention_train_validation(monkeypatch):
    monkeypatch.setenv("PARTIR_FAIL_LAUNCH", "1")
    L = P.lib()
    st = L.partir_attention_train(DUMMY, DUMMY, DUMMY, DUMMY, None, 2, 2048, 8, 128, 1, 0.0, 1, DUMMY, 0, None)
    assert P.STATUS[st] == "PARTIR_E_NULL"
    st = L.partir_attention_train(DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, 2, 2048, 8, 128, 1, 0.0, 1, DUMMY, 0, None)
    assert P.STATUS[st] == "PARTIR_E_HIP"


# ---------------------------------------------------------------------------
# decoder layer on device-local arrays (sequence-parallel norms)
# ---------------------------------------------------------------------------
def dec_sharded(B=2, S=256, D=1024, H=8, F=2048, Rb=2, Rm=4, part=DUMMY, g=DUMMY, ws_bytes=1 << 34):
    nd = Rb * Rm
    arr = (ctypes.c_void_p * nd)(*([part] * nd))
    return P.lib().partir_decoder_layer_sharded(arr, g, g, 1e-6, arr, arr, arr, arr, arr, arr, B, S, D, H, 128, F,
                                                Rb, Rm, DUMMY, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(part=NULL), "PARTIR_E_NULL"),
    (dict(g=NULL), "PARTIR_E_NULL"),
    (dict(part=DUMMY_ODD), "PARTIR_E_LAYOUT"),
    (dict(F=2050), "PARTIR_E_DIVISIBILITY"),
    (dict(Rb=4, B=2), "PARTIR_E_DIVISIBILITY"),      # batch shards hold whole sequences
    (dict(F=1728), "PARTIR_E_LAYOUT"),               # F/R_model = 432 is not a multiple of 64
    (dict(D=512, H=4, Rb=2, Rm=4, F=2048), "PARTIR_E_HIP"),
    (dict(S=128, B=1, Rb=1, Rm=8, F=2048, D=1024), "PARTIR_E_HIP"),   # 16 tokens per device
    (dict(ws_bytes=10), "PARTIR_E_WORKSPACE"),
    (dict(), "PARTIR_E_HIP"),
])
def test_decoder_sharded_validation(kwargs, status):
    assert P.STATUS[dec_sharded(**kwargs)] == status, P.lib().partir_last_error().decode()


@pytest.mark.parametrize("Rb,Rm", [(4, 8), (8, 8), (2, 11), (3, 8)])
def test_decoder_sharded_meshes_beyond_the_part_table_are_refused(Rb, Rm):
    """The Q|K|V projection reads the three weights' blocks through one table
    of 64 parts, so meshes of more than 21 devices are refused before any plan
    is built (the size and plan queries included)."""
    B, S, H = 2 * Rb, 128 * Rm, 2 * Rm
    D, F = H * 128, 64 * Rb * Rm
    assert P.STATUS[dec_sharded(B=B, S=S, D=D, H=H, F=F, Rb=Rb, Rm=Rm)] == "PARTIR_E_UNSUPPORTED"
    assert "at most 21 devices" in P.lib().partir_last_error().decode()
    assert P.lib().partir_decoder_layer_sharded_workspace(B, S, D, H, 128, F, Rb, Rm) == ctypes.c_size_t(-1).value
    with pytest.raises(P.PartirError, match="UNSUPPORTED"):
        P.plan_decoder_layer_sharded(B, S, D, H, 128, F, R_batch=Rb, R_model=Rm)


def test_decoder_sharded_largest_mesh_plans():
    """21 devices (3 x 7) fill 63 entries of the part table: accepted."""
    Rb, Rm = 3, 7
    B, S, H = 3, 128 * 7, 21
    D, F = H * 128, 64 * 21
    assert P.STATUS[dec_sharded(B=B, S=S, D=D, H=H, F=F, Rb=Rb, Rm=Rm)] == "PARTIR_E_HIP"
    assert P.plan_decoder_layer_sharded(B, S, D, H, 128, F, R_batch=Rb, R_model=Rm)["n_virtual_shards"] == 21


def test_decoder_sharded_plan():
    p = P.plan_decoder_layer_sharded(4, 2048, 5120, 40, 128, 13824, R_batch=2, R_model=4)
    t = p["text"]
    assert p["n_sum_loops"] == 2 and p["n_sum_splitk"] == 0 and p["n_virtual_shards"] == 8
    assert t.count("sequence-parallel") == 2 and t.count("fused reduce_scatter") == 2
    # Q|K|V in one launch (three groups of weight blocks), FFN up
    assert t.count("fused all_gather") == 2 and t.count(".fixup:") == 3
    assert P.lib().partir_decoder_layer_sharded_workspace(4, 2048, 5120, 40, 128, 13824, 2, 4) == p["workspace_bytes"]


@pytest.mark.parametrize("M,N,K,tail,parts", [
    (8192, 5120, 5120, 128, 2),    # 640 tiles = 2 waves of 256 + 128: the 128 run as 2 K halves
    (8192, 15360, 5120, 128, 2),   # 1920 tiles
    (8192, 4096, 4096, 0, 1),      # 512 tiles: whole waves
    (8192, 13824, 4096, 0, 1),     # 1728 tiles: 192 left over, 2 x 192 would not fit one wave
    (512, 512, 4096, 4, 4),        # 4 tiles, 64 K tiles: 4 quarters of K each
    (512, 512, 256, 0, 1),         # 4 K tiles: too short to split
    (256, 256, 4096, 0, 1),        # 1 tile: 4 parts would not fill the 8 XCDs evenly
])
def test_last_wave_tail_split(M, N, K, tail, parts):
    """The load-balancing split of the last partial wave of output tiles:
    which tiles, how many K parts, the workspace for their fp32 accumulators
    and the fixup launch that adds them."""
    p = P.plan_loop_matmul(M, N, K)
    t = p["text"]
    if tail:
        assert f"the last {tail} tiles as {parts} K parts" in t and ".fixup:" in t
        assert p["n_launches"] == 2 and p["workspace_bytes"] == tail * parts * 512 * 128 * 4
    else:
        assert ".fixup" not in t and p["n_launches"] == 1 and p["workspace_bytes"] == 0
    assert P.lib().partir_loop_matmul_workspace(M, N, K, P.BF16, P.BF16, P.B_NK, -1, -1, 1, P.SUM_AUTO) == \
        p["workspace_bytes"]


def test_attn_block_backward_plan_reads_operands_in_place():
    """No transposed copies: Wo and W{q,k,v} are the K-contiguous transposed
    right operands of dA and dX (the three as K parts of one product), and
    dY, dQ|dK|dV, X and the attention output the [K, M] / [K, N] operands of
    the weight gradients."""
    B, S, D, H = 4, 2048, 4096, 32
    p = P.plan_attn_block_backward(B, S, D, H, R_batch=2, R_model=8)
    t = p["text"]
    assert "transpose" not in t
    assert t.count("B^T read as K parts Wq | Wk | Wv") == 1             # dX
    assert t.count("A as [K, M] B as [K, N]") == 4                      # dWq, dWk, dWv, dWo
    assert t.count("read in place") == 4
    assert P.lib().partir_attn_block_backward_workspace(B, S, D, H, 128, 2, 8) == p["workspace_bytes"]

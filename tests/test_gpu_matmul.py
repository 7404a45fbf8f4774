"""GPU parity of partir_loop_matmul against the oracle (fp32 and bf16 paths).

Every call goes through the C ABI (ctypes binding).  Element-by-element
comparison with the oracle's shard interpreter on the same seeded inputs; the
measure is max |C_gpu - C_ref| / (|A|.|B|).
"""
import numpy as np
import pytest
import torch

from oracle import partir_oracle as O
from paper_2401_11202_amd import inputs as I
from paper_2401_11202_amd import partir as P
from paper_2401_11202_amd import workloads as W
from tests.gpu_common import TOL_BF16, TOL_F32, accum_bound, host, say

pytestmark = pytest.mark.gpu

AX = {None: O.AXIS_NONE, "M": O.AXIS_M, "N": O.AXIS_N, "K": O.AXIS_K}


def run(A, B, tile, summ, R, b_layout, out_dtype=None, sum_impl="auto"):
    Ad = A.to_device()
    Bd = (B if b_layout == "kn" else I.transposed(B)).to_device()
    C = P.loop_matmul(Ad, Bd, tile=tile, sum=summ, R=R, b_layout=b_layout, out_dtype=out_dtype,
                      sum_impl=sum_impl)
    torch.cuda.synchronize()
    return C


def check(A, B, C, tile, summ, R, tol):
    ref = O.loop_matmul(A.f64(), B.f64(), AX[tile], AX[summ], R)
    norm = O.abs_product(A.f64(), B.f64())
    err = O.normalised_error(host(C), ref, norm)
    say(f"    max normalised error {err:.3e} (tol {tol:g})")
    assert err <= tol
    return err


# ---------------------------------------------------------------------------
def test_f32_sum_over_K_R4_full_size():
    """C[256,256] = A[256,512] B[512,256], #sum over K with 4 shards of 128."""
    w = W.WORKLOADS["matmul_f32_sumK"]
    x = W.make_inputs(w)
    for impl in ("auto", "fused", "splitk"):
        say(f"f32 256x256x512 sum K R=4 impl={impl}")
        C = run(x["A"], x["B"], None, "K", 4, "kn", sum_impl=impl)
        err = check(x["A"], x["B"], C, None, "K", 4, TOL_F32)
        assert err <= accum_bound(512)


@pytest.mark.parametrize("b_layout", ["kn", "nk"])
@pytest.mark.parametrize("tile,summ,R", [(None, None, 1), ("M", None, 4), ("N", None, 4), (None, "K", 4),
                                         ("M", "K", 2), ("N", "K", 4), (None, "K", 1)])
def test_f32_modes_ragged(tile, summ, R, b_layout):
    M, N, K = 200, 144, 80          # ragged against the 64-wide tiles
    A = I.gaussian(101, 0, (M, K), 1.0, "f32")
    B = I.gaussian(101, 1, (K, N), 1.0, "f32")
    for impl in ("fused", "splitk"):
        say(f"f32 {M}x{N}x{K} tile={tile} sum={summ} R={R} {b_layout} {impl}")
        C = run(A, B, tile, summ, R, b_layout, sum_impl=impl)
        check(A, B, C, tile, summ, R, TOL_F32)


@pytest.mark.parametrize("out", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("tile,summ,R", [("M", None, 3), ("N", None, 3), (None, "K", 3), (None, "K", 5),
                                         ("M", "K", 5), ("N", "K", 3)])
def test_bf16_odd_shard_counts(tile, summ, R, out):
    """Odd loop sizes: shards of 200 / 120 rows, 176 columns, 160 / 96 keys
    (none a multiple of the 256-wide tiles), fused and split-K sums."""
    M, N, K = 600, 528, 480
    A = I.gaussian(105, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(105, 1, (K, N), K ** -0.5, "bf16")
    for impl in ("fused", "splitk"):
        say(f"bf16 {M}x{N}x{K} tile={tile} sum={summ} R={R} out={out} {impl}")
        C = run(A, B, tile, summ, R, "nk", out_dtype=out, sum_impl=impl)
        err = check(A, B, C, tile, summ, R, TOL_BF16)
        assert err <= accum_bound(K) + (2.0 ** -8 if out == torch.bfloat16 else 0.0)


@pytest.mark.parametrize("out", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("tile,summ,R", [(None, None, 1), ("M", None, 4), ("N", None, 4), (None, "K", 4),
                                         ("M", "K", 4), ("N", "K", 2), (None, "K", 8)])
def test_bf16_modes_ragged(tile, summ, R, out):
    M, N, K = 600, 528, 448         # several 256-wide tiles with ragged tails
    A = I.gaussian(102, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(102, 1, (K, N), K ** -0.5, "bf16")
    for impl in ("fused", "splitk"):
        say(f"bf16 {M}x{N}x{K} tile={tile} sum={summ} R={R} out={out} {impl}")
        C = run(A, B, tile, summ, R, "nk", out_dtype=out, sum_impl=impl)
        err = check(A, B, C, tile, summ, R, TOL_BF16)
        # fp32 accumulation of exact bf16 products (+ one bf16 rounding of the output)
        bound = accum_bound(K) + (2.0 ** -8 if out == torch.bfloat16 else 0.0)
        assert err <= bound


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_integer_inputs_are_bitwise_exact(dtype):
    """Products and partial sums of small integers are exact in fp32, so every
    shard decomposition must reproduce the unpartitioned product bit for bit."""
    M, N, K = 320, 272, 512
    A = I.small_ints(103, 0, (M, K), dtype=dtype)
    B = I.small_ints(103, 1, (K, N), dtype=dtype)
    ref = O.matmul(A.f64(), B.f64())
    bl = "kn" if dtype == "f32" else "nk"
    for tile, summ, R in [(None, None, 1), ("M", None, 4), ("N", None, 4), (None, "K", 8), ("M", "K", 4)]:
        for impl in ("fused", "splitk"):
            say(f"integer {dtype} tile={tile} sum={summ} R={R} {impl}")
            C = run(A, B, tile, summ, R, bl, out_dtype=torch.float32, sum_impl=impl)
            assert np.array_equal(host(C), ref)


def test_results_are_deterministic():
    A = I.gaussian(104, 0, (512, 1024), 1.0, "bf16")
    B = I.gaussian(104, 1, (1024, 512), 1.0 / 32, "bf16")
    for impl in ("fused", "splitk"):
        c1 = run(A, B, None, "K", 8, "nk", out_dtype=torch.float32, sum_impl=impl)
        c2 = run(A, B, None, "K", 8, "nk", out_dtype=torch.float32, sum_impl=impl)
        assert torch.equal(c1, c2)


def test_shards_write_only_their_slices():
    """Guard bands: C is a view into a larger canary-filled buffer; nothing
    outside the [M, N] window may change."""
    M, N, K = 300, 272, 128
    A = I.gaussian(105, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(105, 1, (K, N), 0.1, "bf16")
    Ad, Bt = A.to_device(), I.transposed(B).to_device()
    for tile, summ, R in [("M", None, 4), ("N", None, 4), (None, "K", 4)]:
        for impl in ("fused", "splitk"):
            big = torch.full((M + 40, N + 48), 1234.5, dtype=torch.float32, device="cuda")
            view = big[16:16 + M, 8:8 + N]
            P.loop_matmul(Ad, Bt, tile=tile, sum=summ, R=R, b_layout="nk", out_dtype=torch.float32,
                          sum_impl=impl, out=view)
            torch.cuda.synchronize()
            mask = torch.ones_like(big, dtype=torch.bool)
            mask[16:16 + M, 8:8 + N] = False
            assert torch.all(big[mask] == 1234.5), (tile, summ, impl)
            err = O.normalised_error(host(view), O.matmul(A.f64(), B.f64()), O.abs_product(A.f64(), B.f64()))
            assert err <= TOL_BF16


def test_fused_and_split_sum_agree():
    A = I.gaussian(106, 0, (512, 2048), 1.0, "bf16")
    B = I.gaussian(106, 1, (2048, 768), 2048 ** -0.5, "bf16")
    f = run(A, B, None, "K", 8, "nk", out_dtype=torch.float32, sum_impl="fused")
    s = run(A, B, None, "K", 8, "nk", out_dtype=torch.float32, sum_impl="splitk")
    norm = O.abs_product(A.f64(), B.f64())
    assert O.normalised_error(host(f), host(s), norm) <= 2 * accum_bound(2048)


def test_validation_errors_leave_output_untouched():
    A = torch.ones((64, 96), dtype=torch.float32, device="cuda")
    B = torch.ones((96, 64), dtype=torch.float32, device="cuda")
    C = torch.full((64, 64), 7.0, device="cuda")
    with pytest.raises(P.PartirError) as e:
        P.loop_matmul(A, B, sum="K", R=5, out=C)
    assert e.value.status == P.ERR["PARTIR_E_DIVISIBILITY"]
    torch.cuda.synchronize()
    assert torch.all(C == 7.0)


# ---------------------------------------------------------------------------
# empty operands
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,out", [("bf16", torch.float32), ("bf16", torch.bfloat16), ("f32", torch.float32)])
def test_empty_contraction_is_the_empty_sum(dtype, out):
    """K = 0: the sum over no K shards is 0 everywhere (exact), whatever the
    loop nest; the output window is fully written."""
    M, N = 300, 272
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    bl = "nk" if dtype == "bf16" else "kn"
    A = torch.empty((M, 0), dtype=tdt, device="cuda")
    B = torch.empty((N, 0) if bl == "nk" else (0, N), dtype=tdt, device="cuda")
    C = torch.empty((M, N), dtype=out, device="cuda")
    for tile, summ, R in [(None, "K", 4), ("M", None, 4), ("N", "K", 2), (None, None, 1)]:
        say(f"empty K {dtype} -> {out} tile={tile} sum={summ} R={R}")
        C.fill_(7.0)
        P.loop_matmul(A, B, tile=tile, sum=summ, R=R, b_layout=bl, out_dtype=out, out=C)
        torch.cuda.synchronize()
        ref = O.loop_matmul(np.zeros((M, 0)), np.zeros((0, N)), AX[tile], AX[summ], R)
        assert np.array_equal(host(C), ref)


def test_empty_output_is_a_no_op():
    """M = 0 or N = 0: every #tile shard is empty; nothing is launched and the
    result has the right (empty) shape."""
    A = I.gaussian(107, 0, (0, 64), 1.0, "bf16").to_device()
    Bt = I.transposed(I.gaussian(107, 1, (64, 48), 1.0, "bf16")).to_device()
    C = P.loop_matmul(A, Bt, tile="M", R=4, b_layout="nk", out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert tuple(C.shape) == (0, 48)
    A2 = I.gaussian(107, 2, (32, 64), 1.0, "bf16").to_device()
    Bt2 = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    C2 = P.loop_matmul(A2, Bt2, tile="N", R=4, b_layout="nk", out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert tuple(C2.shape) == (32, 0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_degenerate_shard_sizes(dtype):
    """R as large as the layout allows: single-row M shards, N shards of one
    16-byte run, K shards of one 16-byte run (64 of them, summed in order)."""
    vec = 8 if dtype == "bf16" else 4
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    bl = "nk" if dtype == "bf16" else "kn"
    cases = [(64, 256, 128, "M", None, 64),            # 64 shards of 1 row
             (96, 32 * vec, 128, "N", None, 32),       # 32 shards of `vec` columns
             (128, 256, 64 * vec, None, "K", 64),      # 64 K shards of `vec`
             (64, 16 * vec, 16 * vec, "M", "K", 16)]   # 16 x 16 nest, 4-row tiles of vec-wide K shards
    for (M, N, K, tile, summ, R) in cases:
        A = I.gaussian(110, 0, (M, K), 1.0, dtype)
        B = I.gaussian(110, 1, (K, N), K ** -0.5, dtype)
        for impl in ("fused", "splitk"):
            say(f"degenerate {dtype} {M}x{N}x{K} tile={tile} sum={summ} R={R} {impl}")
            C = run(A, B, tile, summ, R, bl, out_dtype=torch.float32, sum_impl=impl)
            check(A, B, C, tile, summ, R, tol)


# ---------------------------------------------------------------------------
# The last, partial wave of output tiles split into K parts (load balance):
# 1000 x 304 outputs are 8 tiles of 256 x 256 (16 with #tile N x4), each run
# as 4 workgroups over 17 + 17 + 17 + 14 of the 65 K tiles (K = 4112: the
# last K tile holds 16 columns); a fixup launch adds the parts in order.
@pytest.mark.parametrize("out", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("tile,summ,R", [(None, None, 1), ("M", None, 4), ("N", None, 4), (None, "K", 2),
                                         ("M", "K", 2)])
def test_bf16_last_wave_split_ragged(tile, summ, R, out):
    M, N, K = 1000, 304, 4112
    plan = P.plan_loop_matmul(M, N, K, ab=P.BF16, c=P.F32 if out == torch.float32 else P.BF16,
                              tile=tile, sum=summ, R=R, sum_impl=P.SUM_FUSED)
    assert "K parts of 17 K tiles" in plan["text"], plan["text"]
    A = I.gaussian(121, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(121, 1, (K, N), K ** -0.5, "bf16")
    say(f"bf16 last-wave split {M}x{N}x{K} tile={tile} sum={summ} R={R} out={out}")
    C = run(A, B, tile, summ, R, "nk", out_dtype=out, sum_impl="fused")
    err = check(A, B, C, tile, summ, R, TOL_BF16)
    assert err <= accum_bound(K) + (2.0 ** -8 if out == torch.bfloat16 else 0.0)


def test_last_wave_split_integer_exact_and_deterministic():
    """Small-integer inputs: every partial and their sum are exact in fp32, so
    the split tiles equal the oracle bit for bit; repeated calls agree."""
    M, N, K = 1000, 304, 4112
    A = I.small_ints(122, 0, (M, K), dtype="bf16")
    B = I.small_ints(122, 1, (K, N), dtype="bf16")
    ref = O.matmul(A.f64(), B.f64())
    c1 = run(A, B, "M", None, 4, "nk", out_dtype=torch.float32)
    c2 = run(A, B, "M", None, 4, "nk", out_dtype=torch.float32)
    assert np.array_equal(host(c1), ref) and torch.equal(c1, c2)


def test_last_wave_split_full_size_sampled_rows():
    """8192 x 5120 x 5120 (640 tiles: two whole waves, then 128 tiles as 2 K
    halves of 40 K tiles): whole output rows, sampled across every tile row,
    against the oracle's matmul of those rows."""
    M, N, K = 8192, 5120, 5120
    assert "the last 128 tiles as 2 K parts of 40 K tiles" in P.plan_loop_matmul(M, N, K)["text"]
    A = I.gaussian(123, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(123, 1, (K, N), K ** -0.5, "bf16")
    say(f"bf16 last-wave split {M}x{N}x{K} (sampled rows)")
    C = host(run(A, B, None, None, 1, "nk", out_dtype=torch.float32))
    rows = sorted({0, M - 1} | {256 * t + (37 * t) % 256 for t in range(M // 256)})
    Ar = A.f64()[rows]
    err = O.normalised_error(C[rows], O.matmul(Ar, B.f64()), O.abs_product(Ar, B.f64()))
    say(f"    {len(rows)} rows, max normalised error {err:.3e}")
    assert err <= accum_bound(K)


# ---------------------------------------------------------------------------
# bf16 B given as a row-major [K, N] array (read in place: MN-major tiles and
# transposed fragment reads in the GEMM)
@pytest.mark.parametrize("out", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("tile,summ,R", [(None, None, 1), ("M", None, 4), ("N", None, 4), (None, "K", 4),
                                         ("M", "K", 4), ("N", "K", 2), (None, "K", 8)])
def test_bf16_b_kn_modes_ragged(tile, summ, R, out):
    M, N, K = 600, 544, 448         # several 256-wide tiles with ragged tails
    A = I.gaussian(124, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(124, 1, (K, N), K ** -0.5, "bf16")
    for impl in ("fused", "splitk"):
        say(f"bf16 B[K,N] {M}x{N}x{K} tile={tile} sum={summ} R={R} out={out} {impl}")
        C = run(A, B, tile, summ, R, "kn", out_dtype=out, sum_impl=impl)
        err = check(A, B, C, tile, summ, R, TOL_BF16)
        assert err <= accum_bound(K) + (2.0 ** -8 if out == torch.bfloat16 else 0.0)


def test_bf16_b_kn_integer_exact_and_layouts_agree():
    """Small integers: B as [K, N] and as B^T [N, K] both give the exact
    product, bit for bit; also through the last-wave split (K = 4160)."""
    for M, N, K in [(320, 272, 512), (1000, 320, 4160)]:
        A = I.small_ints(125, 0, (M, K), dtype="bf16")
        B = I.small_ints(125, 1, (K, N), dtype="bf16")
        ref = O.matmul(A.f64(), B.f64())
        for tile, summ, R in [(None, None, 1), ("M", None, 4), ("N", None, 2), (None, "K", 8)]:
            say(f"integer bf16 B[K,N] {M}x{N}x{K} tile={tile} sum={summ} R={R}")
            kn = run(A, B, tile, summ, R, "kn", out_dtype=torch.float32)
            nk = run(A, B, tile, summ, R, "nk", out_dtype=torch.float32)
            assert np.array_equal(host(kn), ref) and torch.equal(kn, nk)


def test_bf16_b_kn_full_size_sampled_rows():
    M, N, K = 8192, 4096, 4096
    A = I.gaussian(126, 0, (M, K), 1.0, "bf16")
    B = I.gaussian(126, 1, (K, N), K ** -0.5, "bf16")
    say(f"bf16 B[K,N] {M}x{N}x{K} (sampled rows)")
    C = host(run(A, B, None, None, 1, "kn", out_dtype=torch.float32))
    rows = sorted({0, M - 1} | {256 * t + (53 * t) % 256 for t in range(M // 256)})
    Ar = A.f64()[rows]
    err = O.normalised_error(C[rows], O.matmul(Ar, B.f64()), O.abs_product(Ar, B.f64()))
    say(f"    {len(rows)} rows, max normalised error {err:.3e}")
    assert err <= accum_bound(K)


@pytest.mark.parametrize("summ,R", [(None, 1), ("K", 4)])
def test_bf16_at_the_largest_leading_dimension(summ, R):
    """K = lda = ldb = 2^24, the largest bf16 leading dimension the boundary
    admits: a 64-row block of an operand then spans exactly 2^31 bytes, the
    top of a buffer descriptor's range.  Entries in {-1, 0, 1} keep every
    partial sum an integer below 2^24, so fp32 accumulation is exact and the
    sampled outputs are compared bit for bit with fp64 dot products."""
    M = N = 64
    K = 1 << 24
    g = torch.Generator(device="cuda").manual_seed(2024)
    A = torch.randint(-1, 2, (M, K), generator=g, device="cuda", dtype=torch.int8).to(torch.bfloat16)
    Bt = torch.randint(-1, 2, (N, K), generator=g, device="cuda", dtype=torch.int8).to(torch.bfloat16)
    say(f"bf16 matmul {M}x{N}x{K} (lda = ldb = 2^24), sum={summ} R={R}")
    C = P.loop_matmul(A, Bt, sum=summ, R=R, b_layout="nk", out_dtype=torch.float32)
    torch.cuda.synchronize()
    c = host(C)
    rng = np.random.default_rng(2024)
    pairs = [(0, 0), (M - 1, N - 1), (M - 1, 0)] + [(int(rng.integers(M)), int(rng.integers(N))) for _ in range(5)]
    a_rows = {i: A[i].float().cpu().numpy().astype(np.float64) for i, _ in pairs}
    b_rows = {j: Bt[j].float().cpu().numpy().astype(np.float64) for _, j in pairs}
    for i, j in pairs:
        assert c[i, j] == float(np.dot(a_rows[i], b_rows[j])), (i, j)
    del A, Bt, C
    torch.cuda.empty_cache()

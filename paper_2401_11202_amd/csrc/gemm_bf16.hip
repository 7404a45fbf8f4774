// bf16 MFMA GEMM for gfx950: C = A . B^T with both operands K-contiguous.
//
// One workgroup computes a 256x256 output tile of one virtual shard with four
// waves (2 x 2), each owning a 128x128 sub-tile as 4 x 4 accumulators of
// v_mfma_f32_32x32x16_bf16.  K advances in 64-wide steps through a
// double-buffered LDS stage (A and B tiles, 32 KiB each) filled from
// registers; global loads are raw buffer loads whose out-of-range lanes read
// zero, which covers ragged M / N / K edges without branches.
//
// Loop semantics realised here (PartIR:Core, Sec. 5 / App. C):
//  * #tile over M or N: the grid enumerates every shard's tiles; a tile never
//    straddles a shard and stores into the shard's slice of C.
//  * #sum over K, fused: the shards' K-ranges are consecutive, so one tile's
//    K loop walks shard 0, 1, ..., R-1 in order into one accumulator.
//  * #sum over K, split: the grid also enumerates the K shards and each writes
//    its own fp32 partial; an ordered reduction (splitk_reduce.hip) sums them.
#include "kernels.h"

namespace partir {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 256, BN = 256, BK = 64, NT = 256;
constexpr int STAGE = (BM + BN) * BK * 2;       // bytes of one LDS stage
constexpr uint32_t OOB = 0x80000000u;          // offset that reads as zero

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)OOB, 0x00020000);
}

__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

template <int EPI, int ACT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_bf16_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---- which tile of which virtual shard ----------------------------------
  const int ntiles = p.tiles_m * p.tiles_n;
  int bid = blockIdx.x;
  const int nwg = gridDim.x;
  // Workgroups go round-robin to the 8 XCDs; give each XCD a contiguous run
  // of the tile order so neighbouring tiles share that XCD's L2.
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  const int split = bid / ntiles;
  const int t = bid - split * ntiles;
  const int per_group = p.group_m * p.tiles_n;
  const int gidx = t / per_group;
  const int first_m = gidx * p.group_m;
  const int gm = min(p.tiles_m - first_m, p.group_m);
  const int rr = t - gidx * per_group;
  const int tm = first_m + rr % gm;
  const int tn = rr / gm;

  const int sm = tm / p.tpm, tmi = tm - sm * p.tpm;
  const int row0 = sm * p.ms + tmi * BM;
  const int rows = min(BM, p.ms - tmi * BM);
  const int per_gn = p.rn * p.tpn;
  const int grp = tn / per_gn, rem = tn - grp * per_gn;
  const int sn = rem / p.tpn, tni = rem - sn * p.tpn;
  const int col0 = sn * p.ns + tni * BN;
  const int cols = min(BN, p.ns - tni * BN);
  const int k_begin = (p.nsplit > 1) ? split * p.ks : 0;
  const int k_end = (p.nsplit > 1) ? k_begin + p.ks : p.K;

  // ---- global -> register loads (8 x 16 B of A and of B per thread) -----------
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A + (int64_t)row0 * p.lda);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.B[grp] + (int64_t)col0 * p.ldb);
  const int lr = tid >> 3;   // tile row 0..31 (+32 i)
  const int lc = tid & 7;    // 16-byte chunk of the 64-wide K step
  uint32_t a_off[8], b_off[8];
  uint32_t a_ok = 0, b_ok = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = lr + 32 * i;
    a_off[i] = (uint32_t)(r * p.lda * 2 + lc * 16);
    b_off[i] = (uint32_t)(r * p.ldb * 2 + lc * 16);
    a_ok |= (uint32_t)(r < rows) << i;
    b_ok |= (uint32_t)(r < cols) << i;
  }
  // LDS tiles are [row][64 k] with the 16-byte chunk index XOR-swizzled by
  // swz(row) = (row & 7) ^ ((row >> 3) & 1), so the 32 rows one MFMA operand
  // read touches spread over all banks.
  const int st_off = lr * 128 + ((lc ^ ((lr & 7) ^ ((lr >> 3) & 1))) << 4);

  i32x4 sa[8], sb[8];
  auto gload = [&](int kt) {
    const int kb = k_begin + kt * BK;
    const bool kv = kb + lc * 8 < k_end;
    const uint32_t so = (uint32_t)kb * 2;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t va = (kv && ((a_ok >> i) & 1)) ? a_off[i] : OOB;
      const uint32_t vb = (kv && ((b_ok >> i) & 1)) ? b_off[i] : OOB;
      sa[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, va, so, 0);
      sb[i] = __builtin_amdgcn_raw_buffer_load_b128(rb, vb, so, 0);
    }
  };
  auto lstore = [&](int buf) {
    char* as = smem + buf * STAGE;
    char* bs = as + BM * BK * 2;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      *(i32x4*)(as + st_off + i * 4096) = sa[i];
      *(i32x4*)(bs + st_off + i * 4096) = sb[i];
    }
  };

  // ---- MFMA operand reads -----------------------------------------------------
  const int h = lane >> 5;
  const int swz = (lane & 7) ^ ((lane >> 3) & 1);
  const int a_rd = (wm * 128 + (lane & 31)) * 128;
  const int b_rd = (wn * 128 + (lane & 31)) * 128;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  auto compute = [&](int buf) {
    const char* as = smem + buf * STAGE;
    const char* bs = as + BM * BK * 2;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int ko = ((2 * kk + h) ^ swz) << 4;
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = *(const bf16x8*)(as + a_rd + i * 4096 + ko);
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = *(const bf16x8*)(bs + b_rd + j * 4096 + ko);
      // B as the first operand: each lane ends up holding 4 consecutive
      // output columns of one output row.
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
    }
  };

  const int nk = (k_end - k_begin + BK - 1) / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    compute(cur);
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds C[m][n..n+3] for each (i, j, g) ---------------------
  const float* bias = p.bias[grp];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ml = wm * 128 + i * 32 + (lane & 31);
    if (ml >= rows) continue;
    const int64_t m = row0 + ml;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl = wn * 128 + j * 32 + 8 * g + 4 * h;
        if (nl >= cols) continue;
        const int64_t n = col0 + nl;
        f32x4 v = {acc[i][j][4 * g + 0], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
        if (EPI == EPI_PARTIAL) {
          *(f32x4*)(p.partial + split * p.part_stride + m * p.part_ld + n) = v;
          continue;
        }
        if (bias) {
          const f32x4 bv = *(const f32x4*)(bias + n);
          v += bv;
        }
        if (ACT) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = gelu_erf(v[e]);
        }
        if (EPI == EPI_BF16) {
          bf16x4 o = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
          *(bf16x4*)((uint16_t*)p.C[grp] + m * p.ldc + n) = o;
        } else if (EPI == EPI_F32) {
          *(f32x4*)((float*)p.C[grp] + m * p.ldc + n) = v;
        } else {  // EPI_RESID_F32
          const f32x4 r = *(const f32x4*)(p.resid + m * p.ldr + n);
          *(f32x4*)((float*)p.C[grp] + m * p.ldc + n) = r + v;
        }
      }
    }
  }
}

template <int EPI, int ACT>
hipError_t launch(const GemmParams& p, hipStream_t s) {
  const int64_t nwg = (int64_t)p.tiles_m * p.tiles_n * p.nsplit;
  hipLaunchKernelGGL((gemm_bf16_kernel<EPI, ACT>), dim3((unsigned)nwg), dim3(NT), 0, s, p);
  return hipGetLastError();
}

}  // namespace

int gemm_bf16_tile_m() { return BM; }
int gemm_bf16_tile_n() { return BN; }

hipError_t launch_gemm_bf16(const GemmParams& p, hipStream_t s) {
  switch (p.epi * 2 + (p.act ? 1 : 0)) {
    case EPI_BF16 * 2 + 0: return launch<EPI_BF16, 0>(p, s);
    case EPI_BF16 * 2 + 1: return launch<EPI_BF16, 1>(p, s);
    case EPI_F32 * 2 + 0: return launch<EPI_F32, 0>(p, s);
    case EPI_F32 * 2 + 1: return launch<EPI_F32, 1>(p, s);
    case EPI_PARTIAL * 2 + 0: return launch<EPI_PARTIAL, 0>(p, s);
    case EPI_RESID_F32 * 2 + 0: return launch<EPI_RESID_F32, 0>(p, s);
    case EPI_RESID_F32 * 2 + 1: return launch<EPI_RESID_F32, 1>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace partir

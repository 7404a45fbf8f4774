// fp32 MFMA GEMM for gfx950 (v_mfma_f32_32x32x2_f32): C = A . B.
//
// 64x64 output tile per workgroup, four waves of 32x32, K in steps of 16
// through LDS held k-major ([k][m] and [k][n]) so each lane's single-element
// MFMA operands are conflict-free reads.  B may be row-major [K, N] or given
// by its transpose [N, K].  Same shard grid as the bf16 GEMM: tiles of #tile
// shards, and for a #sum either one accumulator over all K shards in order or
// one fp32 partial per K shard.
#include "kernels.h"

namespace partir {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int T = 64, BK = 16, NT = 256, PAD = 4;

__global__ __launch_bounds__(NT) void gemm_f32_kernel(GemmF32Params p) {
  __shared__ float As[BK][T + PAD];
  __shared__ float Bs[BK][T + PAD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const int ntiles = p.tiles_m * p.tiles_n;
  const int split = blockIdx.x / ntiles;
  const int t = blockIdx.x - split * ntiles;
  const int tm = t / p.tiles_n, tn = t - (t / p.tiles_n) * p.tiles_n;
  const int sm = tm / p.tpm, tmi = tm - sm * p.tpm;
  const int row0 = sm * p.ms + tmi * T;
  const int rows = min(T, p.ms - tmi * T);
  const int sn = tn / p.tpn, tni = tn - sn * p.tpn;
  const int col0 = sn * p.ns + tni * T;
  const int cols = min(T, p.ns - tni * T);
  const int k_begin = (p.nsplit > 1) ? split * p.ks : 0;
  const int k_end = (p.nsplit > 1) ? k_begin + p.ks : p.K;

  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;

  // loader coordinates: A tile [64 m][16 k] as 256 float4 along k
  const int am = tid >> 2, ak = (tid & 3) * 4;
  for (int kb = k_begin; kb < k_end; kb += BK) {
    {
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (am < rows && kb + ak < k_end) v = *(const f32x4*)(p.A + (int64_t)(row0 + am) * p.lda + kb + ak);
#pragma unroll
      for (int e = 0; e < 4; ++e) As[ak + e][am] = v[e];
    }
    if (p.b_nk) {  // B^T [N, K]: same pattern as A
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (am < cols && kb + ak < k_end) v = *(const f32x4*)(p.B + (int64_t)(col0 + am) * p.ldb + kb + ak);
#pragma unroll
      for (int e = 0; e < 4; ++e) Bs[ak + e][am] = v[e];
    } else {       // B [K, N]: 16 rows of 64 along n
      const int bk = tid >> 4, bn = (tid & 15) * 4;
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (bn < cols && kb + bk < k_end) v = *(const f32x4*)(p.B + (int64_t)(kb + bk) * p.ldb + col0 + bn);
      *(f32x4*)&Bs[bk][bn] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
      const float a = As[kk + (lane >> 5)][wm * 32 + (lane & 31)];
      const float b = Bs[kk + (lane >> 5)][wn * 32 + (lane & 31)];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
    __syncthreads();
  }

  // lane holds C[m = 8g + 4h + e][n = lane & 31] of the wave's 32x32 block
  const int nl = wn * 32 + (lane & 31);
  if (nl >= cols) return;
  float* out = p.C + (p.epi == EPI_PARTIAL ? split * p.part_stride : 0);
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int ml = wm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    if (ml < rows) out[(int64_t)(row0 + ml) * p.ldc + col0 + nl] = acc[v];
  }
}

}  // namespace

int gemm_f32_tile() { return T; }

hipError_t launch_gemm_f32(const GemmF32Params& p, hipStream_t s) {
  const int64_t nwg = (int64_t)p.tiles_m * p.tiles_n * p.nsplit;
  hipLaunchKernelGGL(gemm_f32_kernel, dim3((unsigned)nwg), dim3(NT), 0, s, p);
  return hipGetLastError();
}

}  // namespace partir

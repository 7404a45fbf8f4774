// HBM-bound helpers of the MLP backward pass: the activation backward (dZ
// and H from Z and dH, with the block column sums of dZ for db1 fused) and
// deterministic column sums for the bias gradients.
#include "kernels.h"
#include "device_math.h"

namespace partir {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int TT = 64;          // tile edge
constexpr int TP = TT + 2;      // LDS row pitch in elements (spreads columns over banks)

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// 256 threads per 64 x 64 tile; thread t handles 16-byte chunks (8 elements).
__global__ __launch_bounds__(256) void act_backward_kernel(ActBwdParams p) {
  __shared__ uint16_t tdz[TT][TP];
  const int ntc = (p.cols + TT - 1) / TT;      // 1-D grid: tile (row block, col block)
  const int r0 = (int)(blockIdx.x / ntc) * TT, c0 = (int)(blockIdx.x % ntc) * TT;
  const int tid = threadIdx.x;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int id = tid + 256 * k;
    const int r = id >> 3, c = (id & 7) * 8;
    if (r0 + r < p.rows && c0 + c < p.cols) {
      const int64_t off = (int64_t)(r0 + r) * p.ld + c0 + c;
      const i32x4 zv = *(const i32x4*)(p.Z + off);
      const i32x4 gv = *(const i32x4*)(p.dH + off);
      const uint16_t* z = (const uint16_t*)&zv;
      const uint16_t* g = (const uint16_t*)&gv;
      i32x4 dzv, hv;
      uint16_t* dz = (uint16_t*)&dzv;
      uint16_t* hh = (uint16_t*)&hv;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float x = bf2f(z[j]);
        float y = x, d = 1.0f;
        if (p.act) gelu_erf_and_grad(x, y, d);
        dz[j] = f2bf(bf2f(g[j]) * d);
        hh[j] = f2bf(y);
        tdz[r][c + j] = dz[j];
      }
      *(i32x4*)(p.dZ + off) = dzv;
      *(i32x4*)(p.H + off) = hv;
    }
  }
  __syncthreads();
  if (p.colpart) {
    // column sums of the stored dZ over this tile's rows: four quarters of 16
    // rows, then the quarters in order (a fixed order: deterministic)
    __shared__ float qs[4][TT];
    const int c = tid & (TT - 1), q = tid >> 6;
    const int nr = min(TT, p.rows - r0);
    float s = 0.0f;
    if (c0 + c < p.cols)
      for (int r = q * 16; r < min(nr, q * 16 + 16); ++r) s += bf2f(tdz[r][c]);
    qs[q][c] = s;
    __syncthreads();
    if (q == 0 && c0 + c < p.cols)
      p.colpart[(int64_t)(r0 / TT) * p.cols + c0 + c] = ((qs[0][c] + qs[1][c]) + qs[2][c]) + qs[3][c];
  }
}

// stage 1: partial[b][c] = sum_{r in block b} in[r][c] over blocks of 64
// rows, as four quarters of 16 rows added in order; a thread owns 8 columns
// (one 16-byte load per row)
__global__ __launch_bounds__(256) void colsum_partial_kernel(ColSumParams p) {
  const int c = (blockIdx.y * 256 + threadIdx.x) * 8;
  const int b = blockIdx.x;
  if (c >= p.cols) return;
  const int r0 = b * kColSumChunk, r1 = min(p.rows, r0 + kColSumChunk);
  float tot[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int q = r0; q < r1; q += 16) {
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const int qe = min(r1, q + 16);
#pragma unroll 16
    for (int r = q; r < qe; ++r) {
      const i32x4 v = *(const i32x4*)(p.in + (int64_t)r * p.ld + c);
      const uint16_t* e = (const uint16_t*)&v;
#pragma unroll
      for (int j = 0; j < 8; ++j) s[j] += bf2f(e[j]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) tot[j] += s[j];
  }
  float* dst = p.partial + (int64_t)b * p.cols + c;
#pragma unroll
  for (int j = 0; j < 8; ++j) dst[j] = tot[j];
}

// stage 2: out[c] = sum_b partial[b][c], blocks ascending
__global__ __launch_bounds__(256) void colsum_final_kernel(ColSumParams p) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= p.cols) return;
  const int nb = (p.rows + kColSumChunk - 1) / kColSumChunk;
  float s = 0.0f;
  int b = 0;
  for (; b + 8 <= nb; b += 8) {   // eight loads in flight, added in block order
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = p.partial[(int64_t)(b + j) * p.cols + c];
#pragma unroll
    for (int j = 0; j < 8; ++j) s += v[j];
  }
  for (; b < nb; ++b) s += p.partial[(int64_t)b * p.cols + c];
  p.out[c] = s;
}

}  // namespace

static unsigned tile_grid(int rows, int cols) {
  const int64_t n = (int64_t)((rows + TT - 1) / TT) * ((cols + TT - 1) / TT);
  return n < (int64_t)1 << 31 ? (unsigned)n : 0u;
}

hipError_t launch_act_backward(const ActBwdParams& p, hipStream_t s) {
  if (p.rows == 0 || p.cols == 0) return hipSuccess;
  if (p.rows % 8 || p.cols % 8 || !tile_grid(p.rows, p.cols)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(act_backward_kernel, dim3(tile_grid(p.rows, p.cols)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_colsum(const ColSumParams& p, hipStream_t s) {
  if (p.cols == 0) return hipSuccess;
  if (p.cols % 8) return hipErrorInvalidValue;
  const int nb = (p.rows + kColSumChunk - 1) / kColSumChunk;
  const unsigned g8 = (unsigned)((p.cols / 8 + 255) / 256);
  if (g8 > 65535) return hipErrorInvalidValue;
  if (nb > 0 && !p.partial_ready)
    hipLaunchKernelGGL(colsum_partial_kernel, dim3((unsigned)nb, g8), dim3(256), 0, s, p);
  hipLaunchKernelGGL(colsum_final_kernel, dim3((unsigned)((p.cols + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace partir

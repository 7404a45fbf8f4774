// HBM-bound kernels: the ordered split-K reduction that stands in for the
// all_reduce of a #sum loop, and RMSNorm.
#include "kernels.h"
#include "device_math.h"

namespace partir {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// out[m][n] = epilogue(sum_{r = 0..R-1} partial[r][m][n]), r ascending, so the
// result does not depend on scheduling.  R = 0 is the empty sum (a contraction
// over K = 0): the output is the epilogue applied to zero.  One thread per 4
// columns.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(ReduceParams p) {
  const int nq = p.N >> 2;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.M * nq) return;
  const int m = (int)(idx / nq);
  const int n = (int)(idx - (int64_t)m * nq) * 4;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  if (p.R > 0) {
    const float* src = p.partial + (int64_t)m * p.part_ld + n;
    acc = *(const f32x4*)src;
    for (int r = 1; r < p.R; ++r) acc += *(const f32x4*)(src + r * p.part_stride);
  }
  if (p.bias) acc += *(const f32x4*)(p.bias + n);
  if (p.act) {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = gelu_erf(acc[e]);
  }
  if (p.resid_add) acc += *(const f32x4*)(p.resid + (int64_t)m * p.ldr + n);
  if (p.out_bf16) {
    bf16x4 o = {(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
    *(bf16x4*)((uint16_t*)p.C + (int64_t)m * p.ldc + n) = o;
  } else {
    *(f32x4*)((float*)p.C + (int64_t)m * p.ldc + n) = acc;
  }
}

// rows up to 256 * RMS_REG_CHUNKS wide are held in registers
constexpr int RMS_REG_CHUNKS = 24;

// One wave per row: fp32 sum of squares over D, then y = bf16(g * x * rstd).
// With parts, row r of x lives in the part r / rows_part (device-local arrays).
template <int PARTS>
__device__ __forceinline__ void rmsnorm_body(const RmsParams& p, const RmsParts* t) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= p.rows) return;
  const float* x = p.x + (int64_t)row * p.ldx;
  if (PARTS) {
    const int part = row / t->rows_part;
    x = t->x[part] + (int64_t)(row - part * t->rows_part) * p.ldx;
  }
  uint16_t* y = p.y + (int64_t)row * p.ldy;
  auto store = [&](int c, const f32x4& v, float rstd) {
    const f32x4 g = *(const f32x4*)(p.g + c);
    bf16x4 o = {(__bf16)(g[0] * (v[0] * rstd)), (__bf16)(g[1] * (v[1] * rstd)),
                (__bf16)(g[2] * (v[2] * rstd)), (__bf16)(g[3] * (v[3] * rstd))};
    *(bf16x4*)(y + c) = o;
  };
  auto rstd_of = [&](float ss) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
    return 1.0f / sqrtf(ss / (float)p.D + p.eps);
  };
  if (p.D <= 256 * RMS_REG_CHUNKS) {
    // the row stays in registers: every load issued before the first use,
    // one HBM read of x
    f32x4 v[RMS_REG_CHUNKS];
#pragma unroll
    for (int i = 0; i < RMS_REG_CHUNKS; ++i) {
      const int c = lane * 4 + 256 * i;
      v[i] = c < p.D ? *(const f32x4*)(x + c) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < RMS_REG_CHUNKS; ++i) ss += v[i][0] * v[i][0] + v[i][1] * v[i][1] + v[i][2] * v[i][2] + v[i][3] * v[i][3];
    const float rstd = rstd_of(ss);
#pragma unroll
    for (int i = 0; i < RMS_REG_CHUNKS; ++i) {
      const int c = lane * 4 + 256 * i;
      if (c < p.D) store(c, v[i], rstd);
    }
    return;
  }
  float ss = 0.0f;
  for (int c = lane * 4; c < p.D; c += 256) {
    const f32x4 v = *(const f32x4*)(x + c);
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  const float rstd = rstd_of(ss);
  for (int c = lane * 4; c < p.D; c += 256) store(c, *(const f32x4*)(x + c), rstd);
}

__global__ __launch_bounds__(256) void rmsnorm_kernel(RmsParams p) { rmsnorm_body<0>(p, nullptr); }
__global__ __launch_bounds__(256) void rmsnorm_parts_kernel(RmsParams p, RmsParts t) { rmsnorm_body<1>(p, &t); }

}  // namespace

hipError_t launch_splitk_reduce(const ReduceParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.M * (p.N / 4);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const RmsParams& p, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)((p.rows + 3) / 4)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_parts(const RmsParams& p, const RmsParts& t, hipStream_t s) {
  if (t.rows_part <= 0 || (p.rows + t.rows_part - 1) / t.rows_part > kMaxParts) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rmsnorm_parts_kernel, dim3((unsigned)((p.rows + 3) / 4)), dim3(256), 0, s, p, t);
  return hipGetLastError();
}

}  // namespace partir

// partir_loop_matmul_noalloc: partir_loop_matmul for callers that cannot
// allocate (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc).  The scratch the product needs -- the #sum's fp32
// partials [R][M][N] (split-K), or the K parts of a split last wave of output
// tiles -- lives in a file-scope device array of kScratchBytes instead of a
// caller workspace.  Every GPU the library runs on holds its own copy of the
// array until the process ends.
//
// Host code never passes the array's name to a kernel or a HIP call (in host
// code that name is a stand-in, not a device address): the device address is
// looked up once per device with hipGetSymbolAddress, with that device
// current, and that pointer is what the launches receive as their workspace.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/partir.h"

namespace partir {
void set_last_error(const std::string& msg);   // the C ABI's thread-local message
int validate_loop_matmul_call(const void* A, const void* B, void* C, int64_t M, int64_t N, int64_t K,
                              int64_t lda, int64_t ldb, int64_t ldc, int ab_dtype, int c_dtype, int b_layout,
                              int tile_axis, int sum_axis, int R, int sum_impl);
}

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;   // 64 MiB per device
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // device address of `scratch`, per device

int fail_with(int status, const std::string& msg) {
  partir::set_last_error(std::string(partir_status_string(status)) + ": " + msg);
  return status;
}

// The device address of `scratch` on the current device (looked up once).
int scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_with(PARTIR_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail_with(PARTIR_E_UNSUPPORTED, "device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail_with(PARTIR_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PARTIR_OK;
}

}  // namespace

extern "C" {

int partir_loop_matmul_noalloc(const void* A, const void* B, void* C, int64_t M, int64_t N, int64_t K,
                               int64_t lda, int64_t ldb, int64_t ldc, int ab_dtype, int c_dtype, int b_layout,
                               int tile_axis, int sum_axis, int R, int sum_impl, void* stream) {
  // argument errors first, before any device is touched
  int st = partir::validate_loop_matmul_call(A, B, C, M, N, K, lda, ldb, ldc, ab_dtype, c_dtype, b_layout, tile_axis,
                                             sum_axis, R, sum_impl);
  if (st) return st;
  // the scratch the call needs, from the same planner
  const size_t need = partir_loop_matmul_workspace(M, N, K, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R,
                                                   sum_impl);
  if (need == (size_t)-1) return fail_with(PARTIR_E_SHAPE, "arguments rejected by the workspace query");
  if (need > kScratchBytes)
    return fail_with(PARTIR_E_WORKSPACE, "the call needs " + std::to_string(need) +
                                             " bytes of scratch; partir_loop_matmul_noalloc holds " +
                                             std::to_string(kScratchBytes));
  if (need == 0)
    return partir_loop_matmul(A, B, C, M, N, K, lda, ldb, ldc, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R,
                              sum_impl, nullptr, 0, stream);
  void* ws = nullptr;
  if ((st = scratch_on_current_device(&ws))) return st;
  return partir_loop_matmul(A, B, C, M, N, K, lda, ldb, ldc, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R,
                            sum_impl, ws, kScratchBytes, stream);
}

}  // extern "C"

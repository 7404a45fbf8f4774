// Device helpers shared by the kernels that stream tiles into LDS with
// direct-to-LDS buffer loads (bf16 GEMM, attention forward and backward).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace partir {

typedef short lds_i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) lds_i16x4_t lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;

// Buffer descriptor of a workgroup-uniform base pointer (kept in SGPRs); an
// offset at or beyond `bytes` reads as zero (and writes LDS zeros when the
// load targets LDS).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void* u = (void*)(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(u, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

// ds_read_b64_tr_b16 through a restrict pointer: the alias scope this gives
// the read keeps the compiler's wait insertion from making it wait for every
// LDS DMA in flight (the callers order their LDS stages by explicit vmcnt
// waits and barriers).
__device__ __forceinline__ lds_i16x4_t lds_read_tr16(const char* __restrict__ p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
}

}  // namespace partir

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding)
#define WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) & 15) | (((n) >> 4) << 14)) | (0x7 << 4) | (0xF << 8))

// Vector memory reads through buffer resources (gfx9 family).
//
// A buffer resource describes [base, base + bytes) in four scalar registers;
// a load whose offset falls outside it returns zero. Kernels use this to
// read with branch-free code: a lane whose element lies outside the operand
// passes kOutOfRange instead of being masked off.
#pragma once

#include <hip/hip_runtime.h>

namespace oaa {

constexpr unsigned kOutOfRange = 0x80000000u;

// Resource over `bytes` (< 2^31) bytes at base. base and bytes must be the
// same in every lane; reading them through the first lane tells the compiler
// so and keeps the resource in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_resource(const void* base, unsigned bytes) {
  const unsigned long long a = reinterpret_cast<unsigned long long>(base);
  const unsigned lo = __builtin_amdgcn_readfirstlane(unsigned(a));
  const unsigned hi = __builtin_amdgcn_readfirstlane(unsigned(a >> 32));
  void* pu = reinterpret_cast<void*>((static_cast<unsigned long long>(hi) << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(pu, short(0), int(__builtin_amdgcn_readfirstlane(bytes)), 0x00020000);
}

__device__ __forceinline__ float buffer_load_f1(__amdgpu_buffer_rsrc_t rs, unsigned byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, byte_off, 0, 0));
}

__device__ __forceinline__ float2 buffer_load_f2(__amdgpu_buffer_rsrc_t rs, unsigned byte_off) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(rs, byte_off, 0, 0));
}

}  // namespace oaa

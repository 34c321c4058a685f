// Small device-side helpers shared by the HIP sources of the library
// (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sn_dev {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte chunk
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));   // MFMA bf16 operand of one lane
typedef float f32x4 __attribute__((ext_vector_type(4)));     // 16 x 16 MFMA accumulator of one lane

constexpr int kRsrcWord3 = 0x00020000;  // buffer descriptor word 3 for gfx9-family raw loads

// Values that every lane of a wave computes identically are moved to scalar
// registers explicitly: the compiler cannot prove a load from writable memory
// wave-uniform, and a buffer descriptor it believes divergent forces a loop
// around every buffer load.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ float uni(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x)));
}
__device__ __forceinline__ const char* uni(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return reinterpret_cast<const char*>(((uint64_t)hi << 32) | lo);
}

// Buffer resource over [base, base + bytes); the hardware range check returns
// zeros for a 16-byte load that does not lie wholly inside.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

}  // namespace sn_dev

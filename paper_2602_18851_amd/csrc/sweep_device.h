// Device helpers shared by the sweep kernels (sweeps.hip, layer_form.hip,
// gram.hip): element access of 16-byte chunks, lane and wave reductions.
#pragma once

#include "device_util.h"
#include "kernels.h"

namespace sn {

using namespace sn_dev;

template <typename T>
struct Traits;
template <>
struct Traits<float> {
  static constexpr int VEC = 4;
};
template <>
struct Traits<uint16_t> {  // bf16 bit patterns
  static constexpr int VEC = 8;
};


template <typename T>
__device__ __forceinline__ float elem(const u32x4& q, int c);
template <>
__device__ __forceinline__ float elem<float>(const u32x4& q, int c) {
  return __uint_as_float(q[c]);
}
template <>
__device__ __forceinline__ float elem<uint16_t>(const u32x4& q, int c) {
  const uint32_t w = q[c >> 1];
  return __uint_as_float((c & 1) ? (w & 0xffff0000u) : (w << 16));
}

// Marks a chunk as redefined so the compiler re-derives its float values for
// the second product instead of keeping all of them live across the lane
// shuffles (that would double the register footprint of a tile).
__device__ __forceinline__ void reuse_fence(u32x4& q) { asm volatile("" : "+v"(q)); }

__device__ __forceinline__ float xor_sum(float x, int m) { return x + __shfl_xor(x, m); }

// Sum over the 64 lanes of a wave (butterfly: every lane gets the same bits).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

// Occupancy floor per SIMD: the accumulators grow with GC * DH / 8 floats.
template <int DH, int GC>
constexpr int waves_hint() {
  return GC * DH / kRG >= 128 ? 2 : GC * DH / kRG >= 64 ? 3 : 4;
}

// Sum over the 8 row groups of a wave tile (lanes that share lane mod 8):
// the step inside a 16-lane row is a DPP row rotation by 8 fused into the
// add; the steps across rows are lane shuffles.  Every lane ends with the
// same total for its column.
__device__ __forceinline__ float group_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x128, 0xF, 0xF, false));
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}


// Sum of one value per wave, in wave order.
template <int NW>
__device__ __forceinline__ float sum_waves(const float* red) {
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) s += red[w];
  return s;
}

}  // namespace sn

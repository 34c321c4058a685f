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

// ---- wave-private staging of row tiles through LDS ----------------------
//
// A tile is R rows x 128 bytes.  It is loaded with buffer_load ... lds, which
// writes lane i's 16 bytes to LDS at base + 16 i: instruction j covers rows
// 8 j .. 8 j + 7, eight consecutive lanes reading one 128-byte row segment
// (a coalesced request for the address unit).  In LDS, row r holds its eight
// 16-byte chunks at physical slot c ^ swz(r), swz(r) = (r / 2 mod 8) ^
// (r / 16 mod 2): the row pairs of a 16-row group take eight different
// slots for any one chunk, and the next 16-row group the same slots in
// swapped pairs.  Measured on gfx950 (eight waves per CU, 16-byte reads):
//   - the MFMA operand read of one chunk from 16 rows (lane s: row r0 + s,
//     four chunks per instruction) moves ~460 GB/s per CU with this swizzle,
//     against ~290 GB/s when the slot depends on the row pair alone through
//     a permutation that mixes its bits;
//   - the 32-row, two-chunk pattern moves ~465 GB/s per CU.
// swz has period 32 in r, so a tile row keeps its slot whether the rows are
// counted from the tile or from a 32-row part of it (the projection stages
// each wave's 32 rows from its own base).
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ int stage_swz(int r) { return ((r >> 1) & 7) ^ ((r >> 4) & 1); }

// Issues the loads of one tile: row r of the resource starts at byte
// r * row_bytes; the tile takes columns [col_byte, col_byte + 128).  AUX is the
// cache policy of the loads.
template <int R, int AUX>
__device__ __forceinline__ void stage_issue(__amdgpu_buffer_rsrc_t rsrc, uint8_t* lds, uint32_t col_byte,
                                            uint32_t row_bytes, int lane) {
  const int sr = lane >> 3, p = lane & 7;
#pragma unroll
  for (int j = 0; j < R / 8; ++j) {
    const int r = 8 * j + sr;
    const uint32_t voff = (uint32_t)sr * row_bytes + col_byte + 16u * (uint32_t)(p ^ stage_swz(r));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)(lds + 1024 * j), 16, voff, 8u * j * row_bytes, 0,
                                             AUX);
  }
}

// Logical 16-byte chunk c (0..7) of row r of a staged tile.
__device__ __forceinline__ u32x4 stage_chunk(const uint8_t* lds, int r, int c) {
  return *reinterpret_cast<const u32x4*>(lds + 128 * r + 16 * (c ^ stage_swz(r)));
}

}  // namespace sn_dev

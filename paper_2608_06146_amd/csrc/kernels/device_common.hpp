// Small device helpers shared by the kernels of this library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../schedule.hpp"

namespace padoc {

constexpr float kLn2 = 0.693147180559945309f;

// Device address of key `j` of a range for KV head `kvh` (element offset).
// Packed K/V: [T, Hkv, D] rows; paged: [blocks, Hkv, 16, D] with the block
// taken from the block table.
template <int D, bool PAGED>
__device__ __forceinline__ int64_t key_offset(const RangeRec& r, int32_t j, int32_t kvh, int32_t Hkv,
                                              const int32_t* __restrict__ block_table) {
  if constexpr (PAGED) {
    const int64_t blk = block_table[r.kv_start + (j >> 4)];
    return ((blk * Hkv + kvh) * kBlock + (j & 15)) * (int64_t)D;
  } else {
    return ((r.kv_start + j) * Hkv + kvh) * (int64_t)D;
  }
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Round-to-nearest-even fp32 -> bf16 bits (inputs here are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

}  // namespace padoc

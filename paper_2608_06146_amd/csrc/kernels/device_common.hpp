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

// Zero the bf16 elements at positions >= keep of an 8-element (16-byte)
// chunk; keep may be <= 0 (all zero) or >= 8 (unchanged).
__device__ __forceinline__ uint4 keep_first(uint4 u, int keep) {
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lo = 2 * i;
    const uint32_t m = (lo + 1 < keep) ? 0xffffffffu : (lo < keep ? 0x0000ffffu : 0u);
    w[i] &= m;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

}  // namespace padoc

// Helpers shared by the bf16 matrix-core kernels (the forward / decode work
// item in fwd_item.hpp and the backward in bwd.hip): vector types, the
// workgroup shape, wave-uniform values, the paired transposing LDS read and
// a compile-time loop.
#pragma once

#include <type_traits>

#include "device_common.hpp"

namespace padoc {
namespace tile {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr float kRescaleSlack = 8.0f;  // log2 units: probabilities <= 2^8

__device__ __forceinline__ int64_t uniform64(int64_t x) {
  return (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(x >> 32)) << 32) |
                   (uint32_t)__builtin_amdgcn_readfirstlane((int)x));
}

__device__ __forceinline__ RangeRec uniform_range(RangeRec r) {
  r.kv_start = uniform64(r.kv_start);
  r.n_keys = __builtin_amdgcn_readfirstlane(r.n_keys);
  r.min_lim = __builtin_amdgcn_readfirstlane(r.min_lim);
  r.lim_off = __builtin_amdgcn_readfirstlane(r.lim_off);
  return r;
}

// Two transposing LDS reads (4 bf16 each) joined into one 8-element MFMA
// operand: elements 0-3 from the read at lo, 4-7 from the read at hi.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8_t tr_pair(const uint16_t* lo, const uint16_t* hi) {
  typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
  const i16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(const_cast<uint16_t*>(lo)));
  const i16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(const_cast<uint16_t*>(hi)));
  const short __attribute__((ext_vector_type(8))) ab = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8_t, ab);
}

// f(integral_constant<int, i>) for i = 0 .. N-1: constant indices into
// register arrays, so they stay registers (a loop index that is still a
// variable when the optimizer first looks would place them in scratch
// memory).
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

}  // namespace tile
}  // namespace padoc

// Small device helpers shared by the kernels of this library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../schedule.hpp"

namespace padoc {

constexpr float kLn2 = 0.693147180559945309f;

// Paged K blocks are chunk-major, [Hkv][D/8][16 slots][8]: token t of a
// block lives in slot kslot(t) (bits 2 and 3 of t swapped), so one 8-dim
// chunk of the tokens {0-3, 8-11} (or {4-7, 12-15}) is one 128-byte line.
// kslot is its own inverse.
__device__ __forceinline__ int kslot(int t) { return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1); }

// Element offset of dims [8c, 8c+8) of token t (0..15) in paged K block blk
// for KV head kvh.
template <int D>
__device__ __forceinline__ int64_t paged_k_offset(int64_t blk, int32_t kvh, int32_t Hkv, int t, int c) {
  return ((blk * Hkv + kvh) * (D / 8) + c) * (kBlock * 8) + kslot(t) * 8;
}

// 16-byte load with the non-temporal hint: for K/V that a kernel reads once
// (paged decode), so the caches do not keep lines nobody will read again.
__device__ __forceinline__ uint4 load_stream16(const void* p) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 t = __builtin_nontemporal_load(static_cast<const u32x4*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}

// Plain 16-byte load and store as one vector value (a uint4 struct copy
// would become a memory-to-memory copy through a stack slot).
__device__ __forceinline__ uint4 load16(const void* p) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 t = *static_cast<const u32x4*>(p);
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void store16(void* p, const uint4& v) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  *static_cast<u32x4*>(p) = u32x4{v.x, v.y, v.z, v.w};
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Load of a wave-uniform value through the scalar data cache (s_load).  The
// address must be the same in every lane (it is made so) and the memory
// read-only while the kernel runs.  Scalar loads are counted by lgkmcnt, not
// vmcnt: waiting for one does not wait for the vector loads in flight.
template <class T>
__device__ __forceinline__ T load_scalar(const T* p) {
  static_assert(sizeof(T) % 4 == 0, "scalar loads move whole dwords");
  typedef const __attribute__((address_space(4))) uint32_t* cptr;
  const uint64_t a = (uint64_t)p;
  const uint64_t u = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(a >> 32)) << 32) |
                     (uint32_t)__builtin_amdgcn_readfirstlane((int)a);
  const cptr q = (cptr)u;
  uint32_t w[sizeof(T) / 4];
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) w[i] = q[i];
  T r;
  __builtin_memcpy(&r, w, sizeof(T));
  return r;
}

// max(a, b, c) as one v_max3_f32.  Written as an instruction so the compiler
// does not first canonicalise each operand (it cannot prove that values
// merged from masked and unmasked paths are canonical); inputs here are
// finite or -inf.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Maximum of x over lanes l and l^32 (in every lane): v_permlane32_swap of
// two copies leaves one holding the low half's values in both halves and the
// other the high half's.
__device__ __forceinline__ float max_lane_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max3f(x, __uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Maximum of x over lanes l and l^16 (rows of 16 lanes): v_permlane16_swap
// of two copies pairs each row with its neighbour.
__device__ __forceinline__ float max_lane_rows(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max3f(x, __uint_as_float(r[0]), __uint_as_float(r[1]));
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + x.lo + x.hi for two bf16 values (one v_dot2c_f32_bf16 against 1.0).
__device__ __forceinline__ float add_bf16x2(bf16x2_t x, float acc) {
  const bf16x2_t one = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(x, one, acc, false);
}

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

// Merge of split-KV partial results (decode path).
//
// Softmax attention over a union of disjoint key sets is recovered exactly
// from each set's running max m_i (log2 units), sum l_i and unnormalised
// accumulator o_i (App. E Attn equation, associativity of the normaliser):
//   M = max m_i;  L = sum l_i 2^(m_i - M);  O = sum o_i 2^(m_i - M) / L;
//   LSE = (M + log2 L) ln 2.
// Partials are read in the planner's fixed order, so results are bitwise
// reproducible.  32 threads per (query row, head), 8 per block, over the
// (row, KV head) pairs the plan lists.
#include "device_common.hpp"

namespace padoc {

template <int D, bool BF16>
__global__ __launch_bounds__(256) void lse_combine_kernel(CombineParams p) {
  constexpr int PER = D / 32;
  const int64_t pair = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  const int sub = threadIdx.x & 31;
  if (pair >= p.n_rows * p.G) return;
  const int64_t rk = p.comb_rows[pair / p.G];
  const int h = (int)(pair % p.G);
  const int64_t row = rk / p.Hkv;
  const int g = (int)(rk - row * p.Hkv);
  const int hq = g * p.G + h;
  const int32_t e0 = p.comb_ptr[rk];
  const int32_t e1 = p.comb_ptr[rk + 1];
  if (e0 == e1) return;
  float M = -INFINITY;
  for (int32_t e = e0; e < e1; ++e) M = fmaxf(M, p.part_ml[2 * (int64_t)(p.comb_slot[e] + h)]);
  float L = 0.f;
  float o[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) o[k] = 0.f;
  for (int32_t e = e0; e < e1; ++e) {
    const int64_t slot = p.comb_slot[e] + h;
    const float sc = fast_exp2(p.part_ml[2 * slot] - M);
    L = fmaf(p.part_ml[2 * slot + 1], sc, L);
    const float* src = p.part_o + slot * D + sub * PER;
    if constexpr (PER == 4) {
      const float4 x = *reinterpret_cast<const float4*>(src);
      o[0] = fmaf(x.x, sc, o[0]);
      o[1] = fmaf(x.y, sc, o[1]);
      o[2] = fmaf(x.z, sc, o[2]);
      o[3] = fmaf(x.w, sc, o[3]);
    } else {
      const float2 x = *reinterpret_cast<const float2*>(src);
      o[0] = fmaf(x.x, sc, o[0]);
      o[1] = fmaf(x.y, sc, o[1]);
    }
  }
  const float inv = 1.f / L;
  const int64_t base = (row * p.Hq + hq) * D + sub * PER;
  if constexpr (BF16) {
    uint16_t* dst = static_cast<uint16_t*>(p.o) + base;
    if constexpr (PER == 4) {
      uint2 pk;
      pk.x = (uint32_t)f32_to_bf16_bits(o[0] * inv) | ((uint32_t)f32_to_bf16_bits(o[1] * inv) << 16);
      pk.y = (uint32_t)f32_to_bf16_bits(o[2] * inv) | ((uint32_t)f32_to_bf16_bits(o[3] * inv) << 16);
      *reinterpret_cast<uint2*>(dst) = pk;
    } else {
      *reinterpret_cast<uint32_t*>(dst) =
          (uint32_t)f32_to_bf16_bits(o[0] * inv) | ((uint32_t)f32_to_bf16_bits(o[1] * inv) << 16);
    }
  } else {
    float* dst = static_cast<float*>(p.o) + base;
#pragma unroll
    for (int k = 0; k < PER; ++k) dst[k] = o[k] * inv;
  }
  if (sub == 0) p.lse[row * p.Hq + hq] = (M + __log2f(L)) * kLn2;
}

hipError_t launch_lse_combine(const CombineParams& p, int D, bool bf16, hipStream_t stream) {
  const int64_t pairs = p.n_rows * p.G;
  if (pairs == 0) return hipSuccess;
  const dim3 grid((unsigned)((pairs + 7) / 8)), block(256);
  if (D == 64) {
    if (bf16) hipLaunchKernelGGL((lse_combine_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((lse_combine_kernel<64, false>), grid, block, 0, stream, p);
  } else {
    if (bf16) hipLaunchKernelGGL((lse_combine_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((lse_combine_kernel<128, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace padoc

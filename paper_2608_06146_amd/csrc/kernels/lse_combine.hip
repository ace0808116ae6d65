// Merge of split-KV partial results (decode path).
//
// Softmax attention over a union of disjoint key sets is recovered exactly
// from each set's running max m_i (log2 units), sum l_i and unnormalised
// accumulator o_i (App. E Attn equation, associativity of the normaliser):
//   M = max m_i;  L = sum l_i 2^(m_i - M);  O = sum o_i 2^(m_i - M) / L;
//   LSE = (M + log2 L) ln 2.
// LANES threads per (query row, head), each with D/LANES elements, 256 /
// LANES pairs per block, over the (row, KV head) pairs the plan lists: 8
// lanes (four independent 16-byte loads per partial at D = 128) when there
// are enough pairs to fill the chip, else 32 (more threads to cover the
// loads' latency in a small step).
//
// The partials of a pair are taken in batches of LANES: lane j of the group
// fetches partial j's slot, m and l (independent loads), the batch maximum
// and weighted sum come from butterfly reductions over the group, and the
// O rows are then summed in the planner's order with the weights passed by
// shuffles, so their loads do not wait on each other.  Reductions and sums
// run in a fixed order: results are bitwise reproducible.
#include "device_common.hpp"

namespace padoc {

template <int N>
struct VecF;  // N consecutive floats as one load / store
template <>
struct VecF<2> {
  typedef float2 T;
};
template <>
struct VecF<4> {
  typedef float4 T;
};

template <int D, bool BF16, int LANES>
__global__ __launch_bounds__(256) void lse_combine_kernel(CombineParams p) {
  constexpr int PER = D / LANES;                // elements per thread
  constexpr int VW = PER >= 4 ? 4 : PER;        // floats per vector load
  constexpr int NV = PER / VW;                  // vector loads per partial
  constexpr int U = NV > 1 ? 2 : 8;             // partials whose loads are in flight together
  typedef typename VecF<VW>::T vec_t;
  const int64_t pair = (int64_t)blockIdx.x * (256 / LANES) + (threadIdx.x / LANES);
  const int sub = threadIdx.x % LANES;
  // The step kernel before this one on the stream has taken every private
  // item: its queue counters go back to zero, so a workspace that keeps its
  // schedule is ready for the next call without a new upload.
  if (p.next != nullptr && blockIdx.x == 0 && threadIdx.x < kPrivateQueues) p.next[64 * threadIdx.x] = 0;
  if (pair >= p.n_rows * p.G) return;
  const int4 rec = p.comb_rows[pair / p.G];  // one load: the pair and its slot list
  const int64_t rk = rec.x;
  const int h = (int)(pair % p.G);
  const int64_t row = rk / p.Hkv;
  const int g = (int)(rk - row * p.Hkv);
  const int hq = g * p.G + h;
  const int32_t e0 = rec.y;
  const int32_t e1 = rec.z;
  if (e0 == e1) return;
  const float2* ml = reinterpret_cast<const float2*>(p.part_ml);
  float M = -INFINITY, L = 0.f;
  float o[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) o[k] = 0.f;
  for (int32_t b = e0; b < e1; b += LANES) {
    const int cnt = e1 - b < LANES ? (int)(e1 - b) : LANES;
    int32_t slot = 0;
    float m = -INFINITY, l = 0.f;
    if (sub < cnt) {
      slot = p.comb_slot[b + sub] + h;
      const float2 v = ml[slot];
      m = v.x;
      l = v.y;
    }
    float mb = m;
#pragma unroll
    for (int s = 1; s < LANES; s <<= 1) mb = fmaxf(mb, __shfl_xor(mb, s, LANES));
    const float Mn = fmaxf(M, mb);
    const float alpha = M == -INFINITY ? 0.f : fast_exp2(M - Mn);
    // a partial whose keys were all masked (m = -inf) weighs nothing, also
    // while every partial so far is such a one (Mn = -inf)
    const float sc = m == -INFINITY ? 0.f : fast_exp2(m - Mn);
    float lb = l * sc;
#pragma unroll
    for (int s = 1; s < LANES; s <<= 1) lb += __shfl_xor(lb, s, LANES);
    L = fmaf(L, alpha, lb);
    M = Mn;
#pragma unroll
    for (int k = 0; k < PER; ++k) o[k] *= alpha;
    // U partials per round: all their loads are issued before the first
    // product (a partial past the batch re-reads the last one and is skipped)
    for (int j0 = 0; j0 < cnt; j0 += U) {
      float x[U][PER];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u < cnt ? j0 + u : cnt - 1;
        const int32_t sj = __shfl(slot, j, LANES);
        const vec_t* src = reinterpret_cast<const vec_t*>(p.part_o + (int64_t)sj * D + sub * PER);
#pragma unroll
        for (int k = 0; k < NV; ++k) *reinterpret_cast<vec_t*>(&x[u][VW * k]) = src[k];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (j0 + u < cnt) {
          const float cj = __shfl(sc, j0 + u, LANES);
#pragma unroll
          for (int k = 0; k < PER; ++k) o[k] = fmaf(x[u][k], cj, o[k]);
        }
      }
    }
  }
  const float inv = 1.f / L;
  const int64_t base = (row * p.Hq + hq) * D + sub * PER;
  if constexpr (BF16) {
    uint32_t w[PER / 2];
#pragma unroll
    for (int k = 0; k < PER / 2; ++k)
      w[k] = (uint32_t)f32_to_bf16_bits(o[2 * k] * inv) | ((uint32_t)f32_to_bf16_bits(o[2 * k + 1] * inv) << 16);
    uint32_t* dst = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(p.o) + base);
    if constexpr (PER >= 8) {
#pragma unroll
      for (int k = 0; k < PER / 8; ++k) reinterpret_cast<uint4*>(dst)[k] = make_uint4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
    } else if constexpr (PER == 4) {
      *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
    } else {
      dst[0] = w[0];
    }
  } else {
    float* dst = static_cast<float*>(p.o) + base;
#pragma unroll
    for (int k = 0; k < PER; ++k) o[k] *= inv;
#pragma unroll
    for (int k = 0; k < NV; ++k) reinterpret_cast<vec_t*>(dst)[k] = *reinterpret_cast<const vec_t*>(&o[VW * k]);
  }
  if (sub == 0) p.lse[row * p.Hq + hq] = (M + __log2f(L)) * kLn2;
}

template <int D, bool BF16>
void launch_d(const CombineParams& p, int64_t pairs, hipStream_t stream) {
  // 8 lanes per pair once the pairs fill 256 compute units x 8 wavefronts
  if (pairs >= 256 * 8 * 64 / 8) {
    const dim3 grid((unsigned)((pairs + 31) / 32)), block(256);
    hipLaunchKernelGGL((lse_combine_kernel<D, BF16, 8>), grid, block, 0, stream, p);
  } else {
    const dim3 grid((unsigned)((pairs + 7) / 8)), block(256);
    hipLaunchKernelGGL((lse_combine_kernel<D, BF16, 32>), grid, block, 0, stream, p);
  }
}

hipError_t launch_lse_combine(const CombineParams& p, int D, bool bf16, hipStream_t stream) {
  const int64_t pairs = p.n_rows * p.G;
  if (pairs == 0) return hipSuccess;
  if (D == 64) {
    if (bf16) launch_d<64, true>(p, pairs, stream);
    else launch_d<64, false>(p, pairs, stream);
  } else {
    if (bf16) launch_d<128, true>(p, pairs, stream);
    else launch_d<128, false>(p, pairs, stream);
  }
  return hipGetLastError();
}

}  // namespace padoc

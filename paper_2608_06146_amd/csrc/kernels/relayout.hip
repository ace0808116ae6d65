// Paged K/V blocks in row layout ([block][KV head][16 slots][d], the layout a
// cache that stores each token's row contiguously uses) rewritten into the
// library's paged layouts, so a caller holding such a cache can run the
// decode step (App. E: the step attends over the cached rows of every
// stream; where a row lives is a storage choice).
//
//   K: [block][head][d/8][16][8], token t of a block in slot kslot(t) (bits
//      2 and 3 of t exchanged): thread (block, head, t, piece c) copies the
//      8 dims 8c .. 8c+7 of row t, one 16-byte (bf16) or 32-byte (fp32) run
//      on both sides.
//   V: [block][head][d][16]: workgroup (block, head) reads the 16 rows
//      contiguously into LDS and writes the 16 tokens of each dim d as one
//      run (a 16 x d transpose per block and head).
// A copy: 2 * 16 * Hkv * d elements read and written per block.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>

namespace padoc {
namespace {

constexpr int kSlots = 16;

__device__ __forceinline__ int kslot(int t) { return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1); }

template <typename T>
__global__ __launch_bounds__(256) void relayout_k_kernel(const T* __restrict__ src, T* __restrict__ dst,
                                                         int64_t n_pieces, int D) {
  // piece index = ((block * Hkv + head) * 16 + t) * (D/8) + c
  const int P = D / 8;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_pieces; i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % P);
    const int64_t rt = i / P;  // (block * Hkv + head) * 16 + t
    const int t = (int)(rt % kSlots);
    const int64_t bh = rt / kSlots;
    const T* s = src + (bh * kSlots + t) * D + 8 * c;
    T* d = dst + ((bh * P + c) * kSlots + kslot(t)) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) d[e] = s[e];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void relayout_v_kernel(const T* __restrict__ src, T* __restrict__ dst,
                                                         int64_t n_bh, int D) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);  // [16][D]
  for (int64_t bh = blockIdx.x; bh < n_bh; bh += gridDim.x) {
    const T* s = src + bh * kSlots * D;
    for (int i = threadIdx.x; i < kSlots * D; i += blockDim.x) tile[i] = s[i];
    __syncthreads();
    T* d = dst + bh * (int64_t)D * kSlots;
    for (int i = threadIdx.x; i < kSlots * D; i += blockDim.x) {
      const int dim = i / kSlots, t = i % kSlots;
      d[i] = tile[t * D + dim];
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_relayout_kv(const void* k_rows, const void* v_rows, void* k_cache, void* v_cache, int64_t n_blocks,
                              int Hkv, int D, int elem_bytes, hipStream_t stream) {
  if (n_blocks <= 0) return hipSuccess;
  const int64_t n_bh = n_blocks * Hkv;
  const int64_t n_pieces = n_bh * kSlots * (D / 8);
  const dim3 kgrid((unsigned)std::min<int64_t>((n_pieces + 255) / 256, 65536)), blk(256);
  const dim3 vgrid((unsigned)std::min<int64_t>(n_bh, 65536));
  const size_t lds = (size_t)kSlots * D * elem_bytes;
  if (elem_bytes == 2) {
    hipLaunchKernelGGL(relayout_k_kernel<uint16_t>, kgrid, blk, 0, stream, static_cast<const uint16_t*>(k_rows),
                       static_cast<uint16_t*>(k_cache), n_pieces, D);
    hipLaunchKernelGGL(relayout_v_kernel<uint16_t>, vgrid, blk, lds, stream, static_cast<const uint16_t*>(v_rows),
                       static_cast<uint16_t*>(v_cache), n_bh, D);
  } else {
    hipLaunchKernelGGL(relayout_k_kernel<float>, kgrid, blk, 0, stream, static_cast<const float*>(k_rows),
                       static_cast<float*>(k_cache), n_pieces, D);
    hipLaunchKernelGGL(relayout_v_kernel<float>, vgrid, blk, lds, stream, static_cast<const float*>(v_rows),
                       static_cast<float*>(v_cache), n_bh, D);
  }
  return hipGetLastError();
}

}  // namespace padoc

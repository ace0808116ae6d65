// Append of a decode step's new K/V rows into the paged caches (App. E, the
// "append" of masked parallel decoding: one new input per live stream), and
// the block-table entries of the step's new or moved blocks.
//
// One 64-lane workgroup per (new row, KV head): lane c copies dims c, c+64
// of K into the chunk-major K cache (dims c..c+7 of a token form one
// contiguous 8-element piece, so the lanes of a piece store to adjacent
// addresses) and of V into the d-major V cache (a 2- or 4-byte store per dim
// at a 16-element stride: the step adds one token per block, so there is no
// wider contiguous run to store).  Workgroups past the rows write the
// block-table patches.  The kernel is a copy: 2 * Hkv * d elements read and
// written per row.
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace padoc {
namespace {

template <typename T>
__global__ __launch_bounds__(64) void append_kv_kernel(const T* __restrict__ k_new, const T* __restrict__ v_new,
                                                       T* __restrict__ k_cache, T* __restrict__ v_cache,
                                                       const int32_t* __restrict__ slots, int64_t n_items, int Hkv,
                                                       int D, const int32_t* __restrict__ patch, int64_t n_patch,
                                                       int32_t* __restrict__ block_table) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  if (b < n_items) {
    const int64_t row = b / Hkv;
    const int h = (int)(b - row * Hkv);
    const int32_t blk = slots[2 * row];
    const int32_t t = slots[2 * row + 1];
    const int kslot = (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1);
    const size_t base = ((size_t)blk * Hkv + h) * (size_t)D * 16;
    const T* ks = k_new + (size_t)b * D;
    const T* vs = v_new + (size_t)b * D;
    for (int c = lane; c < D; c += 64) {
      k_cache[base + (size_t)(((c >> 3) * 16 + kslot) * 8 + (c & 7))] = ks[c];
      v_cache[base + (size_t)c * 16 + t] = vs[c];
    }
  } else {
    const int64_t i = (b - n_items) * 64 + lane;
    if (i < n_patch) block_table[patch[2 * i]] = patch[2 * i + 1];
  }
}

}  // namespace

// slots: (block id, slot) per new row, ids < the pool size; patch:
// (table entry, block id) pairs inside the table.  Both were produced by the
// session on the host, which checked them.
hipError_t launch_append_kv(const void* k_new, const void* v_new, void* k_cache, void* v_cache, const int32_t* slots,
                            int64_t n_rows, int Hkv, int D, bool bf16, const int32_t* patch, int64_t n_patch,
                            int32_t* block_table, hipStream_t s) {
  const int64_t items = n_rows * Hkv;
  const int64_t blocks = items + (n_patch + 63) / 64;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  if (bf16)
    hipLaunchKernelGGL(append_kv_kernel<uint16_t>, dim3((unsigned)blocks), dim3(64), 0, s,
                       static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), slots, items, Hkv, D, patch,
                       n_patch, block_table);
  else
    hipLaunchKernelGGL(append_kv_kernel<uint32_t>, dim3((unsigned)blocks), dim3(64), 0, s,
                       static_cast<const uint32_t*>(k_new), static_cast<const uint32_t*>(v_new),
                       static_cast<uint32_t*>(k_cache), static_cast<uint32_t*>(v_cache), slots, items, Hkv, D, patch,
                       n_patch, block_table);
  return hipGetLastError();
}

}  // namespace padoc

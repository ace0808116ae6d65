// bf16 packed forward: one 8-wavefront workgroup per work item (packed K/V,
// final O and LSE); the computation is fwd_item.  The paged form of the tile
// computation (shared keys of a decode step) runs inside
// decode_step_kernel.
#include "fwd_item.hpp"

namespace padoc {

namespace {

template <int D>
__global__ __launch_bounds__(tile::kThreads) void tile_mfma_bf16_kernel(TileParams p) {
  tile::fwd_item<D, false>(p, blockIdx.x);
}

}  // namespace

hipError_t launch_tile_mfma_bf16(const TileParams& p, int n_work, int D, hipStream_t stream) {
  if (n_work <= 0) return hipSuccess;
  const dim3 grid(n_work), block(tile::kThreads);
  if (D == 64)
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<64>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<128>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace padoc

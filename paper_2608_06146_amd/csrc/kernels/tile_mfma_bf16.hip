// bf16 tile kernel of the packed forward: one 8-wavefront workgroup per work
// item (packed K/V, final O and LSE).  The computation is tile_item; its paged
// form (shared keys of a decode step) runs inside decode_step_kernel.
#include "tile_item.hpp"

namespace padoc {

namespace {

template <int D, bool PAGED, bool PARTIAL>
__global__ __launch_bounds__(tile::kThreads) void tile_mfma_bf16_kernel(TileParams p) {
  tile::tile_item<D, PAGED, PARTIAL>(p, blockIdx.x);
}

}  // namespace

hipError_t launch_tile_mfma_bf16(const TileParams& p, int n_work, int D, hipStream_t stream) {
  if (n_work <= 0) return hipSuccess;
  const dim3 grid(n_work), block(tile::kThreads);
  if (D == 64)
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<64, false, false>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<128, false, false>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace padoc

// bf16 tile kernels: one 8-wavefront workgroup per work item, for the packed
// forward (packed K/V, final O and LSE) and for the shared keys of a decode
// step (paged K/V, split partials).  The computation is tile_item.
#include "tile_item.hpp"

namespace padoc {

namespace {

template <int D, bool PAGED, bool PARTIAL>
__global__ __launch_bounds__(tile::kThreads) void tile_mfma_bf16_kernel(TileParams p) {
  tile::tile_item<D, PAGED, PARTIAL>(p, blockIdx.x);
}

template <int D>
void launch_d(const TileParams& p, dim3 grid, bool paged, hipStream_t stream) {
  const dim3 block(tile::kThreads);
  if (paged)
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<D, true, true>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<D, false, false>), grid, block, 0, stream, p);
}

}  // namespace

hipError_t launch_tile_mfma_bf16(const TileParams& p, int n_work, int D, bool paged, hipStream_t stream) {
  if (n_work <= 0) return hipSuccess;
  if (D == 64)
    launch_d<64>(p, dim3(n_work), paged, stream);
  else
    launch_d<128>(p, dim3(n_work), paged, stream);
  return hipGetLastError();
}

}  // namespace padoc

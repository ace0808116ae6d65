// fp32 tile kernel: one thread per (query token, head) column of a work item,
// keys visited one by one with an exact online softmax in fp32 on the vector
// ALUs.  This is the fp32 path of both entry points (the MFMA paths are
// bf16); it reads the same schedules as the bf16 kernels, one workgroup per
// work item (columns col0 .. col0+ncol-1 of the item's task), over packed
// K/V or the paged cache (K blocks chunk-major [d/8][16 slots][8], V blocks
// d-major [d][16]).
//
// Per column and visible key j (App. E Attn equation, with the scale applied
// in log2 units): s = scale*log2(e) * q.k_j; m' = max(m, s);
// l = l*2^(m-m') + 2^(s-m'); acc = acc*2^(m-m') + 2^(s-m') v_j.
#include "device_common.hpp"

namespace padoc {

template <int D, bool PAGED>
__global__ __launch_bounds__(256) void tile_valu_f32_kernel(TileParams p) {
  constexpr bool PARTIAL = PAGED;  // decode plans write split-KV partials
  const WorkRec w = p.work[blockIdx.x];
  if ((int)threadIdx.x >= w.ncol) return;  // no barriers below
  const int c = w.col0 + threadIdx.x;
  const int t = c / p.G;
  const int h = c - t * p.G;
  if (t >= w.ntok) return;
  const int32_t qrow = p.toks[w.tok_begin + t];
  const int32_t hq = w.kvh * p.G + h;
  const float4* qp = reinterpret_cast<const float4*>(static_cast<const float*>(p.q) + ((int64_t)qrow * p.Hq + hq) * D);
  float q[D];
#pragma unroll
  for (int i = 0; i < D / 4; ++i) {
    const float4 x = qp[i];
    q[4 * i] = x.x;
    q[4 * i + 1] = x.y;
    q[4 * i + 2] = x.z;
    q[4 * i + 3] = x.w;
  }
  float m = -INFINITY, l = 0.f;
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;
  const float* K = static_cast<const float*>(p.k);
  const float* V = static_cast<const float*>(p.v);
  for (int r = 0; r < w.rng_count; ++r) {
    const RangeRec R = p.ranges[w.rng_begin + r];
    const int lim = R.lim_off < 0 ? R.n_keys : p.lims[R.lim_off + t];
    for (int j = 0; j < lim; ++j) {
      // K row j: packed [T, Hkv, D]; paged chunk-major blocks (8 dims per piece)
      int64_t off;
      int64_t blk = 0;
      if constexpr (PAGED) {
        blk = p.block_table[R.kv_start + (j >> 4)];
        off = paged_k_offset<D>(blk, w.kvh, p.Hkv, j & 15, 0);
      } else {
        off = ((R.kv_start + j) * p.Hkv + w.kvh) * (int64_t)D;
      }
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < D / 4; ++i) {
        // dims 4i..4i+3: chunk i/2, half i%2 of the piece
        const int64_t ko = PAGED ? off + (i >> 1) * (kBlock * 8) + 4 * (i & 1) : off + 4 * i;
        const float4 x = *reinterpret_cast<const float4*>(K + ko);
        s = fmaf(q[4 * i], x.x, s);
        s = fmaf(q[4 * i + 1], x.y, s);
        s = fmaf(q[4 * i + 2], x.z, s);
        s = fmaf(q[4 * i + 3], x.w, s);
      }
      s *= p.scale_log2;
      // V row j: packed [T, Hkv, D]; paged d-major blocks [Hkv][D][16]
      int64_t voff, vstride;
      if constexpr (PAGED) {
        voff = (blk * p.Hkv + w.kvh) * (int64_t)D * kBlock + (j & 15);
        vstride = kBlock;
      } else {
        voff = off;
        vstride = 1;
      }
      if (s > m) {
        const float a = fast_exp2(m - s);
        l *= a;
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] *= a;
        m = s;
      }
      const float e = fast_exp2(s - m);
      l += e;
#pragma unroll
      for (int dd = 0; dd < D; ++dd) acc[dd] = fmaf(e, V[voff + dd * vstride], acc[dd]);
    }
  }
  if constexpr (PARTIAL) {
    const int64_t slot = (int64_t)w.out_base + c;
    float4* op = reinterpret_cast<float4*>(p.part_o + slot * D);
#pragma unroll
    for (int i = 0; i < D / 4; ++i) op[i] = make_float4(acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]);
    p.part_ml[2 * slot] = m;
    p.part_ml[2 * slot + 1] = l;
  } else {
    const float inv = 1.f / l;
    float4* op = reinterpret_cast<float4*>(static_cast<float*>(p.o) + ((int64_t)qrow * p.Hq + hq) * D);
#pragma unroll
    for (int i = 0; i < D / 4; ++i)
      op[i] = make_float4(acc[4 * i] * inv, acc[4 * i + 1] * inv, acc[4 * i + 2] * inv, acc[4 * i + 3] * inv);
    p.lse[(int64_t)qrow * p.Hq + hq] = (m + __log2f(l)) * kLn2;
  }
}

hipError_t launch_tile_valu_f32(const TileParams& p, int n_work, int D, bool paged, hipStream_t stream) {
  const dim3 grid(n_work), block(kTileCols);
  if (D == 64) {
    if (paged) hipLaunchKernelGGL((tile_valu_f32_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((tile_valu_f32_kernel<64, false>), grid, block, 0, stream, p);
  } else {
    if (paged) hipLaunchKernelGGL((tile_valu_f32_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((tile_valu_f32_kernel<128, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace padoc

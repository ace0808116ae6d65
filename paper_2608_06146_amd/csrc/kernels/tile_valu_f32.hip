// fp32 tile kernel: one thread per (query token, head) column of a work item,
// keys visited one by one with an exact online softmax in fp32 on the vector
// ALUs.  This is the fp32 path of both entry points (the MFMA path is bf16);
// it reads the same schedule as the bf16 kernel.
//
// Per column and visible key j (App. E Attn equation, with the scale applied
// in log2 units): s = scale*log2(e) * q.k_j; m' = max(m, s);
// l = l*2^(m-m') + 2^(s-m'); acc = acc*2^(m-m') + 2^(s-m') v_j.
#include "device_common.hpp"

namespace padoc {

template <int D, bool PAGED, bool PARTIAL>
__global__ __launch_bounds__(256) void tile_valu_f32_kernel(TileParams p) {
  const WorkRec w = p.work[blockIdx.x];
  const int c = threadIdx.x;
  const int t = c / p.G;
  const int h = c - t * p.G;
  if (t >= w.ntok) return;  // no barriers below
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
      const int64_t off = key_offset<D, PAGED>(R, j, w.kvh, p.Hkv, p.block_table);
      const float4* kp = reinterpret_cast<const float4*>(K + off);
      const float4* vp = reinterpret_cast<const float4*>(V + off);
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < D / 4; ++i) {
        const float4 x = kp[i];
        s = fmaf(q[4 * i], x.x, s);
        s = fmaf(q[4 * i + 1], x.y, s);
        s = fmaf(q[4 * i + 2], x.z, s);
        s = fmaf(q[4 * i + 3], x.w, s);
      }
      s *= p.scale_log2;
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
      for (int i = 0; i < D / 4; ++i) {
        const float4 x = vp[i];
        acc[4 * i] = fmaf(e, x.x, acc[4 * i]);
        acc[4 * i + 1] = fmaf(e, x.y, acc[4 * i + 1]);
        acc[4 * i + 2] = fmaf(e, x.z, acc[4 * i + 2]);
        acc[4 * i + 3] = fmaf(e, x.w, acc[4 * i + 3]);
      }
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

hipError_t launch_tile_valu_f32(const TileParams& p, int n_work, int D, bool paged, bool partial,
                                hipStream_t stream) {
  const dim3 grid(n_work), block(256);
#define PADOC_LAUNCH(DD, PG, PT) \
  hipLaunchKernelGGL((tile_valu_f32_kernel<DD, PG, PT>), grid, block, 0, stream, p)
  if (D == 64) {
    if (paged) {
      if (partial) PADOC_LAUNCH(64, true, true); else PADOC_LAUNCH(64, true, false);
    } else {
      if (partial) PADOC_LAUNCH(64, false, true); else PADOC_LAUNCH(64, false, false);
    }
  } else {
    if (paged) {
      if (partial) PADOC_LAUNCH(128, true, true); else PADOC_LAUNCH(128, true, false);
    } else {
      if (partial) PADOC_LAUNCH(128, false, true); else PADOC_LAUNCH(128, false, false);
    }
  }
#undef PADOC_LAUNCH
  return hipGetLastError();
}

}  // namespace padoc

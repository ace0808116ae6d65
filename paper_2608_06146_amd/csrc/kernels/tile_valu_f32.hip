// fp32 kernels (the MFMA paths are bf16).  They read the same schedules as
// the bf16 kernels.
//
// Decode (paged cache: K blocks chunk-major [d/8][16 slots][8], V blocks
// d-major [d][16]): one thread per (query token, head) column of a work item,
// keys visited one by one with an exact online softmax on the vector ALUs;
// outputs are split partials for the combine kernel.  Per column and visible
// key j (App. E Attn equation, scale applied in log2 units):
// s = scale*log2(e) * q.k_j; m' = max(m, s); l = l*2^(m-m') + 2^(s-m');
// acc = acc*2^(m-m') + 2^(s-m') v_j.
//
// Packed forward: tile_f32_split_kernel below.
#include "device_common.hpp"

namespace padoc {

template <int D>
__global__ __launch_bounds__(256) void tile_valu_f32_paged_kernel(TileParams p) {
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
      // K row j: chunk-major block (8 dims per piece)
      const int64_t blk = p.block_table[R.kv_start + (j >> 4)];
      const int64_t off = paged_k_offset<D>(blk, w.kvh, p.Hkv, j & 15, 0);
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < D / 4; ++i) {
        // dims 4i..4i+3: chunk i/2, half i%2 of the piece
        const float4 x = *reinterpret_cast<const float4*>(K + off + (i >> 1) * (kBlock * 8) + 4 * (i & 1));
        s = fmaf(q[4 * i], x.x, s);
        s = fmaf(q[4 * i + 1], x.y, s);
        s = fmaf(q[4 * i + 2], x.z, s);
        s = fmaf(q[4 * i + 3], x.w, s);
      }
      s *= p.scale_log2;
      // V row j: d-major block [Hkv][D][16]
      const int64_t voff = (blk * p.Hkv + w.kvh) * (int64_t)D * kBlock + (j & 15);
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
      for (int dd = 0; dd < D; ++dd) acc[dd] = fmaf(e, V[voff + dd * kBlock], acc[dd]);
    }
  }
  const int64_t slot = (int64_t)w.out_base + c;
  float4* op = reinterpret_cast<float4*>(p.part_o + slot * D);
#pragma unroll
  for (int i = 0; i < D / 4; ++i) op[i] = make_float4(acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]);
  p.part_ml[2 * slot] = m;
  p.part_ml[2 * slot + 1] = l;
}

// Packed fp32 forward, keys split across the wavefronts of a workgroup: one
// workgroup of 8 wavefronts per (work item, group of 16 columns).  Lane
// (c, g) of every wavefront (c = lane % 16, g = lane / 16) holds column c of
// the group and quarter g of the head dimension (its Q and O quarters);
// wavefront w takes keys w, w+8, .. of each 64-key tile.  Tiles are staged
// in LDS by the whole workgroup, the next tile's rows loaded into registers
// while the current one is computed.  A score is the sum of the four
// quarters' partial dot products (two lane swaps); each wavefront keeps its
// own online softmax (log2 units, maximum raised once per tile), and the 8
// key slices of a column are merged through LDS at the end (m = max m_i,
// l = sum l_i 2^(m_i - m), O likewise: App. E Attn equation, the softmax of
// disjoint key sets merged).
constexpr int kF32Cols = 16;    // columns per workgroup
constexpr int kF32Waves = 8;    // key slices
constexpr int kF32Tile = 64;    // keys per staged tile

__device__ __forceinline__ float sum_lane_rows(float x) {  // lanes l, l^16
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_lane_halves(float x) {  // lanes l, l^32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup barrier after this wavefront's LDS accesses complete, without
// the memory fence of __syncthreads (which would also wait for the next
// tile's global loads in flight); the asm statements keep the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt, expcnt not waited for
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int D>
__global__ __launch_bounds__(kF32Waves * 64) void tile_f32_split_kernel(TileParams p) {
  constexpr int DQ = D / 4;                  // head dims per lane
  constexpr int KPW = kF32Tile / kF32Waves;  // keys per wavefront and tile
  constexpr int TILE_F = kF32Tile * D;       // floats of one staged tensor tile
  constexpr int NPF = 2 * TILE_F / 4 / (kF32Waves * 64);  // float4 staged per thread and tile
  constexpr int MERGE_F = (kF32Waves / 2) * 64 * (DQ + 2);
  constexpr int SMEM_F = 2 * TILE_F > MERGE_F ? 2 * TILE_F : MERGE_F;
  static_assert(NPF * kF32Waves * 64 * 4 == 2 * TILE_F, "whole float4 per thread");
  __shared__ __attribute__((aligned(16))) float sm[SMEM_F];

  const int item = blockIdx.x / (kTileCols / kF32Cols);
  const int cg = blockIdx.x % (kTileCols / kF32Cols);
  const WorkRec w = load_scalar(&p.work[item]);
  if (cg * kF32Cols >= w.ncol || w.rng_count <= 0) return;  // the whole workgroup: no barrier is split
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, cc = lane & 15, qd = lane >> 4;
  const int c = w.col0 + cg * kF32Cols + cc;
  const int t = c / p.G;
  const bool valid = cg * kF32Cols + cc < w.ncol && t < w.ntok;
  const int32_t qrow = valid ? p.toks[w.tok_begin + t] : 0;
  const int32_t hq = w.kvh * p.G + (c - t * p.G);
  const float* K = static_cast<const float*>(p.k);
  const float* V = static_cast<const float*>(p.v);

  float qv[DQ];
  {
    const float4* qp = reinterpret_cast<const float4*>(static_cast<const float*>(p.q) + ((int64_t)qrow * p.Hq + hq) * D + qd * DQ);
#pragma unroll
    for (int i = 0; i < DQ / 4; ++i) {
      const float4 x = valid ? qp[i] : make_float4(0.f, 0.f, 0.f, 0.f);
      qv[4 * i] = x.x, qv[4 * i + 1] = x.y, qv[4 * i + 2] = x.z, qv[4 * i + 3] = x.w;
    }
  }
  float m = -INFINITY, l = 0.f;
  float acc[DQ];
#pragma unroll
  for (int d = 0; d < DQ; ++d) acc[d] = 0.f;
  const float sl2 = p.scale_log2;

  // Tile cursor over the item's non-empty ranges: range r, first key kb.
  int r = 0, kb = 0;
  RangeRec R = load_scalar(&p.ranges[w.rng_begin]);
  while (R.n_keys <= 0 && ++r < w.rng_count) R = load_scalar(&p.ranges[w.rng_begin + r]);
  if (r >= w.rng_count) return;  // no keys at all (uniform over the workgroup)
  // Staging: float4 i = tid + 512 j of the K tile (i < 16 D) or V tile
  // (the rest); rows past the range's end repeat its last row (finite; their
  // scores are masked).
  float4 pf[NPF];
  auto fetch = [&](const RangeRec& Rf, int kbf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < NPF; ++j) {
      const int i = tid + kF32Waves * 64 * j;
      const int tensor = i / (TILE_F / 4);
      const int rem = i - tensor * (TILE_F / 4);
      const int row = rem / (D / 4), ch = rem % (D / 4);
      const int key = min(kbf + row, Rf.n_keys - 1);
      pf[j] = *reinterpret_cast<const float4*>((tensor ? V : K) + ((Rf.kv_start + key) * p.Hkv + w.kvh) * (int64_t)D + 4 * ch);
    }
  };
  // This column's key limit in range r (its length when it has no limits).
  auto limit_of = [&](const RangeRec& Rl) -> int {
    return !valid ? 0 : Rl.lim_off < 0 ? Rl.n_keys : p.lims[Rl.lim_off + t];
  };
  int lim_next = limit_of(R);
  fetch(R, kb);
  for (;;) {
    lds_barrier();  // every read of the previous tile is done
#pragma unroll
    for (int j = 0; j < NPF; ++j) reinterpret_cast<float4*>(sm)[tid + kF32Waves * 64 * j] = pf[j];
    // this tile's range and the next tile's position; the next range's
    // limit is loaded before the next tile's rows, so waiting for it does
    // not wait for them
    const int kbc = kb;
    const int lim = lim_next;
    bool more = true;
    kb += kF32Tile;
    if (kb >= R.n_keys) {
      kb = 0;
      for (++r; r < w.rng_count; ++r) {
        R = load_scalar(&p.ranges[w.rng_begin + r]);
        if (R.n_keys > 0) break;
      }
      more = r < w.rng_count;
      if (more) lim_next = limit_of(R);
    }
    if (more) fetch(R, kb);  // lands while this tile is computed
    lds_barrier();
    const float* Ks = sm;
    const float* Vs = sm + TILE_F;
    float s[KPW];
    float mt = -INFINITY;
#pragma unroll
    for (int u = 0; u < KPW; ++u) {
      const int kk = wave + kF32Waves * u;
      const float4* kr = reinterpret_cast<const float4*>(Ks + kk * D + qd * DQ);
      float part = 0.f;
#pragma unroll
      for (int i = 0; i < DQ / 4; ++i) {
        const float4 x = kr[i];
        part = fmaf(qv[4 * i], x.x, part);
        part = fmaf(qv[4 * i + 1], x.y, part);
        part = fmaf(qv[4 * i + 2], x.z, part);
        part = fmaf(qv[4 * i + 3], x.w, part);
      }
      const float full = sum_lane_halves(sum_lane_rows(part)) * sl2;
      s[u] = kbc + kk < lim ? full : -INFINITY;
      mt = fmaxf(mt, s[u]);
    }
    if (mt > m) {
      const float a = fast_exp2(m - mt);  // m = -inf: a = 0 (acc and l are 0)
      l *= a;
#pragma unroll
      for (int d = 0; d < DQ; ++d) acc[d] *= a;
      m = mt;
    }
    const float m_sub = m == -INFINITY ? 0.f : m;
#pragma unroll
    for (int u = 0; u < KPW; ++u) {
      const float e = fast_exp2(s[u] - m_sub);
      l += e;
      const float4* vr = reinterpret_cast<const float4*>(Vs + (wave + kF32Waves * u) * D + qd * DQ);
#pragma unroll
      for (int i = 0; i < DQ / 4; ++i) {
        const float4 x = vr[i];
        acc[4 * i] = fmaf(e, x.x, acc[4 * i]);
        acc[4 * i + 1] = fmaf(e, x.y, acc[4 * i + 1]);
        acc[4 * i + 2] = fmaf(e, x.z, acc[4 * i + 2]);
        acc[4 * i + 3] = fmaf(e, x.w, acc[4 * i + 3]);
      }
    }
    if (!more) break;
  }

  // Merge the key slices: wavefronts [k, 2k) hand (m, l, O quarter) to
  // wavefronts [0, k), for k = 4, 2, 1.  Layout [slot][value][lane].
#pragma unroll
  for (int k = kF32Waves / 2; k >= 1; k >>= 1) {
    __syncthreads();
    if (wave >= k && wave < 2 * k) {
      float* b = sm + (wave - k) * 64 * (DQ + 2) + lane;
      b[0] = m;
      b[64] = l;
#pragma unroll
      for (int d = 0; d < DQ; ++d) b[64 * (d + 2)] = acc[d];
    }
    __syncthreads();
    if (wave < k) {
      const float* b = sm + wave * 64 * (DQ + 2) + lane;
      const float m2 = b[0], l2 = b[64];
      const float mn = fmaxf(m, m2);
      const float ms = mn == -INFINITY ? 0.f : mn;
      const float a1 = fast_exp2(m - ms), a2 = fast_exp2(m2 - ms);
      l = l * a1 + l2 * a2;
#pragma unroll
      for (int d = 0; d < DQ; ++d) acc[d] = acc[d] * a1 + b[64 * (d + 2)] * a2;
      m = mn;
    }
  }
  if (wave != 0 || !valid) return;
  const float inv = 1.f / l;
  float4* op = reinterpret_cast<float4*>(static_cast<float*>(p.o) + ((int64_t)qrow * p.Hq + hq) * D + qd * DQ);
#pragma unroll
  for (int i = 0; i < DQ / 4; ++i)
    op[i] = make_float4(acc[4 * i] * inv, acc[4 * i + 1] * inv, acc[4 * i + 2] * inv, acc[4 * i + 3] * inv);
  if (qd == 0) p.lse[(int64_t)qrow * p.Hq + hq] = (m + __log2f(l)) * kLn2;
}

hipError_t launch_tile_valu_f32(const TileParams& p, int n_work, int D, bool paged, hipStream_t stream) {
  const dim3 grid(n_work), block(kTileCols);
  if (!paged) {
    // packed forward: the key-split kernel, one workgroup per 32 columns
    const dim3 sgrid((unsigned)n_work * (kTileCols / kF32Cols)), sblock(kF32Waves * 64);
    if (D == 64)
      hipLaunchKernelGGL((tile_f32_split_kernel<64>), sgrid, sblock, 0, stream, p);
    else
      hipLaunchKernelGGL((tile_f32_split_kernel<128>), sgrid, sblock, 0, stream, p);
    return hipGetLastError();
  }
  if (D == 64)
    hipLaunchKernelGGL((tile_valu_f32_paged_kernel<64>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((tile_valu_f32_paged_kernel<128>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace padoc

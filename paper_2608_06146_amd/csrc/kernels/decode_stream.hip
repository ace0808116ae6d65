// Split-KV decode kernel over the paged cache, one wave item per wavefront.
//
// A wave item is up to 32 columns (query token x head of one KV-head group)
// against one key chunk (App. E: one decode step of the live streams; Attn
// equation with the ancestor mask).  Each wavefront streams its keys straight
// from HBM into matrix-core operand registers, 32 keys per step, and keeps
// the next step's loads in flight while it computes the current one:
//
//   S^T = K Q^T       v_mfma_f32_32x32x16_bf16; accumulator row m of the
//                     step holds key perm_key(m) (bits 2 and 3 of m swapped)
//   online softmax    one column per lane, the other half of its keys in
//                     lane ^ 32
//   O^T += V^T P^T    with the permutation above, lane half h's eight P^T
//                     values are the keys 16j + 8h .. +7 of the step, which a
//                     d-major V block ([d][16 slots]) delivers as one 16-byte
//                     load per lane -- no LDS, no transposes, no barriers.
//
// The B operand (Q fragments) is kept in a per-wave LDS slice rather than in
// registers, so two 8-wave workgroups' worth of waves fit per SIMD pair.
// Waves of one workgroup that belong to the same page's shared group stream
// identical addresses in step, so the prefix and layout-stream keys are read
// from HBM once and served to the sibling waves from the compute unit's
// cache.  Keys past a range's end are never loaded; V lanes of a partially
// used block are zeroed, so sentinel or stale slots never enter a product.
// The partial (unnormalised O, running max in log2 units, sum) of every
// column is written for the fixed-order combine kernel.
#include "device_common.hpp"

namespace padoc {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int perm_key(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& u) { return *reinterpret_cast<const bf16x8_t*>(&u); }

// Zero the bf16 elements at positions >= keep of an 8-element chunk (keep
// may be <= 0 or >= 8).
__device__ __forceinline__ uint4 keep_first(uint4 u, int keep) {
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lo = 2 * i;
    const uint32_t m = (lo + 1 < keep) ? 0xffffffffu : (lo < keep ? 0x0000ffffu : 0u);
    w[i] &= m;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <int D, int NB>
__device__ __forceinline__ void stream_item(const TileParams& p, const WorkRec& w, const int lane,
                                            uint16_t* __restrict__ qs) {
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int CPR = D / 8;  // 16-byte chunks per Q row
  const int l32 = lane & 31, hf = lane >> 5;
  const int G = p.G;
  const int kvh = w.kvh;
  const int64_t Hkv = p.Hkv;
  const uint16_t* Kc = static_cast<const uint16_t*>(p.k);
  const uint16_t* Vc = static_cast<const uint16_t*>(p.v);
  const int32_t* bt = p.block_table;

  int tok[NB];
  bool valid[NB];
  int32_t qrow[NB], hq[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int c = nb * 32 + l32;
    const int t = c / G;
    tok[nb] = t;
    valid[nb] = t < w.ntok;
    qrow[nb] = valid[nb] ? p.toks[w.tok_begin + t] : 0;
    hq[nb] = kvh * G + (c - t * G);
  }
  // Q tile of this wave in LDS: row = column l32 (32 rows), 16-byte chunk c
  // of row r stored at chunk c ^ (r % CPR) so the fragment reads below hit
  // distinct banks.  Lane (l32, hf) writes half hf of its row.
  const uint16_t* Q = static_cast<const uint16_t*>(p.q);
  {
    const uint16_t* qp = Q + ((int64_t)qrow[0] * p.Hq + hq[0]) * D;
#pragma unroll
    for (int i = 0; i < CPR / 2; ++i) {
      const int c = hf * (CPR / 2) + i;
      const uint4 z = valid[0] ? *reinterpret_cast<const uint4*>(qp + c * 8) : make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4*>(qs + l32 * D + ((c ^ (l32 % CPR)) * 8)) = z;
    }
  }
  auto qfrag = [&](int kk) -> bf16x8_t {
    const int c = 2 * kk + hf;  // d = kk*16 + hf*8 .. +7
    return as_bf16x8(*reinterpret_cast<const uint4*>(qs + l32 * D + ((c ^ (l32 % CPR)) * 8)));
  };

  const int kperm = perm_key(l32);  // key of this lane's K row within a step

  // Loads of one 32-key step, branch-free: addresses are clamped to a valid
  // block of the range and lanes past its end are zeroed after the load.
  // K and V each have one register set; the next step's K is loaded right
  // after the score MFMAs consumed the current K, the next V right after the
  // PV MFMAs consumed the current V, so each load has about one step of
  // compute to arrive.
  uint4 kreg[NKK];
  uint4 vreg[NDB][2];
  int64_t vb0 = 0, vb1 = 0;  // blocks of the step whose V is loaded next
  auto load_k = [&](const RangeRec& R, int kb) {
    const int nk = R.n_keys;
    const int64_t base = R.kv_start + (kb >> 4);
    vb0 = bt[base];
    vb1 = bt[base + ((kb + 16 < nk) ? 1 : 0)];
    const bool ok = kb + kperm < nk;
    const uint16_t* kp = Kc + (((kperm & 16) ? vb1 : vb0) * Hkv + kvh) * (kBlock * D) + (kperm & 15) * D + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const uint4 x = *reinterpret_cast<const uint4*>(kp + kk * 16);
      kreg[kk] = ok ? x : make_uint4(0, 0, 0, 0);
    }
  };
  auto load_v = [&](int nk, int kb) {
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int keep = nk - (kb + 16 * jj + 8 * hf);
      const uint16_t* vp = Vc + ((jj ? vb1 : vb0) * Hkv + kvh) * (kBlock * D) + l32 * kBlock + 8 * hf;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        vreg[db][jj] = keep_first(*reinterpret_cast<const uint4*>(vp + db * 32 * kBlock), keep);
    }
  };

  float m_run[NB], l_run[NB];
  f32x16_t acc[NDB][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = -INFINITY;
    l_run[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[db][nb][i] = 0.f;
  }

  int ri = 0, st = 0;
  RangeRec R = p.ranges[w.rng_begin];
  int lim[NB];
  auto load_lims = [&]() {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      lim[nb] = R.lim_off < 0 ? R.n_keys : (valid[nb] ? p.lims[R.lim_off + tok[nb]] : 0);
  };
  load_lims();
  const float sl2 = p.scale_log2;
  load_k(R, 0);
  load_v(R.n_keys, 0);

  while (true) {
    int nri = ri, nst = st + 1;
    RangeRec NR = R;
    bool has_next = true;
    if (nst * 32 >= R.n_keys) {
      nri = ri + 1;
      nst = 0;
      if (nri < w.rng_count)
        NR = p.ranges[w.rng_begin + nri];
      else
        has_next = false;
    }
    const int kb = st * 32;
    f32x16_t S[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 16; ++i) S[nb][i] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8_t a = as_bf16x8(kreg[kk]);
      S[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qfrag(kk), S[0], 0, 0, 0);
    }
    if (has_next) load_k(NR, nst * 32);  // also selects the next step's blocks for load_v

    if (kb + 32 > R.min_lim) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kb + perm_key((i >> 2) * 8 + hf * 4 + (i & 3));
          if (key >= lim[nb]) S[nb][i] = -INFINITY;
        }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[nb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[nb], mx * sl2);
      const float m_sub = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[nb] - m_sub);
      m_run[nb] = m_new;
      float ls = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float e = fast_exp2(fmaf(S[nb][i], sl2, -m_sub));
        S[nb][i] = e;
        ls += e;
      }
      l_run[nb] = fmaf(l_run[nb], alpha, ls);
#pragma unroll
      for (int db = 0; db < NDB; ++db) acc[db][nb] *= alpha;
    }
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      bf16x8_t pb[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f32x8_t x;
#pragma unroll
        for (int s = 0; s < 8; ++s) x[s] = S[nb][8 * jj + s];
        pb[nb] = __builtin_convertvector(x, bf16x8_t);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8_t a = as_bf16x8(vreg[db][jj]);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[db][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[nb], acc[db][nb], 0, 0, 0);
      }
    }
    if (!has_next) break;
    load_v(NR.n_keys, nst * 32);
    if (nri != ri) {
      R = NR;
      ri = nri;
      load_lims();
    }
    st = nst;
  }

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float lt = l_run[nb] + __shfl_xor(l_run[nb], 32);
    if (!valid[nb]) continue;
    const int64_t slot = (int64_t)w.out_base + nb * 32 + l32;
    float* op = p.part_o + slot * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int d0 = db * 32 + i4 * 8 + hf * 4;
        *reinterpret_cast<float4*>(op + d0) = make_float4(acc[db][nb][4 * i4], acc[db][nb][4 * i4 + 1],
                                                          acc[db][nb][4 * i4 + 2], acc[db][nb][4 * i4 + 3]);
      }
    if (hf == 0) {
      p.part_ml[2 * slot] = m_run[nb];
      p.part_ml[2 * slot + 1] = lt;
    }
  }
}

template <int D>
__global__ __launch_bounds__(64 * kDecodeWaves) void decode_stream_kernel(TileParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t qs[kDecodeWaves][32 * D];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const WorkRec w = p.work[blockIdx.x * kDecodeWaves + wave];
  if (w.ntok <= 0 || w.rng_count <= 0) return;  // idle wave; no barriers in this kernel
  stream_item<D, 1>(p, w, lane, qs[wave]);
}

}  // namespace

hipError_t launch_decode_stream_bf16(const TileParams& p, int n_items, int D, hipStream_t stream) {
  const dim3 grid((n_items + kDecodeWaves - 1) / kDecodeWaves), block(64 * kDecodeWaves);
  if (D == 64)
    hipLaunchKernelGGL((decode_stream_kernel<64>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((decode_stream_kernel<128>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace padoc

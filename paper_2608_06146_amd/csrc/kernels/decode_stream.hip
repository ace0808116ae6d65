// Split-KV decode kernel over the paged cache, one wave item per wavefront.
//
// A wave item is up to 64 columns (query token x head of one KV-head group)
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

// Zero the bf16 elements at positions >= keep (0..8) of an 8-element chunk.
__device__ __forceinline__ uint4 keep_first(uint4 u, int keep) {
  if (keep >= 8) return u;
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lo = 2 * i;
    const uint32_t m = (lo + 1 < keep) ? 0xffffffffu : (lo < keep ? 0x0000ffffu : 0u);
    w[i] &= m;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <int D>
struct StepRegs {
  uint4 k[D / 16];        // K operand: this lane's key row, d = kk*16 + hf*8 .. +7
  uint4 v[D / 32][2];     // V^T operand: d = db*32 + l32, keys 16j + 8hf .. +7
};

template <int D, int NB>
__device__ __forceinline__ void stream_item(const TileParams& p, const WorkRec& w, const int lane) {
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
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
  bf16x8_t bq[NB][NKK];
  const uint16_t* Q = static_cast<const uint16_t*>(p.q);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const uint16_t* qp = Q + ((int64_t)qrow[nb] * p.Hq + hq[nb]) * D + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const uint4 z = valid[nb] ? *reinterpret_cast<const uint4*>(qp + kk * 16) : make_uint4(0, 0, 0, 0);
      bq[nb][kk] = as_bf16x8(z);
    }
  }

  const int kperm = perm_key(l32);  // key of this lane's K row within a step

  auto load_step = [&](const RangeRec& R, int kb, StepRegs<D>& s) {
    const int nk = R.n_keys;
    const int64_t base = R.kv_start + (kb >> 4);
    const int64_t b0 = bt[base];
    const int64_t b1 = (kb + 16 < nk) ? (int64_t)bt[base + 1] : b0;
    // K rows
    const int j = kb + kperm;
    if (j < nk) {
      const int64_t blk = (kperm & 16) ? b1 : b0;
      const uint16_t* kp = Kc + ((blk * Hkv + kvh) * kBlock + (kperm & 15)) * D + hf * 8;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) s.k[kk] = *reinterpret_cast<const uint4*>(kp + kk * 16);
    } else {
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) s.k[kk] = make_uint4(0, 0, 0, 0);
    }
    // V^T rows (d-major blocks)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int first = kb + 16 * jj + 8 * hf;  // first key of this lane's 8
      const int keep = nk - first;
      const int64_t blk = jj ? b1 : b0;
      if (keep > 0) {
        const uint16_t* vp = Vc + ((blk * Hkv + kvh) * D + l32) * kBlock + 8 * hf;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          s.v[db][jj] = keep_first(*reinterpret_cast<const uint4*>(vp + (int64_t)db * 32 * kBlock), keep);
      } else {
#pragma unroll
        for (int db = 0; db < NDB; ++db) s.v[db][jj] = make_uint4(0, 0, 0, 0);
      }
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
  StepRegs<D> cur, nxt;
  load_step(R, 0, cur);
  const float sl2 = p.scale_log2;

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
    if (has_next) load_step(NR, nst * 32, nxt);

    const int kb = st * 32;
    f32x16_t S[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 16; ++i) S[nb][i] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8_t a = as_bf16x8(cur.k[kk]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) S[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[nb][kk], S[nb], 0, 0, 0);
    }
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
        const bf16x8_t a = as_bf16x8(cur.v[db][jj]);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[db][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[nb], acc[db][nb], 0, 0, 0);
      }
    }

    if (!has_next) break;
    if (nri != ri) {
      R = NR;
      ri = nri;
      load_lims();
    }
    st = nst;
    cur = nxt;
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
__global__ __launch_bounds__(256, 1) void decode_stream_kernel(TileParams p) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const WorkRec w = p.work[blockIdx.x * 4 + wave];
  if (w.ntok <= 0 || w.rng_count <= 0) return;  // idle wave; no barriers in this kernel
  if (w.nblk == 1)
    stream_item<D, 1>(p, w, lane);
  else
    stream_item<D, 2>(p, w, lane);
}

}  // namespace

hipError_t launch_decode_stream_bf16(const TileParams& p, int n_items, int D, hipStream_t stream) {
  const dim3 grid((n_items + 3) / 4), block(256);
  if (D == 64)
    hipLaunchKernelGGL((decode_stream_kernel<64>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((decode_stream_kernel<128>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace padoc

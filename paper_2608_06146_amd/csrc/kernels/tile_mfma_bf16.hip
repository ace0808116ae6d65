// bf16 packed-forward tile kernel for gfx950 (CDNA4) matrix cores.
//
// One workgroup (4 waves) processes one work item: up to 256 columns
// (query token x head of one KV-head group; GQA heads of a token share every
// K/V tile) against the item's key ranges, 64 keys per step.  Per step the
// workgroup stages the K tile row-major and the V tile transposed in LDS,
// then every wave, for its 64 columns:
//   S^T = K Q^T            v_mfma_f32_32x32x16_bf16, keys on M, columns on N
//   online softmax         per column = per lane (the 32x32 accumulator
//                          layout gives a lane one column and 16 key rows;
//                          the other 16 rows are in lane^32)
//   O^T += V^T P^T         P^T comes straight from the S^T registers
// (App. E Attn equation; App. C tree-varlen relation).  Only tiles of
// ancestor prefixes and the own causal range are ever visited: the planner
// lists no other segment.  Tiles wholly below every column's limit skip the
// mask; keys past a range's end are zero-filled in LDS so no stale or
// sentinel memory enters a product.
//
// Accumulation is fp32; scores are scaled into log2 units so the
// exponentials are single v_exp_f32; O is rounded to bf16 (RNE) at the end.
#include "device_common.hpp"

namespace padoc {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Position of key r (0..63) inside a transposed V row.  Within each group of
// 16 keys, lane half 0 of the 32x32 P^T fragment holds keys
// {0,1,2,3,8,9,10,11} and half 1 holds {4..7,12..15}; storing them in that
// order makes each half's 8 keys one contiguous 16-byte LDS read.
__device__ __forceinline__ int vt_pos(int r) {
  const int q = r & 15;
  return (r & ~15) + ((q >> 2) & 1) * 8 + (q >> 3) * 4 + (q & 3);
}

template <int D, bool PAGED, bool PARTIAL>
__global__ __launch_bounds__(256, 1) void tile_mfma_bf16_kernel(TileParams p) {
  constexpr int KT = kTileKeys;     // 64 keys per step
  constexpr int KS = D + 8;         // K row stride in LDS (elements); +8 spreads banks
  constexpr int VS = KT + 8;        // V^T row stride in LDS
  constexpr int NKK = D / 16;       // K-slices of the score product
  constexpr int NDB = D / 32;       // 32-row blocks of O^T
  constexpr int CPR = D / 8;        // 16-byte chunks per key row
  constexpr int KPT = KT * CPR / 256;        // K chunks per thread
  constexpr int VPT = KT * CPR / 512;        // V key-pair chunks per thread

  __shared__ __attribute__((aligned(16))) uint16_t Ks[KT * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VS];

  const WorkRec w = p.work[blockIdx.x];
  if (w.rng_count <= 0) return;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int G = p.G;

  int tok[2];
  bool valid[2];
  int32_t qrow[2], hq[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int c = wave * 64 + nb * 32 + l32;
    const int t = c / G;
    tok[nb] = t;
    valid[nb] = t < w.ntok;
    qrow[nb] = valid[nb] ? p.toks[w.tok_begin + t] : 0;
    hq[nb] = w.kvh * G + (c - t * G);
  }

  // Q fragments (B operand of S^T = K Q^T): lane (column l32, half hf) holds
  // d = kk*16 + hf*8 .. +7.
  const uint16_t* Q = static_cast<const uint16_t*>(p.q);
  bf16x8_t bq[2][NKK];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const uint16_t* qp = Q + ((int64_t)qrow[nb] * p.Hq + hq[nb]) * D + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      if (valid[nb]) {
        bq[nb][kk] = *reinterpret_cast<const bf16x8_t*>(qp + kk * 16);
      } else {
        const uint4 z = make_uint4(0, 0, 0, 0);
        bq[nb][kk] = *reinterpret_cast<const bf16x8_t*>(&z);
      }
    }
  }

  const uint16_t* Kg = static_cast<const uint16_t*>(p.k);
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v);
  uint4 kr[KPT], vr[2 * VPT];

  auto load_tile = [&](const RangeRec& R, int kt) {
    const int kbase = kt * KT;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + 256 * i;
      const int key = c / CPR, dc = c % CPR;
      const int j = kbase + key;
      if (j < R.n_keys)
        kr[i] = *reinterpret_cast<const uint4*>(Kg + key_offset<D, PAGED>(R, j, w.kvh, p.Hkv, p.block_table) + dc * 8);
      else
        kr[i] = make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + 256 * i;
      const int pr = u % (KT / 2), dc = u / (KT / 2);
      const int j0 = kbase + 2 * pr;
      if (j0 < R.n_keys)
        vr[2 * i] = *reinterpret_cast<const uint4*>(Vg + key_offset<D, PAGED>(R, j0, w.kvh, p.Hkv, p.block_table) + dc * 8);
      else
        vr[2 * i] = make_uint4(0, 0, 0, 0);
      if (j0 + 1 < R.n_keys)
        vr[2 * i + 1] =
            *reinterpret_cast<const uint4*>(Vg + key_offset<D, PAGED>(R, j0 + 1, w.kvh, p.Hkv, p.block_table) + dc * 8);
      else
        vr[2 * i + 1] = make_uint4(0, 0, 0, 0);
    }
  };

  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + 256 * i;
      const int key = c / CPR, dc = c % CPR;
      *reinterpret_cast<uint4*>(&Ks[key * KS + dc * 8]) = kr[i];
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + 256 * i;
      const int pr = u % (KT / 2), dc = u / (KT / 2);
      const int pos = vt_pos(2 * pr);
      const uint32_t a[4] = {vr[2 * i].x, vr[2 * i].y, vr[2 * i].z, vr[2 * i].w};
      const uint32_t b[4] = {vr[2 * i + 1].x, vr[2 * i + 1].y, vr[2 * i + 1].z, vr[2 * i + 1].w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        // d = dc*8 + 2m holds (key 2pr, key 2pr+1) low halves; d+1 the high halves
        *reinterpret_cast<uint32_t*>(&Vt[(dc * 8 + 2 * m) * VS + pos]) = (a[m] & 0xffffu) | (b[m] << 16);
        *reinterpret_cast<uint32_t*>(&Vt[(dc * 8 + 2 * m + 1) * VS + pos]) = (a[m] >> 16) | (b[m] & 0xffff0000u);
      }
    }
  };

  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};
  f32x16_t acc[NDB][2];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[db][nb][i] = 0.f;

  int ri = 0, kt = 0;
  RangeRec R = p.ranges[w.rng_begin];
  int lim[2];
  auto load_lims = [&]() {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
      lim[nb] = R.lim_off < 0 ? R.n_keys : (valid[nb] ? p.lims[R.lim_off + tok[nb]] : 0);
  };
  load_lims();
  load_tile(R, 0);
  const float sl2 = p.scale_log2;

  while (true) {
    __syncthreads();  // every wave is done reading the previous tile
    store_tile();
    __syncthreads();

    // Prefetch the next tile into registers while this one is computed.
    int nri = ri, nkt = kt + 1;
    RangeRec NR = R;
    bool has_next = true;
    if (nkt * KT >= R.n_keys) {
      nri = ri + 1;
      nkt = 0;
      if (nri < w.rng_count)
        NR = p.ranges[w.rng_begin + nri];
      else
        has_next = false;
    }
    if (has_next) load_tile(NR, nkt);

    // S^T = K Q^T for 64 keys x 64 columns.
    f32x16_t S[2][2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int i = 0; i < 16; ++i) S[mb][nb][i] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&Ks[(mb * 32 + l32) * KS + kk * 16 + hf * 8]);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          S[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[nb][kk], S[mb][nb], 0, 0, 0);
      }
    }

    if ((kt + 1) * KT > R.min_lim) {
      // Partial tile: key (mb, i) of this lane is
      // kt*64 + mb*32 + (i/4)*8 + hf*4 + i%4.
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = kt * KT + mb * 32 + (i >> 2) * 8 + hf * 4 + (i & 3);
            if (key >= lim[nb]) S[mb][nb][i] = -INFINITY;
          }
    }

    // Online softmax, one column per lane (shared with lane ^ 32).
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float mx = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[mb][nb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[nb], mx * sl2);
      const float m_sub = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[nb] - m_sub);
      m_run[nb] = m_new;
      float ls = 0.f;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float e = fast_exp2(fmaf(S[mb][nb][i], sl2, -m_sub));
          S[mb][nb][i] = e;
          ls += e;
        }
      l_run[nb] = fmaf(l_run[nb], alpha, ls);
#pragma unroll
      for (int db = 0; db < NDB; ++db) acc[db][nb] *= alpha;
    }

    // O^T += V^T P^T, 16 keys per MFMA: keys mb*32 + 16j + [0,16).
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        bf16x8_t pb[2];
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          f32x8_t x;
#pragma unroll
          for (int s = 0; s < 8; ++s) x[s] = S[mb][nb][8 * j + s];
          pb[nb] = __builtin_convertvector(x, bf16x8_t);
        }
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8_t a =
              *reinterpret_cast<const bf16x8_t*>(&Vt[(db * 32 + l32) * VS + mb * 32 + 16 * j + hf * 8]);
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            acc[db][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[nb], acc[db][nb], 0, 0, 0);
        }
      }
    }

    if (!has_next) break;
    if (nri != ri) {
      R = NR;
      ri = nri;
      load_lims();
    }
    kt = nkt;
  }

  // Epilogue.  Lane (column, hf) holds d = db*32 + (i/4)*8 + hf*4 + i%4.
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const float lt = l_run[nb] + __shfl_xor(l_run[nb], 32);
    if (!valid[nb]) continue;
    if constexpr (PARTIAL) {
      const int64_t slot = (int64_t)w.out_base + wave * 64 + nb * 32 + l32;
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
    } else {
      const float inv = 1.f / lt;
      uint16_t* op = static_cast<uint16_t*>(p.o) + ((int64_t)qrow[nb] * p.Hq + hq[nb]) * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int d0 = db * 32 + i4 * 8 + hf * 4;
          uint2 pk;
          pk.x = (uint32_t)f32_to_bf16_bits(acc[db][nb][4 * i4] * inv) |
                 ((uint32_t)f32_to_bf16_bits(acc[db][nb][4 * i4 + 1] * inv) << 16);
          pk.y = (uint32_t)f32_to_bf16_bits(acc[db][nb][4 * i4 + 2] * inv) |
                 ((uint32_t)f32_to_bf16_bits(acc[db][nb][4 * i4 + 3] * inv) << 16);
          *reinterpret_cast<uint2*>(op + d0) = pk;
        }
      if (hf == 0) p.lse[(int64_t)qrow[nb] * p.Hq + hq[nb]] = (m_run[nb] + __log2f(lt)) * kLn2;
    }
  }
}

hipError_t launch_tile_mfma_bf16(const TileParams& p, int n_work, int D, hipStream_t stream) {
  const dim3 grid(n_work), block(256);
  if (D == 64)
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<64, false, false>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((tile_mfma_bf16_kernel<128, false, false>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace padoc

// Backward of the packed tree forward (bf16, gfx950 matrix cores).
//
// The gradient of sum(dO * O) with O = softmax(scale * q K^T + A_M) V over
// each query's visible keys (App. E Attn equation with the ancestor mask;
// App. C tree-varlen relation, the backend the paper trains with), written
// per query row i and visible key j:
//   P_ij  = exp(scale q_i.k_j - LSE_i)      (recomputed from the forward LSE)
//   dV_j  = sum_i P_ij dO_i
//   dP_ij = dO_i . v_j,   D_i = dO_i . O_i
//   dS_ij = P_ij (dP_ij - D_i)
//   dQ_i  = scale sum_j dS_ij k_j,   dK_j = scale sum_i dS_ij q_i
// Four kernels:
//   bwd_prep   D per (row, head); zero the fp32 dK / dV accumulators
//   bwd_dq     query-major: the forward's work items (256 columns x the
//              item's key ranges); per 64-key tile S^T, dP^T, dS^T and
//              dQ^T += K^T dS^T; dQ is complete per item and written directly
//   bwd_dkdv   key-major: up to 128 keys of one segment against the query
//              columns that see them, 32 columns per step; waves 4-7 compute
//              S and P for 32 keys each and dK^T += Q^T dS, waves 0-3
//              dV^T += dO^T P for the same keys with P handed over through
//              LDS; results go to fp32 rows (stored by an item that holds the
//              whole run, added by the pieces of a split run)
//   bwd_finalize  fp32 accumulators -> bf16 dK, dV (round to nearest even)
// All products are v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  An
// operand whose contraction index is not contiguous in memory (K^T for dQ,
// dO^T and Q^T for dV and dK) is read from its row-major LDS block with the
// transposing LDS read of gfx950 (within each group of 16 lanes, lane r
// supplies the address of 4 consecutive elements and lane 4a+b receives
// element b of the pieces of lanes a, 4+a, 8+a and 12+a), two reads per
// operand, in the key / column order of the probabilities' registers.
#include <algorithm>

#include "device_common.hpp"
#include "tile_common.hpp"

namespace padoc {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& u) { return *reinterpret_cast<const bf16x8_t*>(&u); }

// Row-major LDS blocks of CPR 16-byte chunks per row store chunk c of row r
// at chunk c ^ sw(r): the row reads of the matrix products (16 rows, one
// chunk) and the transposing reads (4 rows, 4 aligned chunks) then each
// touch distinct banks.  CPR = 16 (d = 128): one row per 256-byte bank row;
// CPR = 8 (d = 64): two rows per bank row, so the swizzle keys on the row
// pair.
template <int CPR>
__device__ __forceinline__ int swizzled_chunk(int r, int c) {
  const int sw = CPR == 16 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
  return c ^ sw;
}

// ------------------------------------------------------------------ prep

template <int D>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdParams p, int64_t n_rows, int64_t n_acc4) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n_rows; r += nwaves) {
    const uint16_t* o = static_cast<const uint16_t*>(p.o) + r * D;
    const uint16_t* g = static_cast<const uint16_t*>(p.dout) + r * D;
    float acc = 0.f;
#pragma unroll
    for (int e = lane; e < D; e += 64) acc = fmaf(bf16_bits_to_f32(o[e]), bf16_bits_to_f32(g[e]), acc);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m);
    if (lane == 0) p.dd[r] = acc;
  }
  const int64_t nth = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_acc4; i += nth) {
    reinterpret_cast<float4*>(p.dk_acc)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    reinterpret_cast<float4*>(p.dv_acc)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// ------------------------------------------------------------------ dQ

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_dq_kernel(BwdParams p) {
  constexpr int KT = kTileKeys;  // 64 keys per tile
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int CPR = D / 8;
  constexpr int KPT = KT * CPR / kThreads;  // row pieces per thread (2 or 1)

  // K and V tiles: KT rows of D elements with swizzled 16-byte chunks (see
  // swizzled_chunk), read by rows for S and dP and transposed (K^T) for dQ.
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KT * D];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[KT * D];
  auto at = [&](int r, int c) { return r * D + (swizzled_chunk<CPR>(r, c) << 3); };

  const WorkRec w = p.work[blockIdx.x];
  if (w.rng_count <= 0) return;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int G = p.G, kvh = w.kvh;
  const int64_t Hkv = p.Hkv;
  const int col = wave * 32 + l32;
  const int tok = col / G;
  const bool valid = tok < w.ntok;
  const int32_t qrow = valid ? p.toks[w.tok_begin + tok] : 0;
  const int32_t hq = kvh * G + (col - tok * G);
  const int64_t qoff = ((int64_t)qrow * p.Hq + hq) * D;

  bf16x8_t bq[NKK], bdo[NKK];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(p.q) + qoff + hf * 8;
    const uint16_t* gp = static_cast<const uint16_t*>(p.dout) + qoff + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      bq[kk] = as_bf16x8(valid ? load16(qp + kk * 16) : make_uint4(0, 0, 0, 0));
      bdo[kk] = as_bf16x8(valid ? load16(gp + kk * 16) : make_uint4(0, 0, 0, 0));
    }
  }
  const float lse2 = valid ? p.lse[(int64_t)qrow * p.Hq + hq] * kLog2e : 0.f;
  const float dcol = valid ? p.dd[(int64_t)qrow * p.Hq + hq] : 0.f;
  const float sl2 = p.scale_log2;

  const uint16_t* Kg = static_cast<const uint16_t*>(p.k);
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v);
  // row pieces (key, 16-byte chunk)
  int r_key[KPT], r_dc[KPT];
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int u = tid + kThreads * i;
    r_key[i] = u / CPR;
    r_dc[i] = u % CPR;
  }

  struct Cursor {
    int ri, kt;
    RangeRec R;
    int ok, unused;
  };
  auto advance = [&](Cursor& c) {
    if (++c.kt * KT >= c.R.n_keys) {
      c.kt = 0;
      if (++c.ri < w.rng_count)
        c.R = p.ranges[w.rng_begin + c.ri];
      else
        c.ok = 0;
    }
  };
  uint4 kr[KPT], vr[KPT];
  // Tile loads: rows past the range end repeat its last row (finite values
  // whose scores the mask removes).
  auto load = [&](const Cursor& c) {
    const int kbase = c.kt * KT, last = c.R.n_keys - 1 - kbase;
    const int64_t row0 = c.R.kv_start + kbase;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int kc = r_key[i] <= last ? r_key[i] : last;
      const int64_t off = ((row0 + kc) * Hkv + kvh) * D + r_dc[i] * 8;
      kr[i] = load16(Kg + off);
      vr[i] = load16(Vg + off);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      store16(&Ks[at(r_key[i], r_dc[i])], kr[i]);
      store16(&Vs[at(r_key[i], r_dc[i])], vr[i]);
    }
  };
  // K^T operand of dQ^T += K^T dS^T for keys mb*32 + 16j + 4*half + {0..3},
  // {8..11} and d block db: two transposing reads (lane r of a 16-lane group
  // supplies key row .. + r/4, elements d0 + 4*(r%4) .. +3)
  const int tr_r = (lane & 15) >> 2, tr_c = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1), tr_o = 4 * (lane & 1);
  auto ktf = [&](int mb, int j, int db) __attribute__((always_inline)) -> bf16x8_t {
    const int r0 = mb * 32 + 16 * j + 4 * hf + tr_r, c = 4 * db + tr_c;
    return tile::tr_pair(Ks + at(r0, c) + tr_o, Ks + at(r0 + 8, c) + tr_o);
  };
  auto lim_of = [&](const RangeRec& R) -> int {
    return R.lim_off < 0 ? R.n_keys : (valid ? p.lims[R.lim_off + tok] : 0);
  };

  f32x16_t acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = 0.f;

  Cursor C{0, 0, p.ranges[w.rng_begin], 1, 0};
  Cursor L = C;
  load(L);
  advance(L);
  int lim = lim_of(C.R);
  for (;;) {
    store();
    __syncthreads();
    if (L.ok) load(L);  // next tile, in flight during this one
    const int kb = C.kt * KT;
    const bool partial = kb + KT > C.R.min_lim;
    const int rel = lim - kb - hf * 4;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      f32x16_t S, dP;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        S[i] = 0.f;
        dP[i] = 0.f;
      }
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        const int off = at(mb * 32 + l32, 2 * kk + hf);
        S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8_t*>(&Ks[off]), bq[kk], S, 0, 0, 0);
        dP = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8_t*>(&Vs[off]), bdo[kk], dP, 0, 0, 0);
      }
      // element i: key mb*32 + (i/4)*8 + hf*4 + i%4 of the tile, this lane's column
      bf16x8_t ds[2];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const bool vis = !partial || mb * 32 + (i >> 2) * 8 + (i & 3) < rel;
        const float pr = vis ? fast_exp2(fmaf(S[i], sl2, -lse2)) : 0.f;
        ds[i >> 3][i & 7] = (__bf16)(pr * (dP[i] - dcol));
      }
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ktf(mb, j, db), ds[j], acc[db], 0, 0, 0);
        }
    }
    __syncthreads();
    const int ri_before = C.ri;
    advance(C);
    if (!C.ok) break;
    if (C.ri != ri_before) lim = lim_of(C.R);
    advance(L);
  }

  if (!valid) return;
  const float sc = p.scale;
  uint16_t* op = static_cast<uint16_t*>(p.dq) + qoff;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i4 = 0; i4 < 4; ++i4) {
      const int d0 = db * 32 + i4 * 8 + hf * 4;
      uint2 pk;
      pk.x = (uint32_t)f32_to_bf16_bits(acc[db][4 * i4] * sc) | ((uint32_t)f32_to_bf16_bits(acc[db][4 * i4 + 1] * sc) << 16);
      pk.y = (uint32_t)f32_to_bf16_bits(acc[db][4 * i4 + 2] * sc) |
             ((uint32_t)f32_to_bf16_bits(acc[db][4 * i4 + 3] * sc) << 16);
      *reinterpret_cast<uint2*>(op + d0) = pk;
    }
}

// ------------------------------------------------------------------ dK, dV

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_dkdv_kernel(BwdParams p) {
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int CPR = D / 8;
  // Q / dO blocks: 32 rows of D elements with swizzled 16-byte chunks
  auto at = [&](int r, int c) { return r * D + (swizzled_chunk<CPR>(r, c) << 3); };

  // Two stages: block i is computed from stage i%2 while block i+1 is stored
  // into the other one (one barrier per block).
  struct Stage {
    uint16_t q[32 * D];  // Q rows (row = column of the block), swizzled chunks
    uint16_t g[32 * D];  // dO rows
    float ls[32];         // LSE * log2(e) per column
    float dd[32];         // dO . O per column
    int lm[32];           // keys of the item the column sees
  };
  __shared__ __attribute__((aligned(16))) Stage st[2];
  // P of the block in bf16 per key group (wave & 3), as the dK wavefront's
  // lanes hold it: [group][j][lane][8]
  __shared__ __attribute__((aligned(16))) __bf16 Psh[4][2][64 * 8];

  const BwdRec b = p.bwd[blockIdx.x];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const bool kwave = wave >= 4;          // waves 4-7: dK; 0-3: dV
  const int key = (wave & 3) * 32 + l32;  // this lane's key within the item
  const int key_hi = (wave & 3) * 32 + 32;  // end of this wavefront's keys
  const int G = p.G, kvh = b.kvh;
  const int64_t Hkv = p.Hkv;

  // B operands of S = Q K^T and dP = dO V^T: this lane's key, d = kk*16 + hf*8 ..
  bf16x8_t bk[NKK], bv[NKK];
  {
    const int kc = key < b.n_keys ? key : b.n_keys - 1;
    const int64_t off = ((b.key_row0 + kc) * Hkv + kvh) * D + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      bk[kk] = as_bf16x8(load16(static_cast<const uint16_t*>(p.k) + off + kk * 16));
      bv[kk] = as_bf16x8(kwave ? load16(static_cast<const uint16_t*>(p.v) + off + kk * 16) : make_uint4(0, 0, 0, 0));
    }
  }

  // Staging geometry: thread -> (column, 16-byte chunk) of a 32-column block,
  // columns fastest (16 lanes of a store write 16 rows of one chunk, which
  // the swizzle spreads over all banks); with d = 64 the upper half of the
  // threads repeats the lower half's loads and stores nothing.  Every thread
  // also loads the per-column scalars of column tid % 32 (threads < 32 store
  // them), so all threads issue the same loads and the compiler's load wait
  // counts stay exact.
  const int s_col = tid % 32, s_dc = (tid / 32) % CPR;
  const bool s_on = tid < 32 * CPR;
  const int c_end = b.col0 + b.ncol;
  // Register sets [i % 2]: Q / dO pieces and column scalars of a block
  // loaded two blocks ahead of its LDS store; the Q rows of its columns are
  // fetched one block before that.
  uint4 qr[2], gr[2];
  float lr[2], dr[2];
  int mr[2];
  // Per set: Q row, token within the item and head of this thread's column
  // (column tid % 32 of the block; past c_end: the last column, flagged).
  int rq[2], tq[2], hq[2];
  bool okq[2];
  // fetch_rows visits the blocks in order, 32 columns apart: the column's
  // (token, head) = (column / G, column % G) advances by (32 / G, 32 % G)
  // with one carry, so no division runs per block.
  int f_col = b.col0 + s_col, f_t = f_col / G, f_h = f_col % G;
  const int t32 = 32 / G, h32 = 32 % G;
  const int t_end = (c_end - 1) / G, h_end = (c_end - 1) % G;
  auto fetch_rows = [&](auto xc) __attribute__((always_inline)) {
    constexpr int X = decltype(xc)::value;
    const bool ok = f_col < c_end;
    tq[X] = ok ? f_t : t_end;
    hq[X] = ok ? f_h : h_end;
    okq[X] = ok;
    rq[X] = p.btoks[b.tok_begin + tq[X]];
    f_col += 32;
    f_t += t32;
    f_h += h32;
    if (f_h >= G) {
      f_h -= G;
      ++f_t;
    }
  };
  // A column past c_end carries the last column's (finite) Q, dO, LSE and
  // D with a limit of 0: its P and dS are exactly 0, so it adds nothing.
  auto load = [&](auto xc) __attribute__((always_inline)) {
    constexpr int X = decltype(xc)::value;
    const int64_t rh = (int64_t)rq[X] * p.Hq + kvh * G + hq[X];
    const int64_t off = rh * D + s_dc * 8;
    qr[X] = load16(static_cast<const uint16_t*>(p.q) + off);
    gr[X] = load16(static_cast<const uint16_t*>(p.dout) + off);
    lr[X] = p.lse[rh] * kLog2e;
    dr[X] = p.dd[rh];
    const int m = p.blims[b.lim_begin + tq[X]];
    mr[X] = okq[X] ? m : 0;
  };
  auto store = [&](auto xc, Stage& S) {
    constexpr int X = decltype(xc)::value;
    if (s_on) {
      store16(&S.q[at(s_col, s_dc)], qr[X]);
      store16(&S.g[at(s_col, s_dc)], gr[X]);
    }
    if (tid < 32) {
      S.ls[tid] = lr[X];
      S.dd[tid] = dr[X];
      S.lm[tid] = mr[X];
    }
  };

  f32x16_t acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = 0.f;
  const float sl2 = p.scale_log2;

  // A operand d x columns (Q^T or dO^T) of d block db and column group j:
  // lane (d, half) gets columns 16j + 4*half + {0..3} and + {8..11} of row
  // d, with two transposing reads (lane r of a 16-lane group supplies row
  // 16j + 4*half (+8) + r/4, elements d0 + 4*(r%4) .. +3).
  const int tr_r = (lane & 15) >> 2, tr_c = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1), tr_o = 4 * (lane & 1);
  auto trf = [&](const uint16_t* blk, int j, int db) __attribute__((always_inline)) -> bf16x8_t {
    const int r0 = 16 * j + 4 * hf + tr_r, c = 4 * db + tr_c;
    return tile::tr_pair(blk + at(r0, c) + tr_o, blk + at(r0 + 8, c) + tr_o);
  };

  // Block computation from one stage.  The dK wavefront of each key group
  // (wave w + 4) computes S and P and hands P (bf16, in its score registers'
  // layout) to the dV wavefront of the same keys (wave w) through LDS; the
  // dV wavefront reads it after the block's first barrier, so S and the
  // exponentials run once per key group.  Fragments of each product group
  // are requested together before its matrix products.
  auto compute = [&](const Stage& S) __attribute__((always_inline)) {
    bf16x8_t fa[NKK];
    bf16x8_t fb[2 * NDB];
    float pr[16];
    if (kwave) {
      // S = Q K^T: columns on M, this wave's 32 keys on N.  Element i of a
      // lane is column (i/4)*8 + hf*4 + i%4 of the block and key `key`.
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) fa[kk] = *reinterpret_cast<const bf16x8_t*>(&S.q[at(l32, 2 * kk + hf)]);
      f32x16_t sc;
#pragma unroll
      for (int i = 0; i < 16; ++i) sc[i] = 0.f;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk], bk[kk], sc, 0, 0, 0);
      // P = exp(S - LSE), zero past each column's limit.  When every column
      // of the block sees all 32 keys of this wavefront (limits are at most
      // n_keys, so the keys are real), the mask is skipped.
      float lv[16];
      int mv[16];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int cb = q4 * 8 + hf * 4;  // columns cb .. cb+3 = elements 4*q4 .. 4*q4+3
        const float4 l4 = *reinterpret_cast<const float4*>(&S.ls[cb]);
        const int4 m4 = *reinterpret_cast<const int4*>(&S.lm[cb]);
        lv[4 * q4] = l4.x, lv[4 * q4 + 1] = l4.y, lv[4 * q4 + 2] = l4.z, lv[4 * q4 + 3] = l4.w;
        mv[4 * q4] = m4.x, mv[4 * q4 + 1] = m4.y, mv[4 * q4 + 2] = m4.z, mv[4 * q4 + 3] = m4.w;
      }
      int mn = mv[0];
#pragma unroll
      for (int i = 1; i < 16; ++i) mn = min(mn, mv[i]);
      mn = min(mn, __shfl_xor(mn, 32));  // lanes l and l^32 hold the other 16 columns
      if (__builtin_amdgcn_readfirstlane((int)(mn >= key_hi))) {
#pragma unroll
        for (int i = 0; i < 16; ++i) pr[i] = fast_exp2(fmaf(sc[i], sl2, -lv[i]));
      } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) pr[i] = key < mv[i] ? fast_exp2(fmaf(sc[i], sl2, -lv[i])) : 0.f;
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        bf16x8_t pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = (__bf16)pr[8 * j + e];
        *reinterpret_cast<bf16x8_t*>(&Psh[wave & 3][j][lane * 8]) = pb;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          fb[j * NDB + db] = trf(S.g, j, db);
    }
    __syncthreads();  // P of this block is in Psh
    if (!kwave) {
      // dV^T += dO^T P: d on M (block db), keys on N, columns on K
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8_t pb = *reinterpret_cast<const bf16x8_t*>(&Psh[wave][j][lane * 8]);
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j * NDB + db], pb, acc[db], 0, 0, 0);
      }
    } else {
      // dP = dO V^T; dS = P (dP - D); dK^T += Q^T dS
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) fa[kk] = *reinterpret_cast<const bf16x8_t*>(&S.g[at(l32, 2 * kk + hf)]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          fb[j * NDB + db] = trf(S.q, j, db);
      f32x16_t dP;
#pragma unroll
      for (int i = 0; i < 16; ++i) dP[i] = 0.f;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) dP = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk], bv[kk], dP, 0, 0, 0);
      float dsv[16];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 d4 = *reinterpret_cast<const float4*>(&S.dd[q4 * 8 + hf * 4]);
        const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) dsv[4 * q4 + e] = pr[4 * q4 + e] * (dP[4 * q4 + e] - dv[e]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        bf16x8_t sb;
#pragma unroll
        for (int e = 0; e < 8; ++e) sb[e] = (__bf16)dsv[8 * j + e];
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j * NDB + db], sb, acc[db], 0, 0, 0);
      }
    }
  };

  // Block i is computed from stage i % 2 and its pieces sit in register set
  // i % 2 until stored (at step i-1); step i stores block i+1, loads block
  // i+2 into set i % 2 and fetches the rows of block i+3 into row set
  // (i+1) % 2.
  using Set0 = std::integral_constant<int, 0>;
  using Set1 = std::integral_constant<int, 1>;
  fetch_rows(Set0{});  // block 0
  load(Set0{});
  fetch_rows(Set1{});  // block 1
  load(Set1{});
  store(Set0{}, st[0]);
  fetch_rows(Set0{});  // block 2
  __syncthreads();
  auto step = [&](auto xc, int c0) {
    constexpr int X = decltype(xc)::value;
    using Y = std::integral_constant<int, X ^ 1>;
    compute(st[X]);
    if (c0 + 32 < c_end) store(Y{}, st[X ^ 1]);  // that stage was last read before the previous barrier
    load(xc);           // block i+2
    fetch_rows(Y{});    // block i+3
    __syncthreads();
  };
  for (int c0 = b.col0;;) {
    step(Set0{}, c0);
    c0 += 32;
    if (c0 >= c_end) break;
    step(Set1{}, c0);
    c0 += 32;
    if (c0 >= c_end) break;
  }

  if (key >= b.n_keys) return;
  // acc[db] element i: d = db*32 + (i/4)*8 + hf*4 + i%4, key `key`.  An item
  // that holds all of its key run's columns stores its rows; the pieces of a
  // split run add into them (rows start at zero).
  float* dst = (kwave ? p.dk_acc : p.dv_acc) + ((b.key_row0 + key) * Hkv + kvh) * D;
  const float sc = kwave ? p.scale : 1.f;
  if (b.col0 == 0 && b.ncol == b.ntok * G) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4)
        *reinterpret_cast<float4*>(dst + db * 32 + i4 * 8 + hf * 4) =
            make_float4(acc[db][4 * i4] * sc, acc[db][4 * i4 + 1] * sc, acc[db][4 * i4 + 2] * sc,
                        acc[db][4 * i4 + 3] * sc);
  } else {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) atomicAdd(dst + db * 32 + (i >> 2) * 8 + hf * 4 + (i & 3), acc[db][i] * sc);
  }
}

// ------------------------------------------------------------------ finalize

__global__ __launch_bounds__(256) void bwd_finalize_kernel(BwdParams p, int64_t n4) {
  const int64_t nth = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += nth) {
    const float4 a = reinterpret_cast<const float4*>(p.dk_acc)[i];
    const float4 c = reinterpret_cast<const float4*>(p.dv_acc)[i];
    uint2 ka, va;
    ka.x = (uint32_t)f32_to_bf16_bits(a.x) | ((uint32_t)f32_to_bf16_bits(a.y) << 16);
    ka.y = (uint32_t)f32_to_bf16_bits(a.z) | ((uint32_t)f32_to_bf16_bits(a.w) << 16);
    va.x = (uint32_t)f32_to_bf16_bits(c.x) | ((uint32_t)f32_to_bf16_bits(c.y) << 16);
    va.y = (uint32_t)f32_to_bf16_bits(c.z) | ((uint32_t)f32_to_bf16_bits(c.w) << 16);
    reinterpret_cast<uint2*>(p.dk)[i] = ka;
    reinterpret_cast<uint2*>(p.dv)[i] = va;
  }
}

}  // namespace

hipError_t launch_tree_attn_bwd(const BwdParams& p, int n_work, int n_bwd, int D, hipStream_t stream) {
  const int64_t n_rows = p.n_q * p.Hq;
  const int64_t n_acc4 = p.T * p.Hkv * D / 4;
  const int64_t want = (std::max(n_rows / 4, n_acc4 / 256) + 1);
  const dim3 prep_grid((unsigned)std::min<int64_t>(want, 4096)), blk256(256), blk512(kThreads);
  if (D == 64)
    hipLaunchKernelGGL((bwd_prep_kernel<64>), prep_grid, blk256, 0, stream, p, n_rows, n_acc4);
  else
    hipLaunchKernelGGL((bwd_prep_kernel<128>), prep_grid, blk256, 0, stream, p, n_rows, n_acc4);
  if (n_work > 0) {
    if (D == 64)
      hipLaunchKernelGGL((bwd_dq_kernel<64>), dim3(n_work), blk512, 0, stream, p);
    else
      hipLaunchKernelGGL((bwd_dq_kernel<128>), dim3(n_work), blk512, 0, stream, p);
  }
  if (n_bwd > 0) {
    if (D == 64)
      hipLaunchKernelGGL((bwd_dkdv_kernel<64>), dim3(n_bwd), blk512, 0, stream, p);
    else
      hipLaunchKernelGGL((bwd_dkdv_kernel<128>), dim3(n_bwd), blk512, 0, stream, p);
  }
  if (n_acc4 > 0) {
    const dim3 fin_grid((unsigned)std::min<int64_t>(n_acc4 / 256 + 1, 4096));
    hipLaunchKernelGGL(bwd_finalize_kernel, fin_grid, blk256, 0, stream, p, n_acc4);
  }
  return hipGetLastError();
}

}  // namespace padoc

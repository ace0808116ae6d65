// bf16 tile computation for gfx950 (CDNA4) matrix cores: one work item --
// of the packed forward, or of the shared-key part of a decode step (paged
// K/V, split partials) -- on the 8 wavefronts of a 512-thread workgroup
// (the kernels are in tile_mfma_bf16.hip).
//
// An item is up to 256 columns (query token x head of one KV-head group: the
// G heads of a token share every K/V tile) against the item's key ranges, 64
// keys per tile.  K tiles are staged row-major and V tiles transposed in a
// two-stage LDS ring with one barrier per tile; a tile's global loads are
// issued two tiles before its LDS store (two staging register sets).  Each
// wavefront owns 32 columns and, per tile:
//   S^T = K Q^T         v_mfma_f32_32x32x16_bf16, keys on M, columns on N
//                       (a lane owns one column and 16 of 32 key rows of a
//                       half; the other 16 rows sit in lane^32), both 32-key
//                       halves issued back to back
//   online softmax      per half: half 0's runs while half 1's products are
//                       in flight, half 1's while half 0's PV products run
//   O^T += V^T P^T      P^T comes straight from the score registers
// (App. E Attn equation; App. C tree-varlen relation).  Only tiles of
// ancestor prefixes and the own causal range are visited: the planner lists
// no other segment.  Tiles wholly below every column's limit skip the mask.
// Keys past a range's end never contribute: their K/V rows are copies of the
// range's last row (finite), their scores are masked to -inf, and paged V
// chunks past the end are zeroed in LDS, so no stale or sentinel memory
// enters a product.
//
// Accumulation is fp32 and scores are in log2 units, so each probability is
// one v_exp_f32; the softmax denominator sums the bf16-rounded probabilities
// that enter the PV product, so O is their exact weighted mean.  The
// reference maximum of a column is raised only when a half's maximum exceeds
// it by more than 2^8 (probabilities stay <= 256); the accumulator is
// rescaled only then.  Any reference gives the same O and LSE.  O is rounded
// to bf16 (RNE) at the end.
//
// Paged K/V: K blocks are chunk-major ([d/8][16 slots][8]) and land in the
// row-major LDS tile piece by piece; V blocks are d-major ([d][16 tokens]),
// so a 16-byte load holds 8 consecutive keys of one d row and lands in the
// transposed LDS tile as two 8-byte stores.  A tile's block ids come from one
// vector load issued a tile ahead of its K/V loads.
#pragma once

#include <type_traits>

#include "device_common.hpp"

namespace padoc {
namespace tile {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kStages = 2;
constexpr float kRescaleSlack = 8.0f;  // log2 units: probabilities <= 2^8

// Position of key r (0..63) inside a transposed V row.  Within each group of
// 16 keys, lane half 0 of the 32x32 P^T fragment holds keys
// {0,1,2,3,8,9,10,11} and half 1 holds {4..7,12..15}; storing them in that
// order makes each half's 8 keys one contiguous 16-byte LDS read.
__device__ __forceinline__ int vt_pos(int r) {
  const int q = r & 15;
  return (r & ~15) + ((q >> 2) & 1) * 8 + (q >> 3) * 4 + (q & 3);
}

__device__ __forceinline__ int64_t uniform64(int64_t x) {
  return (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(x >> 32)) << 32) |
                   (uint32_t)__builtin_amdgcn_readfirstlane((int)x));
}

__device__ __forceinline__ RangeRec uniform_range(RangeRec r) {
  r.kv_start = uniform64(r.kv_start);
  r.n_keys = __builtin_amdgcn_readfirstlane(r.n_keys);
  r.min_lim = __builtin_amdgcn_readfirstlane(r.min_lim);
  r.lim_off = __builtin_amdgcn_readfirstlane(r.lim_off);
  return r;
}

// One work item (up to 256 columns) on the 8 wavefronts of a workgroup.
template <int D, bool PAGED, bool PARTIAL>
__device__ __forceinline__ void tile_item(const TileParams& p, int item) {
  constexpr int KT = kTileKeys;  // 64 keys per tile
  constexpr int KS = D + 8;      // K row stride in LDS (elements); +8 spreads banks
  constexpr int VS = KT + 8;     // V^T row stride in LDS
  constexpr int NKK = D / 16;    // K-slices of the score product
  constexpr int NDB = D / 32;    // 32-row blocks of O^T
  constexpr int CPR = D / 8;     // 16-byte chunks per key row
  constexpr int KPT = KT * CPR / kThreads;           // K chunks per thread (2 or 1)
  constexpr int VPT = PAGED ? 8 * D / kThreads : 1;  // V loads per thread (paged chunks / packed pairs)
  constexpr int NB = KT / kBlock;                    // blocks per tile (paged)

  __shared__ __attribute__((aligned(16))) uint16_t Ks[kStages][KT * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kStages][D * VS];

  const WorkRec w = p.work[item];
  if (w.rng_count <= 0) return;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int G = p.G;
  const int kvh = w.kvh;
  const int64_t Hkv = p.Hkv;

  // This lane's column.
  const int col = wave * 32 + l32;
  const int tok = col / G;
  const bool valid = tok < w.ntok;
  const int32_t qrow = valid ? p.toks[w.tok_begin + tok] : 0;
  const int32_t hq = kvh * G + (col - tok * G);

  // Q fragments (B operand of S^T = K Q^T): d = kk*16 + hf*8 .. +7.
  bf16x8_t bq[NKK];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(p.q) + ((int64_t)qrow * p.Hq + hq) * D + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const uint4 z = valid ? *reinterpret_cast<const uint4*>(qp + kk * 16) : make_uint4(0, 0, 0, 0);
      bq[kk] = *reinterpret_cast<const bf16x8_t*>(&z);
    }
  }

  const uint16_t* Kg = static_cast<const uint16_t*>(p.k);
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v);

  // Per-thread load geometry (independent of the tile).
  // K piece u (16 bytes): packed K rows are read row by row; paged K blocks
  // are chunk-major, so consecutive threads take consecutive slots of one
  // chunk (token kslot(slot)).  Either way a wave reads 1 KB contiguous.
  int k_key[KPT], k_dc[KPT];
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int u = tid + kThreads * i;
    if constexpr (PAGED) {
      const int bi = u / (kBlock * CPR), rem = u % (kBlock * CPR);
      k_key[i] = bi * kBlock + kslot(rem % kBlock);
      k_dc[i] = rem / kBlock;
    } else {
      k_key[i] = u / CPR;
      k_dc[i] = u % CPR;
    }
  }
  // packed V: key pair (2pr, 2pr+1) and 16-byte chunk dc (threads >= 32*CPR idle)
  const int v_pr = tid % (KT / 2), v_dc = tid / (KT / 2);
  const bool v_on = PAGED || v_dc < CPR;

  // Two staging register sets: a tile's global loads are issued two
  // iterations before its LDS store.
  uint4 kr[2][KPT], vr[2][2 * VPT];
  int vkeep[2][PAGED ? VPT : 1];  // paged V: keys of each chunk inside the range

  // Block ids of a tile: lane l (mod NB) loads the id of block l with a
  // vector load.  Scalar loads would share the LDS wait counter (and return
  // out of order), so every LDS wait would also wait for the block table.
  auto fetch_idv = [&](const RangeRec& R, int kt) -> int {
    const int kbase = kt * KT, bi = lane & (NB - 1);
    return p.block_table[R.kv_start + (kbase >> 4) + ((kbase + bi * kBlock < R.n_keys) ? bi : 0)];
  };
  // Global -> registers, branch-free.  Rows past the range end are read from
  // the range's last row (finite data whose scores the mask removes); paged
  // V chunks, which may reach into unwritten slots, are zeroed past the end
  // when they are stored, a tile later, so no load is waited for early.
  auto load_tile = [&](auto xc, const RangeRec& R, int kt, int idv) {
    constexpr int X = decltype(xc)::value;
    int64_t ids[NB] = {};
    if constexpr (PAGED) {
#pragma unroll
      for (int bi = 0; bi < NB; ++bi) ids[bi] = __builtin_amdgcn_readlane(idv, bi);
    }
    const int kbase = kt * KT;
    const int last = R.n_keys - 1 - kbase;  // >= 0
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int key = k_key[i];
      const int kc = key <= last ? key : last;
      const uint4 x = PAGED ? load_stream16(Kg + paged_k_offset<D>(ids[kc >> 4], kvh, (int32_t)Hkv, kc & 15, k_dc[i]))
                            : *reinterpret_cast<const uint4*>(Kg + ((R.kv_start + kbase + kc) * Hkv + kvh) * (int64_t)D +
                                                              k_dc[i] * 8);
      kr[X][i] = x;
    }
    if constexpr (PAGED) {
#pragma unroll
      for (int i = 0; i < VPT; ++i) {
        const int u = tid + kThreads * i;
        const int bi = u / (2 * D), rem = u % (2 * D);
        const int d = rem >> 1, h = rem & 1;
        const int keep = R.n_keys - (kbase + bi * kBlock + h * 8);
        const int64_t blk = ids[keep > 0 ? bi : 0];
        vr[X][i] = load_stream16(Vg + ((blk * Hkv + kvh) * D + d) * kBlock + h * 8);
        vkeep[X][i] = keep;
      }
    } else {
      if (v_on) {
        const int k0 = 2 * v_pr, k1 = k0 + 1;
        const int c0 = k0 <= last ? k0 : last, c1 = k1 <= last ? k1 : last;
        const uint4 x0 = *reinterpret_cast<const uint4*>(Vg + ((R.kv_start + kbase + c0) * Hkv + kvh) * D + v_dc * 8);
        const uint4 x1 = *reinterpret_cast<const uint4*>(Vg + ((R.kv_start + kbase + c1) * Hkv + kvh) * D + v_dc * 8);
        vr[X][0] = x0;
        vr[X][1] = x1;
      }
    }
  };
  auto store_tile = [&](auto xc, int s) {
    constexpr int X = decltype(xc)::value;
#pragma unroll
    for (int i = 0; i < KPT; ++i) *reinterpret_cast<uint4*>(&Ks[s][k_key[i] * KS + k_dc[i] * 8]) = kr[X][i];
    if constexpr (PAGED) {
#pragma unroll
      for (int i = 0; i < VPT; ++i) {
        const int u = tid + kThreads * i;
        const int bi = u / (2 * D), rem = u % (2 * D);
        const int d = rem >> 1, h = rem & 1;
        // keys 8h..8h+3 of block bi -> positions 4h..4h+3, keys 8h+4..8h+7 -> 8+4h..
        uint16_t* row = &Vt[s][d * VS + bi * 16];
        const uint4 x = keep_first(vr[X][i], vkeep[X][i]);
        *reinterpret_cast<uint2*>(row + 4 * h) = make_uint2(x.x, x.y);
        *reinterpret_cast<uint2*>(row + 8 + 4 * h) = make_uint2(x.z, x.w);
      }
    } else if (v_on) {
      const int pos = vt_pos(2 * v_pr);
      const uint32_t a[4] = {vr[X][0].x, vr[X][0].y, vr[X][0].z, vr[X][0].w};
      const uint32_t b[4] = {vr[X][1].x, vr[X][1].y, vr[X][1].z, vr[X][1].w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        // d = dc*8 + 2m holds (key 2pr, key 2pr+1) low halves; d+1 the high halves
        *reinterpret_cast<uint32_t*>(&Vt[s][(v_dc * 8 + 2 * m) * VS + pos]) = (a[m] & 0xffffu) | (b[m] << 16);
        *reinterpret_cast<uint32_t*>(&Vt[s][(v_dc * 8 + 2 * m + 1) * VS + pos]) = (a[m] >> 16) | (b[m] & 0xffff0000u);
      }
    }
  };

  // Tile cursors (wave-uniform): C = tile being computed, L = next to load.
  // No implicit padding: copies of a padded struct keep the padding in
  // memory (the compiler would place it in LDS).
  struct Cursor {
    int ri, kt;
    RangeRec R;
    int ok, unused;
  };
  auto advance = [&](Cursor& c) {
    if (++c.kt * KT >= c.R.n_keys) {
      c.kt = 0;
      if (++c.ri < w.rng_count)
        c.R = uniform_range(p.ranges[__builtin_amdgcn_readfirstlane(w.rng_begin + c.ri)]);  // scalar loads
      else
        c.ok = 0;
    }
  };
  Cursor C{0, 0, uniform_range(p.ranges[w.rng_begin]), 1, 0};
  Cursor L = C;
  // This column's limit entry for a cursor's range: one unconditional load
  // (of a valid int when the range has no limits), interpreted only in the
  // mask.  Loads are never skipped or copied right after being issued, so
  // the compiler's wait counts stay exact across iterations.
  auto fetch_lim = [&](int32_t lim_off) -> int {
    const int32_t* lp = lim_off < 0 ? &p.work[item].ntok : p.lims + lim_off + (valid ? tok : 0);
    return *lp;
  };
  int limr[2];  // [t % 2]: limit entry of tile t's range
  limr[0] = fetch_lim(C.R.lim_off);

  float m_run = -INFINITY, l_run = 0.f;
  f32x16_t acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = 0.f;
  const float sl2 = p.scale_log2;

  // Prologue: tile 0 into LDS stage 0, tiles 1 and 2 into register sets 0
  // and 1.  Tile t lives in stage t % 2.
  using Set0 = std::integral_constant<int, 0>;
  using Set1 = std::integral_constant<int, 1>;
  // load_next(X) loads L's tile into staging set X using the block ids in
  // idv[X^1] and requests the ids of the tile after it into idv[X] first, so
  // waiting for ids never waits for the newest tile's data.  Past the item's
  // last tile the loader re-reads a valid tile of its last range (not
  // staged), so every iteration issues the same loads.
  int idv[2] = {0, 0};
  bool staged[2] = {false, false};  // register set holds a loaded tile not yet in LDS
  auto load_next = [&](auto xc) {
    constexpr int X = decltype(xc)::value;
    const bool real = L.ok;
    Cursor nx = L;
    advance(nx);
    if constexpr (PAGED) idv[X] = fetch_idv(nx.R, nx.kt);
    load_tile(xc, L.R, L.kt, idv[X ^ 1]);
    L = nx;
    staged[X] = real;
  };
  if constexpr (PAGED) idv[0] = fetch_idv(L.R, L.kt);
  load_next(Set1{});  // tile 0 (set 1, ids in idv[0])
  store_tile(Set1{}, 0);
  staged[1] = false;
  load_next(Set0{});  // tile 1
  load_next(Set1{});  // tile 2
  __syncthreads();

  // O^T += V^T P^T, 16 keys per MFMA: key group g = (mb, j) holds keys
  // mb*32 + 16j + [0,16).
  auto vfrag = [&](const uint16_t* vt, int g, bf16x8_t (&a)[NDB]) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      a[db] = *reinterpret_cast<const bf16x8_t*>(&vt[(db * 32 + l32) * VS + (g >> 1) * 32 + 16 * (g & 1) + hf * 8]);
  };
  // PV products of half mb (key groups 2mb and 2mb+1).
  auto pv_half = [&](const uint16_t* vt, int mb, const bf16x8_t (&P)[2][2]) {
    bf16x8_t vf0[NDB], vf1[NDB];
    vfrag(vt, 2 * mb, vf0);
    vfrag(vt, 2 * mb + 1, vf1);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf0[db], P[mb][0], acc[db], 0, 0, 0);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf1[db], P[mb][1], acc[db], 0, 0, 0);
  };

  int s = 0;
  // Iteration t (register set X = t % 2) consumes tile t, stores tile t+1
  // (loaded two iterations ago into set X) and loads tile t+3 into set X.
  auto iter = [&](auto xc) -> bool {
    constexpr int X = decltype(xc)::value;
    const uint16_t* ks = Ks[s];
    const int kb = C.kt * KT;
    // the next tile's cursor, and its limit entry (requested before this
    // iteration's tile loads)
    Cursor cn = C;
    advance(cn);
    limr[X ^ 1] = fetch_lim(cn.ok ? cn.R.lim_off : C.R.lim_off);

    // S^T = K Q^T for 64 keys x 32 columns, as two 32-key halves (M blocks);
    // half 1's products are issued before half 0's softmax, and half 0's PV
    // products before half 1's softmax, so the matrix core has independent
    // work while the vector units exponentiate.
    f32x16_t S[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) S[mb][i] = 0.f;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&ks[(mb * 32 + l32) * KS + kk * 16 + hf * 8]);
        S[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[kk], S[mb], 0, 0, 0);
      }
    }
    const bool partial = kb + KT > C.R.min_lim;
    // key of element i of half mb for this lane: kb + hf*4 + mb*32 + (i/4)*8 + i%4
    const int rel = (C.R.lim_off < 0 ? C.R.n_keys : (valid ? limr[X] : 0)) - kb - hf * 4;
    bf16x8_t P[2][2];
    // Online softmax of one half with a lazily raised reference maximum.
    auto softmax_half = [&](auto mbc) {
      constexpr int mb = decltype(mbc)::value;
      if (partial) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (mb * 32 + (i >> 2) * 8 + (i & 3) >= rel) S[mb][i] = -INFINITY;
      }
      float m = max3f(S[mb][0], S[mb][1], S[mb][2]);
#pragma unroll
      for (int i = 3; i < 15; i += 2) m = max3f(m, S[mb][i], S[mb][i + 1]);
      const float mx = max_lane_halves(max3f(m, S[mb][15], S[mb][15])) * sl2;
      const bool raise = mx > m_run + kRescaleSlack;
      if (__any(raise)) {
        // raising lanes: factor 2^(old - new) (0 when nothing was seen yet);
        // the others keep their reference (factor 1, also when still -inf)
        const float alpha = raise ? fast_exp2(m_run - mx) : 1.f;
        m_run = raise ? mx : m_run;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) acc[db] *= alpha;
      }
      const float m_sub = m_run == -INFINITY ? 0.f : m_run;
      // the row sum adds the bf16 probabilities the PV product uses
      float ls0 = 0.f, ls1 = 0.f;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        f32x8_t x;
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = fast_exp2(fmaf(S[mb][8 * j + e], sl2, -m_sub));
        P[mb][j] = __builtin_convertvector(x, bf16x8_t);
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
          ls0 = add_bf16x2(bf16x2_t{P[mb][j][e], P[mb][j][e + 1]}, ls0);
          ls1 = add_bf16x2(bf16x2_t{P[mb][j][e + 2], P[mb][j][e + 3]}, ls1);
        }
      }
      l_run += ls0 + ls1;
    };
    softmax_half(std::integral_constant<int, 0>{});
    pv_half(Vt[s], 0, P);
    softmax_half(std::integral_constant<int, 1>{});
    pv_half(Vt[s], 1, P);

    // Stage the next tile (its stage held tile t-1, last read before the
    // previous barrier) and start loading the one three ahead.
    const int s1 = s == kStages - 1 ? 0 : s + 1;
    if (staged[X]) {
      store_tile(xc, s1);
      staged[X] = false;
    }
    load_next(xc);
    __syncthreads();

    C = cn;
    if (!C.ok) return false;
    s = s1;
    return true;
  };
  while (iter(Set0{}) && iter(Set1{})) {
  }

  // Epilogue.  Lane (column, hf) holds d = db*32 + (i/4)*8 + hf*4 + i%4.
  const float lt = l_run + __shfl_xor(l_run, 32);
  if (!valid) return;
  if constexpr (PARTIAL) {
    const int64_t slot = (int64_t)w.out_base + col;
    float* op = p.part_o + slot * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int d0 = db * 32 + i4 * 8 + hf * 4;
        *reinterpret_cast<float4*>(op + d0) =
            make_float4(acc[db][4 * i4], acc[db][4 * i4 + 1], acc[db][4 * i4 + 2], acc[db][4 * i4 + 3]);
      }
    if (hf == 0) {
      p.part_ml[2 * slot] = m_run;
      p.part_ml[2 * slot + 1] = lt;
    }
  } else {
    const float inv = 1.f / lt;
    uint16_t* op = static_cast<uint16_t*>(p.o) + ((int64_t)qrow * p.Hq + hq) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int d0 = db * 32 + i4 * 8 + hf * 4;
        uint2 pk;
        pk.x = (uint32_t)f32_to_bf16_bits(acc[db][4 * i4] * inv) |
               ((uint32_t)f32_to_bf16_bits(acc[db][4 * i4 + 1] * inv) << 16);
        pk.y = (uint32_t)f32_to_bf16_bits(acc[db][4 * i4 + 2] * inv) |
               ((uint32_t)f32_to_bf16_bits(acc[db][4 * i4 + 3] * inv) << 16);
        *reinterpret_cast<uint2*>(op + d0) = pk;
      }
    if (hf == 0) p.lse[(int64_t)qrow * p.Hq + hq] = (m_run + __log2f(lt)) * kLn2;
  }
}

}  // namespace tile
}  // namespace padoc

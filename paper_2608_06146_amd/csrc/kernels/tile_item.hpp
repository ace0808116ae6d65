// bf16 tile computation for gfx950 (CDNA4) matrix cores: one work item --
// of the packed forward, or of the shared-key part of a decode step (paged
// K/V, split partials) -- on the 8 wavefronts of a 512-thread workgroup
// (the kernels are in tile_mfma_bf16.hip).
//
// An item is up to 256 columns (query token x head of one KV-head group: the
// G heads of a token share every K/V tile) against the item's key ranges, 64
// keys per tile.  Each wavefront owns 32 columns; per tile t it computes
//   S^T = K Q^T         v_mfma_f32_32x32x16_bf16, keys on M, columns on N
//                       (a lane owns one column and 16 of 32 key rows of a
//                       half; the other 16 rows sit in lane^32)
//   online softmax      VALU: mask, row max, exponentials, bf16 P^T
//   O^T += V^T P^T      P^T comes straight from the score registers
// (App. E Attn equation; App. C tree-varlen relation).  Only tiles of
// ancestor prefixes and the own causal range are visited: the planner lists
// no other segment.  Tiles wholly below every column's limit skip the mask.
//
// Ping-pong schedule.  Wavefronts w and w+4 share a SIMD.  Each wavefront
// alternates a matrix-core phase (PV of tile t-1, then S of tile t) and a
// vector phase (softmax of tile t, LDS staging, global loads), and the two
// halves of the workgroup run them half a step apart: while waves 0-3 issue
// MFMAs, waves 4-7 exponentiate, and the reverse, separated by two
// workgroup barriers per tile.  So each SIMD's matrix core has a wavefront
// with independent work while the other one runs its softmax.
//
// LDS holds two K stages and two V stages.  Step t reads K(t) and V(t-1)
// and stores K(t+1) and V(t) into the stages last read at step t-1; global
// loads for the stores of step t+2 (K(t+3), V(t+2)) are issued in step t, so
// every load has two steps to land.  Keys past a range's end never
// contribute: their K/V rows are copies of the range's last row (finite),
// their scores are masked to -inf, and paged V chunks past the end are zeroed
// when stored, so no stale or sentinel memory enters a product.
//
// Accumulation is fp32 and scores are in log2 units, so each probability is
// one v_exp_f32; the softmax denominator sums the bf16-rounded probabilities
// that enter the PV product, so O is their exact weighted mean.  The
// reference maximum of a column is raised only when a tile's maximum exceeds
// it by more than 2^8 (probabilities stay <= 256); the accumulator is
// rescaled only then.  Any reference gives the same O and LSE.  O is rounded
// to bf16 (RNE) at the end.
//
// Packed K/V rows land in row-major LDS tiles as they are (16-byte pieces).
// The V^T operand of the PV product is read from the row-major V tile with
// the transposing LDS read of gfx950 (ds_read_b64_tr_b16: within each group
// of 16 lanes, lane r supplies the address of 4 consecutive elements, and
// lane 4a+b receives element b of the pieces of lanes a, 4+a, 8+a and 12+a),
// two reads per fragment: lane (d, half) gets keys 4*half + 0..3 and
// 8 + 4*half + 0..3 of a 16-key group for its d, the key order of its P^T.
// Paged K/V: K blocks are chunk-major ([d/8][16 slots][8]) and land in the
// row-major LDS tile piece by piece; V blocks are d-major ([d][16 tokens]),
// so a 16-byte load holds 8 consecutive keys of one d row and lands in the
// transposed LDS tile as two 8-byte stores.  A tile's block ids come from one
// vector load issued a step ahead of its K (or V) loads.
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
constexpr float kRescaleSlack = 8.0f;  // log2 units: probabilities <= 2^8

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

// Two transposing LDS reads (4 bf16 each) joined into one 8-element MFMA
// operand: elements 0-3 from the read at lo, 4-7 from the read at hi.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8_t tr_pair(const uint16_t* lo, const uint16_t* hi) {
  typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
  const i16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(const_cast<uint16_t*>(lo)));
  const i16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(const_cast<uint16_t*>(hi)));
  const short __attribute__((ext_vector_type(8))) ab = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8_t, ab);
}

// f(integral_constant<int, i>) for i = 0 .. N-1: constant indices into the
// staging register arrays, so they stay registers (a loop index that is
// still a variable when the optimizer first looks would place them in
// scratch memory).
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// One work item (up to 256 columns) on the 8 wavefronts of a workgroup.
template <int D, bool PAGED, bool PARTIAL>
__device__ __forceinline__ void tile_item(const TileParams& p, int item) {
  constexpr int KT = kTileKeys;  // 64 keys per tile
  constexpr int KS = D + 8;      // K row stride in LDS (elements); +8 spreads banks
  constexpr int VS = KT + 8;     // paged: V^T row stride in LDS
  // packed: V row stride in LDS; +32 elements puts the 4 rows one transposing
  // read touches per pass in disjoint bank windows
  constexpr int VSR = D + 32;
  constexpr int VEL = PAGED ? D * VS : KT * VSR;  // elements of one V stage
  constexpr int NKK = D / 16;    // K-slices of the score product
  constexpr int NDB = D / 32;    // 32-row blocks of O^T
  constexpr int CPR = D / 8;     // 16-byte chunks per key row
  constexpr int KPT = KT * CPR / kThreads;           // K chunks per thread (2 or 1)
  constexpr int VPT = PAGED ? 8 * D / kThreads : KPT;  // V loads per thread (paged chunks / packed pieces)
  constexpr int NB = KT / kBlock;                    // blocks per tile (paged)

  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KT * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][VEL];

  const WorkRec w = p.work[item];
  if (w.rng_count <= 0) return;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int G = p.G;
  const int kvh = w.kvh;
  const int64_t Hkv = p.Hkv;

  // Tiles of the item (wave-uniform).
  int n_tiles = 0;
  for (int r = 0; r < w.rng_count; ++r)
    n_tiles += (p.ranges[__builtin_amdgcn_readfirstlane(w.rng_begin + r)].n_keys + KT - 1) / KT;
  n_tiles = __builtin_amdgcn_readfirstlane(n_tiles);

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

  // Per-thread load geometry (independent of the tile).  Every global load
  // is a wave-uniform (scalar) tile or block base plus a per-thread 32-bit
  // element offset, so a load costs no 64-bit vector address arithmetic.
  // K piece u (16 bytes): packed K rows are read row by row; paged K blocks
  // are chunk-major, so consecutive threads take consecutive slots of one
  // chunk (token kslot(slot)).  Either way a wave reads 1 KB contiguous, and
  // a wave's paged pieces all lie in one block (k_blk, wave-uniform).
  const uint32_t HD = (uint32_t)Hkv * D;  // elements per packed K/V row
  int k_key[KPT], k_dc[KPT], k_blk[KPT];
  uint32_t k_off[KPT];
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int u = tid + kThreads * i;
    if constexpr (PAGED) {
      const int bi = u / (kBlock * CPR), rem = u % (kBlock * CPR);
      const int slot = rem % kBlock;
      k_key[i] = bi * kBlock + kslot(slot);
      k_dc[i] = rem / kBlock;
      k_blk[i] = __builtin_amdgcn_readfirstlane(bi);
      k_off[i] = ((uint32_t)kvh * (D / 8) + k_dc[i]) * (kBlock * 8) + slot * 8;
    } else {
      k_key[i] = u / CPR;
      k_dc[i] = u % CPR;
      k_blk[i] = 0;
      k_off[i] = (uint32_t)kvh * D + k_dc[i] * 8;
    }
  }
  // paged V: chunk i of a thread is d row d, keys 8h .. 8h+7 of block bi
  // (bi wave-uniform).  packed V: the pieces of K (same rows and chunks).
  int v_blk[VPT], v_d[VPT], v_h[VPT];
  uint32_t v_off[VPT];
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int u = tid + kThreads * i;
    const int bi = u / (2 * D), rem = u % (2 * D);
    v_blk[i] = __builtin_amdgcn_readfirstlane(bi);
    v_d[i] = rem >> 1;
    v_h[i] = rem & 1;
    v_off[i] = ((uint32_t)kvh * D + v_d[i]) * kBlock + v_h[i] * 8;
  }
  // packed V^T fragments: this lane's element offset of its transposing read
  // within a 16-key group and 32-row block (lane r of a 16-lane group reads
  // key row 4*half + r/4, d columns 16*(group&1) + 4*(r%4) .. +3)
  const int v_tr = (4 * hf + ((lane & 15) >> 2)) * VSR + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // Tile cursors (wave-uniform).  No implicit padding: copies of a padded
  // struct keep the padding in memory (the compiler would place it in LDS).
  struct Cursor {
    int ri, kt;
    RangeRec R;
    int ok, tb;  // tb: the item's tiles before this range
  };
  // Past the item's last tile a cursor keeps pointing at a valid tile of the
  // last range (kt * KT < n_keys always holds), so loads stay in bounds.
  auto advance = [&](Cursor& c) {
    if (++c.kt * KT >= c.R.n_keys) {
      c.kt = 0;
      if (++c.ri < w.rng_count) {
        c.tb += (c.R.n_keys + KT - 1) / KT;
        c.R = uniform_range(p.ranges[__builtin_amdgcn_readfirstlane(w.rng_begin + c.ri)]);  // scalar loads
      } else {
        c.ok = 0;
      }
    }
  };

  // Staging registers: set b%2 holds bundle b = K(b) and V(b-1).
  uint4 kr[2][KPT], vr[2][VPT];
  int vkeep[2][PAGED ? VPT : 1];  // paged V: keys of each chunk inside the range
  bool vfull[2] = {true, true};     // paged V: the whole tile lies inside the range

  // Paged: the block ids of every tile of the item are read once, at the
  // start (thread u: tile u / NB, block u % NB; an item has at most
  // kMaxItemTiles tiles, so one id per thread), into LDS; a step's loads then
  // wait for no block-table read.  Blocks wholly past a range's end take the
  // id of the tile's first block.  Lane l (mod NB) of a wavefront reads the
  // id of block l of a tile.
  __shared__ int32_t tile_ids[PAGED ? kMaxItemTiles * NB : 1];
  static_assert(!PAGED || kMaxItemTiles * NB == kThreads, "one block id per thread");
  if constexpr (PAGED) {
    const int tile = tid / NB, bi = tid % NB;
    if (tile < n_tiles) {
      int64_t start = 0;
      int kbase = 0, nk = 0;
      for (int r = 0, tb = 0; r < w.rng_count; ++r) {
        const RangeRec R = uniform_range(p.ranges[__builtin_amdgcn_readfirstlane(w.rng_begin + r)]);
        const int nt = (R.n_keys + KT - 1) / KT;
        if (tile >= tb && tile < tb + nt) {
          start = R.kv_start;
          kbase = (tile - tb) * KT;
          nk = R.n_keys;
        }
        tb += nt;
      }
      tile_ids[tid] = p.block_table[start + (kbase >> 4) + ((kbase + bi * kBlock < nk) ? bi : 0)];
    }
    __syncthreads();
  }
  auto fetch_idv = [&](const Cursor& c) -> int { return tile_ids[(c.tb + c.kt) * NB + (lane & (NB - 1))]; };
  // Global -> registers, branch-free.  Packed rows past the range end are
  // read from the range's last row (the buffer may end there).  Paged slots
  // past the end are read as they are (their block exists: the block ids of
  // blocks wholly past the end are the tile's first block): their scores are
  // masked and their V chunks zeroed when stored.
  auto load_k = [&](auto xc, const Cursor& c, int idv) {
    constexpr int X = decltype(xc)::value;
    const int kbase = c.kt * KT;
    static_for<KPT>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr (PAGED) {
        const int64_t blk = __builtin_amdgcn_readlane(idv, k_blk[i]);
        kr[X][i] = load_stream16(Kg + blk * (int64_t)(HD * kBlock) + k_off[i]);
      } else {
        const int last = c.R.n_keys - 1 - kbase;  // >= 0
        const int kc = k_key[i] <= last ? k_key[i] : last;
        const uint16_t* tb = Kg + (c.R.kv_start + kbase) * (int64_t)HD;
        kr[X][i] = load16(tb + (__umul24((uint32_t)kc, HD) + k_off[i]));
      }
    });
  };
  auto load_v = [&](auto xc, const Cursor& c, int idv) {
    constexpr int X = decltype(xc)::value;
    const int kbase = c.kt * KT;
    if constexpr (PAGED) {
      static_for<VPT>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const int64_t blk = __builtin_amdgcn_readlane(idv, v_blk[i]);
        vr[X][i] = load_stream16(Vg + blk * (int64_t)(HD * kBlock) + v_off[i]);
        vkeep[X][i] = c.R.n_keys - (kbase + v_blk[i] * kBlock + v_h[i] * 8);
        vfull[X] = c.R.n_keys - kbase >= KT;
      });
    } else {
      const int last = c.R.n_keys - 1 - kbase;
      const uint16_t* tb = Vg + (c.R.kv_start + kbase) * (int64_t)HD;
      static_for<VPT>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const int kc = k_key[i] <= last ? k_key[i] : last;
        vr[X][i] = load16(tb + (__umul24((uint32_t)kc, HD) + k_off[i]));
      });
    }
  };
  auto store_k = [&](auto xc, uint16_t* ks) {
    constexpr int X = decltype(xc)::value;
    static_for<KPT>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      store16(&ks[k_key[i] * KS + k_dc[i] * 8], kr[X][i]);
    });
  };
  auto store_v = [&](auto xc, uint16_t* vt) {
    constexpr int X = decltype(xc)::value;
    if constexpr (PAGED) {
      static_for<VPT>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        // keys 8h..8h+3 of block bi -> positions 4h..4h+3, keys 8h+4..8h+7 -> 8+4h..
        uint16_t* row = &vt[v_d[i] * VS + v_blk[i] * 16];
        const uint4 x = vfull[X] ? vr[X][i] : keep_first(vr[X][i], vkeep[X][i]);
        *reinterpret_cast<uint2*>(row + 4 * v_h[i]) = make_uint2(x.x, x.y);
        *reinterpret_cast<uint2*>(row + 8 + 4 * v_h[i]) = make_uint2(x.z, x.w);
      });
    } else {
      static_for<VPT>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        store16(&vt[k_key[i] * VSR + k_dc[i] * 8], vr[X][i]);
      });
    }
  };

  // Bundle loader: K from cursor Lk (tile b), V from cursor Lv (tile b-1,
  // the previous Lk).  Block ids of the next K and V tiles are requested
  // first, into the other id slot, so waiting for ids never waits for the
  // newest tile data.  Past the item's end the cursors re-read a valid tile
  // (never stored), so every step issues the same loads.
  const RangeRec R0 = uniform_range(p.ranges[w.rng_begin]);
  Cursor Lk{0, 0, R0, 1, 0};
  Cursor Lv = Lk;
  int idk[2] = {0, 0}, idv[2] = {0, 0};  // [slot]: block ids of a K / V tile
  // In two parts (K, then V), so a step can spread them over its MFMAs.
  Cursor nk = Lk;
  auto load_bundle_k = [&](auto xc) {
    constexpr int X = decltype(xc)::value;
    nk = Lk;
    advance(nk);
    if constexpr (PAGED) {
      idk[X] = fetch_idv(nk);
      idv[X] = fetch_idv(Lk);
    }
    load_k(xc, Lk, idk[X ^ 1]);
  };
  auto load_bundle_v = [&](auto xc) {
    constexpr int X = decltype(xc)::value;
    load_v(xc, Lv, idv[X ^ 1]);
    Lv = Lk;
    Lk = nk;
  };
  auto load_bundle = [&](auto xc) {
    load_bundle_k(xc);
    load_bundle_v(xc);
  };

  // Compute cursor (tile of the next S product) and this column's limit
  // entry per tile: one unconditional load per tile (of a valid int when
  // the range has no limits), interpreted only in the mask.
  Cursor C{0, 0, R0, 1, 0};
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

  f32x16_t S[2];     // scores of the last S product (two 32-key halves)
  bf16x8_t P[2][2];  // probabilities of the last softmax
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) P[g >> 1][g & 1][e] = (__bf16)0.f;
  // mask data of the tile in S: whether any column is cut, and this lane's
  // limit relative to the tile (keys of the lane's rows at or past it are
  // masked)
  int s_rel = 0;
  bool s_partial = false;

  // Online softmax of the tile in S with a lazily raised reference maximum.
  auto softmax = [&]() {
    if (s_partial) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (mb * 32 + (i >> 2) * 8 + (i & 3) >= s_rel) S[mb][i] = -INFINITY;
    }
    // row maximum as a tree of v_max3 (depth 4)
    float t1[11];
#pragma unroll
    for (int j = 0; j < 10; ++j) {
      const int e = 3 * j;
      t1[j] = max3f(S[e >> 4][e & 15], S[(e + 1) >> 4][(e + 1) & 15], S[(e + 2) >> 4][(e + 2) & 15]);
    }
    t1[10] = max3f(S[1][14], S[1][15], S[1][15]);
    const float t2a = max3f(t1[0], t1[1], t1[2]), t2b = max3f(t1[3], t1[4], t1[5]);
    const float t2c = max3f(t1[6], t1[7], t1[8]), t2d = max3f(t1[9], t1[10], t1[10]);
    const float m = max3f(max3f(t2a, t2b, t2c), t2d, t2d);
    const float mx = max_lane_halves(m) * sl2;
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
    for (int mb = 0; mb < 2; ++mb)
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

  // Matrix-core phase: PV of the previous tile (V^T stage vt, P), then S of
  // the current one (K stage ks).  The A operands (16-byte LDS fragments)
  // stream through a ring of kPrefetch registers, so each MFMA's fragment
  // was requested kPrefetch MFMAs earlier.  No scalar loads are in flight
  // here (the barrier before drained them), so the LDS waits are exact.  At
  // the first step P is zero and V^T stage 1 is zeroed, so the PV adds
  // nothing; after the last tile the S product reads a stale stage and its
  // result is never used.
  constexpr int NPV = 4 * NDB, NMF = NPV + 2 * NKK, kPrefetch = PAGED ? 6 : 8;
  auto mfma_phase = [&](const uint16_t* ks, const uint16_t* vt, auto&& hook) {
    // fragment of MFMA i: PV key group g = i / NDB (keys (g/2)*32 + 16(g%2)
    // + [0,16)) and d block i % NDB; then S K-slice kk = j / 2 of half j % 2
    auto frag = [&](int i) -> bf16x8_t {
      if (i < NPV) {
        const int g = i / NDB, db = i % NDB;
        if constexpr (PAGED) {
          return *reinterpret_cast<const bf16x8_t*>(&vt[(db * 32 + l32) * VS + (g >> 1) * 32 + 16 * (g & 1) + hf * 8]);
        } else {
          // keys (g/2)*32 + 16(g%2) + 4*half + {0..3} and {8..11}
          const uint16_t* b = vt + v_tr + ((g >> 1) * 32 + 16 * (g & 1)) * VSR + db * 32;
          return tr_pair(b, b + 8 * VSR);
        }
      }
      const int j = i - NPV, kk = j >> 1, mb = j & 1;
      return *reinterpret_cast<const bf16x8_t*>(&ks[(mb * 32 + l32) * KS + kk * 16 + hf * 8]);
    };
    bf16x8_t f[kPrefetch];
#pragma unroll
    for (int i = 0; i < kPrefetch; ++i) f[i] = frag(i);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) S[mb][e] = 0.f;
    // the scheduler may not sink the reads back towards their uses
    __builtin_amdgcn_sched_barrier(0);
    static_for<NMF>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      const bf16x8_t a = f[i % kPrefetch];
      if constexpr (i < NPV) {
        constexpr int g = i / NDB, db = i % NDB;
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, P[g >> 1][g & 1], acc[db], 0, 0, 0);
      } else {
        constexpr int j = i - NPV, kk = j >> 1, mb = j & 1;
        S[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[kk], S[mb], 0, 0, 0);
      }
      if constexpr (i + kPrefetch < NMF) f[i % kPrefetch] = frag(i + kPrefetch);
      hook(ic);  // work placed between this MFMA and the next
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // Vector phase of tile c (parity Y): mask data from the compute cursor and
  // the tile's limit entry limr[Y], softmax, then the cursor moves to tile
  // c+1 and that tile's limit entry is requested into limr[Y^1].
  auto valu_phase = [&](auto yc) {
    constexpr int Y = decltype(yc)::value;
    const int kb = C.kt * KT;
    s_partial = kb + KT > C.R.min_lim;
    // key of element i of half mb for this lane: kb + hf*4 + mb*32 + (i/4)*8 + i%4
    s_rel = (C.R.lim_off < 0 ? C.R.n_keys : (valid ? limr[Y] : 0)) - kb - hf * 4;
    softmax();
    Cursor cn = C;
    advance(cn);
    limr[Y ^ 1] = fetch_lim(cn.ok ? cn.R.lim_off : C.R.lim_off);
    C = cn;
  };

  // Staging of step t: store bundle t+1 (K(t+1) into K stage (t+1)%2, V(t)
  // into V stage t%2; both stages were last read at step t-1) from register
  // set (t+1)%2, then load bundle t+3 into the same set.  Past the item's end
  // the stores write re-read tiles into stages nobody reads again.
  // It runs inside the step's matrix-core phase, a part after MFMAs 2, 5, 8
  // and 11 (the phase reads K stage t%2 and V stage (t-1)%2, the stores
  // write the other two), so its vector work fills the gaps between MFMAs
  // of this wavefront while the other half of the workgroup runs its
  // softmax on the vector ALU.
  auto staging = [&](auto xc, bool store) {
    return [&, store](auto ic) {
      constexpr int X = decltype(xc)::value;  // t % 2
      constexpr int i = decltype(ic)::value;
      using Next = std::integral_constant<int, X ^ 1>;
      if constexpr (i == 2) {
        if (store) store_k(Next{}, Ks[X ^ 1]);
      } else if constexpr (i == 5) {
        if (store) store_v(Next{}, Vt[X]);
      } else if constexpr (i == 8) {
        load_bundle_k(Next{});
      } else if constexpr (i == 11) {
        load_bundle_v(Next{});
      }
    };
  };

  // Prologue: bundle 0 (K(0)) into LDS, bundles 1 and 2 into register sets.
  // Bundle 1 is requested before K(0) is stored, so K(0), K(1) and V(0) are
  // in flight together (a short item is a chain of load latencies).
  using Set0 = std::integral_constant<int, 0>;
  using Set1 = std::integral_constant<int, 1>;
  if constexpr (PAGED) {
    idk[1] = fetch_idv(Lk);
    idv[1] = idk[1];
  }
  load_bundle(Set0{});  // bundle 0: K(0) (its V part re-reads tile 0, unused)
  load_bundle(Set1{});  // bundle 1: K(1), V(0)
  store_k(Set0{}, Ks[0]);
  for (int i = tid; i < VEL / 8; i += kThreads) reinterpret_cast<uint4*>(Vt[1])[i] = make_uint4(0, 0, 0, 0);
  load_bundle(Set0{});  // bundle 2: K(2), V(1)
  __syncthreads();

  // Step t: leading half (waves 0-3): matrix phase (with the staging),
  // barrier, vector phase, barrier.  Lagging half (waves 4-7): vector phase
  // of step t-1's scores, barrier, matrix phase (with the staging), barrier.
  // Both halves pass the same barriers.
  // The last step (t = n_tiles) stores nothing: bundle n_tiles + 1 holds no
  // tile the item uses, and waiting for its loads would only add latency.
  // Its loads are still issued (of a valid tile, never read): every step
  // issues the same loads, so the compiler's waits for a register set stay
  // exact (a load under a branch makes it wait for every load in flight).
  if (wave < 4) {
    auto step = [&](auto xc, int t) {
      constexpr int X = decltype(xc)::value;
      mfma_phase(Ks[X], Vt[X ^ 1], staging(xc, t < n_tiles));
      __syncthreads();
      if (t < n_tiles) valu_phase(xc);  // tile t
      __syncthreads();
    };
    for (int t = 0;;) {
      step(Set0{}, t);
      if (++t > n_tiles) break;
      step(Set1{}, t);
      if (++t > n_tiles) break;
    }
  } else {
    auto step = [&](auto xc, int t) {
      constexpr int X = decltype(xc)::value;
      if (t >= 1) valu_phase(std::integral_constant<int, X ^ 1>{});  // tile t-1
      __syncthreads();
      mfma_phase(Ks[X], Vt[X ^ 1], staging(xc, t < n_tiles));
      __syncthreads();
    };
    for (int t = 0;;) {
      step(Set0{}, t);
      if (++t > n_tiles) break;
      step(Set1{}, t);
      if (++t > n_tiles) break;
    }
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

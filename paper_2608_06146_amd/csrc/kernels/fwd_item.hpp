// Packed forward work item (bf16, gfx950 matrix cores): the attention of up
// to 256 columns (query token x head of one KV-head group: the G heads of a
// token share every K/V tile) against the item's key ranges, i.e. the
// ancestor prefixes and the own causal range the planner lists (App. E Attn
// equation; App. C tree-varlen relation), on the 8 wavefronts of a
// 512-thread workgroup, 32 columns per wavefront, 64 keys per tile:
//   S^T = K Q^T      v_mfma_f32_32x32x16_bf16 (keys on M, columns on N: a
//                    lane owns one column and 16 of the 32 keys of a half)
//   online softmax   log2 units, lazily raised reference maximum
//   O^T += V^T P^T   P^T straight from the score registers; V^T read with
//                    the transposing LDS read (ds_read_b64_tr_b16)
//
// Staging.  Each 1 KB piece of a K or V tile is one global_load_lds_dwordx4
// of one wavefront: lane l's 16 bytes land at byte 16*l of the piece, so no
// register holds staged data and no LDS store instruction runs (2 pieces of
// K and 2 of V per wavefront and tile at d = 128; 1 and 1 at d = 64).  Rows
// are stored without padding; the 16-byte chunks of a row are permuted (the
// lane picks which global chunk lands in its slot) so the reads are free of
// bank conflicts:
//   K stage: chunk c of row r sits at position c ^ kswz(r), so the 16 rows
//            one 16-byte fragment read touches fall in 16 distinct banks;
//   V stage: chunk c of row r sits at position c ^ vswz(r), so the 4 rows x
//            4 chunks one transposing read touches do.
// Four K and four V stages, four stages of per-column limit entries.
//
// Schedule.  Every wavefront software-pipelines its own tiles; step t (one
// workgroup barrier) issues
//   group A: S(t+1) = K(t+1) Q^T (16 MFMAs) with the exponentials, bf16
//            conversions and row sums of tile t placed between them;
//   group B: O^T += V(t)^T P(t)^T (16 MFMAs) with the scaling of S(t+1) to
//            log2 units relative to the reference maximum and the loads of
//            K(t+3), V(t+2) and the limit entries of tile t+3 between them.
// Both wavefronts of a SIMD (waves w and w+4) run this, so the matrix core
// alternates between them while each issues its vector work in the gaps (one
// wavefront issues vector instructions at about half the rate two reach).
// In group A the younger wavefront of each SIMD runs at raised priority:
// with equal priorities the older one wins every contested issue slot and
// its partner's exponentials trail into a single-wavefront tail.
//
// Reference maximum.  A column's probabilities are 2^(s*scale*log2(e) - m)
// for a reference m that is raised only when a tile's maximum exceeds it by
// more than 2^8, so every probability stays <= 2^8; the exact row maximum is
// computed only for the first tile and when a tile's probabilities sum to
// more than 2^8 (or overflow) -- then the tile's scores are recomputed from
// K, still in its stage, and the accumulator is rescaled.  That is exactly
// the set of tiles whose maximum passes the reference by more than the
// slack, so the result equals that of a per-tile maximum.  The row sum adds
// the bf16-rounded probabilities the PV product uses; O is rounded to bf16
// (RNE) at the end.
//
// Loads and waits.  Step t reads K(t+1), V(t) and the limits of tile t+1,
// loaded at step t-2, and (on the slow path) K(t) and the limits of tile t;
// its loads (K(t+3), V(t+2), limits of tile t+3) go to the stages of tiles
// t-1 and t-2, so no stage a wavefront may still read is written.  Each wavefront waits for
// its own loads of step t-2 (an immediate count: only the 2*IPW+1 loads of
// step t-1 may still be in flight) before the barrier that starts step t.
// Every step issues the same loads (past the item's end they re-read a valid
// tile into a stage nobody reads), so the counts are exact, and the item
// waits for all of them before it ends.  Keys past a range's end read the
// range's last row (the buffer may end there); their scores are masked.
#pragma once

#include "tile_common.hpp"

namespace padoc {
namespace tile {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

template <int D>
struct FwdGeom {
  static constexpr int KT = kTileKeys;         // keys per tile
  static constexpr int CPR = D / 8;            // 16-byte chunks per K/V row
  static constexpr int RPI = 1024 / (2 * D);   // rows per 1 KB load (64 lanes x 16 bytes)
  static constexpr int NI = KT / RPI;          // 1 KB loads per tile and tensor
  static constexpr int IPW = NI / kWaves;      // ... per wavefront
  static constexpr int SEL = KT * D;           // elements of one stage
  static_assert(IPW >= 1 && NI == IPW * kWaves, "whole 1 KB loads per wavefront");
  // Chunk position permutations (their own inverses).
  __device__ static int kswz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
  __device__ static int vswz(int r) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }
};

// s_waitcnt with only the vector-memory counter limited to n (< 16).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// Workgroup barrier without a memory fence (a fence would wait for every
// load in flight, including the ones two steps ahead); the asm statement
// keeps the compiler from moving memory operations across it.
__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Direct global -> LDS loads as statements the compiler does not track:
// lane l's bytes come from base + voff (voff per lane, in bytes) and land at
// LDS address lds + size*l.  The compiler's own wait insertion would treat
// them as pending LDS writes of unknown target and drain every load in
// flight before unrelated LDS reads; the kernel waits for them itself.
// M0 is named in the clobber list (the compiler keeps nothing in it in these
// kernels; clang warns that it is a reserved register).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(const lds_void_t*)p; }
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
// The same with the non-temporal hint (paged K/V, read once per call: the
// caches need not keep the lines).
__device__ __forceinline__ void dma16_nt(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt" ::"s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2" ::"s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int D, bool PAGED>
__device__ __forceinline__ void fwd_item(const TileParams& p, int item) {
  using Gm = FwdGeom<D>;
  constexpr int KT = Gm::KT, CPR = Gm::CPR, RPI = Gm::RPI, IPW = Gm::IPW, SEL = Gm::SEL;
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;

  // One buffer: K stages 0-3, then V stages 0-3 (so every fragment read is a
  // per-lane base plus an immediate offset below 64 KB); limit stages.
  __shared__ __attribute__((aligned(1024))) uint16_t smem[8 * SEL];
  __shared__ int32_t Lb[4][kThreads];
  constexpr int NBT = KT / kBlock;  // paged blocks per tile
  __shared__ int32_t tile_ids[PAGED ? kMaxItemTiles * NBT : 1];
  static_assert(!PAGED || kMaxItemTiles * NBT == kThreads, "one block id per thread");

  const WorkRec w = load_scalar(&p.work[item]);
  if (w.rng_count <= 0) return;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int G = p.G;
  const int kvh = w.kvh;

  int n_tiles = 0;
  for (int r = 0; r < w.rng_count; ++r)
    n_tiles += (load_scalar(&p.ranges[w.rng_begin + r]).n_keys + KT - 1) / KT;
  n_tiles = __builtin_amdgcn_readfirstlane(n_tiles);

  const int col = wave * 32 + l32;
  const int tok = col / G;
  const bool valid = tok < w.ntok;
  const int32_t qrow = valid ? p.toks[w.tok_begin + tok] : 0;
  const int32_t hq = kvh * G + (col - tok * G);

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
  const uint32_t HD = (uint32_t)p.Hkv * D;

  // Load geometry.  Piece i = wave*IPW + j of a K tile holds tile rows
  // RPI*i .. +RPI-1; lane l fills row RPI*i + l/CPR at chunk position l%CPR,
  // i.e. global chunk (l%CPR) ^ kswz(row).  Packed: row r is K/V row
  // kv_start + kbase + r.  Paged: row r is slot r%16 of the tile's block
  // r/16 (K blocks are chunk-major with token t in slot kslot(t), so the
  // rows are in slot order); a V tile is stored block by block as the cache
  // holds it ([block][d][16 tokens], the two 8-token halves of d row swapped
  // when bit 3 of d is set), piece i holding d rows 32*(i%(D/32)) .. +31 of
  // block i/(D/32).
  int ld_row[IPW];
  uint32_t ld_k[IPW], ld_v[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int i = wave * IPW + j;
    const int r = RPI * i + lane / CPR, pp = lane % CPR;
    ld_row[j] = r;
    if constexpr (PAGED) {
      const int c = pp ^ Gm::kswz(r);
      ld_k[j] = (((uint32_t)kvh * (D / 8) + c) * kBlock + (r % kBlock)) * 8;
      const int d = 32 * (i % (D / 32)) + (lane >> 1), h = (lane & 1) ^ ((d >> 3) & 1);
      ld_v[j] = ((uint32_t)kvh * D + d) * kBlock + 8 * h;
    } else {
      ld_k[j] = (uint32_t)kvh * D + 8 * (pp ^ Gm::kswz(r));
      ld_v[j] = (uint32_t)kvh * D + 8 * (pp ^ Gm::vswz(r));
    }
  }
  const uint16_t* rkb[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) rkb[kk] = smem + l32 * D + 8 * ((2 * kk + hf) ^ Gm::kswz(l32));
  // V^T fragment bases.  Packed (transposing reads): lane r of a 16-lane
  // group reads key row 4*hf + (r%16)/4 (+ the key group's offset, a
  // multiple of 4) and the 4 d values 32*db + 16*((l/16)%2) + 4*(r%4) .. +3.
  // Paged (16-byte reads): lane (l32, hf) reads tokens 8*hf .. +7 of d row
  // 32*db + l32 of the key group's block.
  const uint16_t* rvb[NDB];
  if constexpr (PAGED) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      rvb[db] = smem + 4 * SEL + (32 * db + l32) * kBlock + 8 * (hf ^ ((l32 >> 3) & 1));
  } else {
    const int vr = 4 * hf + ((lane & 15) >> 2);
    const int sw = Gm::vswz(vr);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d = 32 * db + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      rvb[db] = smem + 4 * SEL + vr * D + 8 * ((d >> 3) ^ sw) + (d & 7);
    }
  }

  struct Cursor {
    int ri, kt;
    RangeRec R;
    int ok, tb;
  };
  auto advance = [&](Cursor& c) {
    if (++c.kt * KT >= c.R.n_keys) {
      c.kt = 0;
      if (++c.ri < w.rng_count) {
        c.tb += (c.R.n_keys + KT - 1) / KT;
        c.R = load_scalar(&p.ranges[w.rng_begin + c.ri]);
      } else {
        c.ok = 0;
      }
    }
  };
  // Stage of tile t: t % 4 (compile-time: the loop is unrolled by 4).
  auto kst = [&](auto sc) -> uint16_t* { return smem + (decltype(sc)::value % 4) * SEL; };
  auto vst = [&](auto sc) -> uint16_t* { return smem + (4 + decltype(sc)::value % 4) * SEL; };
  auto lst = [&](auto sc) -> int32_t* { return Lb[decltype(sc)::value % 4]; };
  // Block ids (paged): lane l (mod NBT) of a wavefront holds the id of block
  // l of the tile at cursor c (read from the item's staged ids).
  auto tile_blocks = [&](const Cursor& c) -> int {
    if constexpr (PAGED) return tile_ids[(c.tb + c.kt) * NBT + (lane & (NBT - 1))];
    else return 0;
  };
  // This wavefront's pieces of the K (or V: is_v) tile at cursor c into stage
  // st; ids: the tile's block ids (paged).
  auto load_tile = [&](const uint16_t* g, const Cursor& c, uint16_t* st, const uint32_t* ldc, bool is_v, int ids) {
    const uint32_t sb = lds_addr(st) + wave * IPW * 1024;
    if constexpr (PAGED) {
      // slots past a range's end are read as they are (their blocks exist:
      // ids of blocks wholly past the end are the tile's first block)
#pragma unroll
      for (int j = 0; j < IPW; ++j) {
        const int i = wave * IPW + j;
        const int b = is_v ? i / (D / 32) : (RPI * i) / kBlock;
        const int64_t blk = __builtin_amdgcn_readlane(ids, b);
        dma16_nt(g + blk * (int64_t)(HD * kBlock), 2 * ldc[j], sb + j * 1024);
      }
    } else {
      const int kbase = c.kt * KT;
      const int last = c.R.n_keys - 1 - kbase;
      const uint16_t* tb = g + uniform64(c.R.kv_start + kbase) * (int64_t)HD;
#pragma unroll
      for (int j = 0; j < IPW; ++j) {
        const int r = ld_row[j] <= last ? ld_row[j] : last;
        dma16(tb, 2 * (__umul24((uint32_t)r, HD) + ldc[j]), sb + j * 1024);
      }
    }
  };
  auto load_lim = [&](const Cursor& c, int32_t* dst) {
    const int32_t lim_off = c.R.lim_off;
    const int32_t* lb = lim_off < 0 ? &p.work[item].ntok : p.lims + lim_off;
    dma4(lb, lim_off < 0 || !valid ? 0u : 4u * tok, lds_addr(dst + wave * 64));
  };

  const RangeRec R0 = load_scalar(&p.ranges[w.rng_begin]);
  Cursor Lk{0, 0, R0, 1, 0};  // next tile to load (K, V, limits)
  Cursor C = Lk;              // tile whose scores were computed last

  float m_run = -INFINITY, l_run = 0.f, m_sub = 0.f, alpha = 1.f;
  bool any_raise = false;
  // Some valid column has seen no key yet (its reference is still -inf and
  // its probabilities are taken relative to 0): the exact path runs.
  bool any_fresh = true;
  f32x16_t acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = 0.f;
  const float sl2 = p.scale_log2;
  f32x16_t Sb[2][2];  // [tile parity][32-key half]
  bf16x8_t P[2][2];

  // Mask of the tile at cursor C in score buffer Y, limit entries in lim.
  auto mask_tile = [&](auto yc, const int32_t* lim) {
    constexpr int Y = decltype(yc)::value;
    const int kb = C.kt * KT;
    if (kb + KT > C.R.min_lim) {
      // element i of half mb of lane (col, hf) is tile row mb*32 + 8*(i/4) +
      // 4*hf + i%4; paged rows are in slot order (bits 2 and 3 of the key
      // swapped within each block)
      const int rel = (C.R.lim_off < 0 ? C.R.n_keys : (valid ? lim[tid] : 0)) - kb - hf * (PAGED ? 8 : 4);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = PAGED ? mb * 32 + 16 * ((i >> 3) & 1) + 4 * ((i >> 2) & 1) + (i & 3)
                                : mb * 32 + (i >> 2) * 8 + (i & 3);
          if (key >= rel) Sb[Y][mb][i] = -INFINITY;
        }
    }
  };
  // Row maximum of score buffer Y as a v_max3 tree, in pieces 0..6; piece 6
  // raises the reference maximum where the tile's maximum exceeds it by
  // more than 2^8 and sets the rescale factor alpha of those columns.
  float t1[11], t2[4];
  auto stats_piece = [&](auto yc, auto kc) {
    constexpr int Y = decltype(yc)::value, k = decltype(kc)::value;
    auto e3 = [&](int j) {
      const int e = 3 * j;
      return max3f(Sb[Y][e >> 4][e & 15], Sb[Y][(e + 1) >> 4][(e + 1) & 15], Sb[Y][(e + 2) >> 4][(e + 2) & 15]);
    };
    if constexpr (k == 0) { t1[0] = e3(0); t1[1] = e3(1); t1[2] = e3(2); }
    if constexpr (k == 1) { t1[3] = e3(3); t1[4] = e3(4); }
    if constexpr (k == 2) { t1[5] = e3(5); t1[6] = e3(6); t1[7] = e3(7); }
    if constexpr (k == 3) { t1[8] = e3(8); t1[9] = e3(9); t1[10] = max3f(Sb[Y][1][14], Sb[Y][1][15], Sb[Y][1][15]); }
    if constexpr (k == 4) {
      t2[0] = max3f(t1[0], t1[1], t1[2]);
      t2[1] = max3f(t1[3], t1[4], t1[5]);
      t2[2] = max3f(t1[6], t1[7], t1[8]);
      t2[3] = max3f(t1[9], t1[10], t1[10]);
    }
    if constexpr (k == 5) t2[0] = max3f(max3f(t2[0], t2[1], t2[2]), t2[3], t2[3]);
    if constexpr (k == 6) {
      const float mx = max_lane_halves(t2[0]) * sl2;
      const bool raise = mx > m_run + kRescaleSlack;
      alpha = raise ? fast_exp2(m_run - mx) : 1.f;
      m_run = raise ? mx : m_run;
      m_sub = m_run == -INFINITY ? 0.f : m_run;
      any_raise = __any(raise);
      any_fresh = __any(valid && m_run == -INFINITY);
    }
  };
  // Exponentials of score buffer Y, in pieces 0..15 (two scores each; every
  // fourth piece converts 8 of them to bf16 and adds them to the row sum).
  // SCALED: the buffer already holds log2-unit scores relative to the
  // reference; else they are scaled here.
  float xs[32];
  float ls0 = 0.f, ls1 = 0.f;
  auto exp_piece = [&](auto yc, auto kc, auto scc) {
    constexpr int Y = decltype(yc)::value, k = decltype(kc)::value;
    constexpr bool SCALED = decltype(scc)::value;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      constexpr int e0 = 2 * k;
      const int e = e0 + u;
      if constexpr (SCALED)
        xs[e] = fast_exp2(Sb[Y][e >> 4][e & 15]);
      else
        xs[e] = fast_exp2(fmaf(Sb[Y][e >> 4][e & 15], sl2, -m_sub));
    }
    if constexpr (k % 4 == 3) {
      constexpr int g = k / 4;  // P[g/2][g%2] = scores 8g .. 8g+7
      f32x8_t x;
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = xs[8 * g + e];
      P[g >> 1][g & 1] = __builtin_convertvector(x, bf16x8_t);
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        ls0 = add_bf16x2(bf16x2_t{P[g >> 1][g & 1][e], P[g >> 1][g & 1][e + 1]}, ls0);
        ls1 = add_bf16x2(bf16x2_t{P[g >> 1][g & 1][e + 2], P[g >> 1][g & 1][e + 3]}, ls1);
      }
    }
  };

  // Scores of buffer Y to log2 units relative to the reference maximum, in
  // pieces 0..15 (two scores each).
  auto fma_piece = [&](auto yc, auto kc) {
    constexpr int Y = decltype(yc)::value, k = decltype(kc)::value;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = 2 * k + u;
      Sb[Y][e >> 4][e & 15] = fmaf(Sb[Y][e >> 4][e & 15], sl2, -m_sub);
    }
  };

  constexpr int kPre = 6;  // fragment reads in flight
  // MFMAs of the score product (NA) and of the PV product (NB); the 16
  // pieces of the exponentials and of the scaling are spread evenly over them.
  constexpr int NA = 2 * NKK, NB = 4 * NDB, kPieces = 16;
  static_assert(kPieces % NA == 0 && kPieces % NB == 0 && NB >= 4, "pieces per MFMA");
  // Score product S(t') = K(t') Q^T into buffer Y from stage ks, with
  // hook(i) after MFMA i.
  auto s_product = [&](auto yc, auto ksc, auto&& hook) {
    constexpr int Y = decltype(yc)::value, KS = decltype(ksc)::value % 4;
    auto frag = [&](int i) -> bf16x8_t {
      const int kk = i >> 1, mb = i & 1;
      return *reinterpret_cast<const bf16x8_t*>(rkb[kk] + KS * SEL + mb * 32 * D);
    };
    bf16x8_t f[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) f[i] = frag(i);
    __builtin_amdgcn_sched_barrier(0);
    static_for<NA>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      constexpr int kk = i >> 1, mb = i & 1;
      const bf16x8_t a = f[i % kPre];
      if constexpr (kk == 0)
        Sb[Y][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[kk], f32x16_t{}, 0, 0, 0);
      else
        Sb[Y][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[kk], Sb[Y][mb], 0, 0, 0);
      if constexpr (i + kPre < NA) f[i % kPre] = frag(i + kPre);
      hook(ic);
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  // O^T += V^T P^T from stage vt, with hook(i) after MFMA i.
  // O^T += V^T P^T from V stage vsc%4 (rvb: per-lane bases), with hook(i)
  // after MFMA i.
  auto pv_product = [&](auto vsc, auto&& hook) {
    constexpr int VS = decltype(vsc)::value % 4;
    auto frag = [&](int i) -> bf16x8_t {
      const int g = i / NDB, db = i % NDB;
      if constexpr (PAGED) {
        return *reinterpret_cast<const bf16x8_t*>(rvb[db] + VS * SEL + g * kBlock * D);
      } else {
        const uint16_t* b = rvb[db] + VS * SEL + ((g >> 1) * 32 + 16 * (g & 1)) * D;
        return tr_pair(b, b + 8 * D);
      }
    };
    bf16x8_t f[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) f[i] = frag(i);
    __builtin_amdgcn_sched_barrier(0);
    static_for<NB>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      constexpr int g = i / NDB, db = i % NDB;
      acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[i % kPre], P[g >> 1][g & 1], acc[db], 0, 0, 0);
      if constexpr (i + kPre < NB) f[i % kPre] = frag(i + kPre);
      hook(ic);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // Paged V slots of the tile at cursor C at or past its range's end are
  // zeroed in V stage vst (its scores are masked, so P is 0 there, but the
  // cache slots may hold anything, and 0 * NaN is NaN).  Thread u takes d row
  // u % D of block u / D; the caller has waited for the stage's loads and a
  // barrier separates this from the stage's reads.
  auto zero_v_tail = [&](uint16_t* vs) {
    if constexpr (PAGED) {
      const int keep = C.R.n_keys - C.kt * KT;  // valid keys of the tile
      if (keep < KT && tid < NBT * D) {
        const int b = tid / D, d = tid % D;
#pragma unroll
        for (int hp = 0; hp < 2; ++hp) {
          const int kh = keep - (16 * b + 8 * (hp ^ ((d >> 3) & 1)));  // valid keys of this 8-key half
          if (kh < 8) {
            uint4* q = reinterpret_cast<uint4*>(vs + b * D * kBlock + d * kBlock + 8 * hp);
            *q = kh <= 0 ? make_uint4(0, 0, 0, 0) : keep_first(*q, kh);
          }
        }
      }
      if (keep < KT) __builtin_amdgcn_s_waitcnt(0xC07F);  // LDS stores done before the next barrier
    }
  };

  // Prologue: K, V and the limit entries of tiles 0..2; then S(0), its
  // mask, its exact row maximum and its scaling, and the zeroed tail of V(0).
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  if constexpr (PAGED) {
    // The block ids of every tile of the item (thread u: tile u / NBT, block
    // u % NBT; an item has at most kMaxItemTiles tiles), read once into LDS
    // so no step waits for a block-table read.  Blocks wholly past a range's
    // end take the id of the tile's first block.
    const int tile = tid / NBT, bi = tid % NBT;
    if (tile < n_tiles) {
      int64_t start = 0;
      int kbase = 0, nk = 0;
      for (int r = 0, tb = 0; r < w.rng_count; ++r) {
        const RangeRec R = load_scalar(&p.ranges[w.rng_begin + r]);
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
    __builtin_amdgcn_s_waitcnt(0);
    bar();
  }
  static_for<3>([&](auto sc) {
    const int ids = tile_blocks(Lk);
    load_tile(Kg, Lk, kst(sc), ld_k, false, ids);
    load_tile(Vg, Lk, vst(sc), ld_v, true, ids);
    load_lim(Lk, lst(sc));
    advance(Lk);
  });
  __builtin_amdgcn_s_waitcnt(0);
  bar();
  if constexpr (PAGED) {
    zero_v_tail(vst(I0{}));
    __builtin_amdgcn_s_waitcnt(0);
    bar();
  }
  s_product(I0{}, I0{}, [&](auto) {});
  mask_tile(I0{}, Lb[0]);
  static_for<7>([&](auto kc) { stats_piece(I0{}, kc); });
  static_for<kPieces>([&](auto kc) { fma_piece(I0{}, kc); });

  // Step t (SC = t mod 4): tile t's scaled scores are in buffer SC%2; K, V
  // and the limits of tiles t+1 and t+2 are in their stages (loaded at steps
  // t-2 and t-1; this step's barrier is preceded by the wait for those of
  // step t-2), and K(t), V(t) and the limits of tile t still are (the slow
  // path reads K(t)).  The step's loads (tile t+3) go to the stages of tile
  // t-1, which every wavefront finished reading before this barrier.  The
  // paged V slots of tile t+1 past its range's end are zeroed here, read
  // after the next barrier.
  using Scaled = std::integral_constant<bool, true>;
  using Raw = std::integral_constant<bool, false>;
  auto step = [&](auto sc, int t) {
    constexpr int SC = decltype(sc)::value;
    using Y = std::integral_constant<int, SC % 2>;
    using YN = std::integral_constant<int, (SC + 1) % 2>;
    wait_vm<2 * IPW + 1>();  // this wavefront's loads of step t-2 have landed
    bar();
    ls0 = 0.f;
    ls1 = 0.f;
    if (wave >= 4) __builtin_amdgcn_s_setprio(1);
    s_product(YN{}, std::integral_constant<int, SC + 1>{}, [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      static_for<kPieces / NA>([&](auto uc) {
        exp_piece(Y{}, std::integral_constant<int, i * (kPieces / NA) + decltype(uc)::value>{}, Scaled{});
      });
    });
    __builtin_amdgcn_s_setprio(0);
    // Tile t's probabilities and sums are complete here (else the compiler
    // sinks their computation past the branches below, next to their use).
    asm volatile("" ::"v"(P[0][0]), "v"(P[0][1]), "v"(P[1][0]), "v"(P[1][1]), "v"(ls0), "v"(ls1));
    if (any_fresh || __any(!(ls0 + ls1 <= 256.f))) {
      // some probability exceeds 2^8 (or overflowed): the tile's maximum
      // passed the reference by more than the slack (or a column has no
      // reference yet)
      s_product(Y{}, std::integral_constant<int, SC>{}, [&](auto) {});
      mask_tile(Y{}, lst(std::integral_constant<int, SC>{}));
      static_for<7>([&](auto kc) { stats_piece(Y{}, kc); });
      if (any_raise) {
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) acc[db] *= alpha;
      }
      ls0 = 0.f;
      ls1 = 0.f;
      static_for<kPieces>([&](auto kc) { exp_piece(Y{}, kc, Raw{}); });
    }
    l_run += ls0 + ls1;
    advance(C);
    if (t + 1 < n_tiles) {
      mask_tile(YN{}, lst(std::integral_constant<int, SC + 1>{}));
      zero_v_tail(vst(std::integral_constant<int, SC + 1>{}));
    }
    const int ids = tile_blocks(Lk);
    pv_product(std::integral_constant<int, SC>{}, [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      static_for<kPieces / NB>([&](auto uc) {
        fma_piece(YN{}, std::integral_constant<int, i * (kPieces / NB) + decltype(uc)::value>{});
      });
      if constexpr (i == NB / 2) load_tile(Kg, Lk, kst(std::integral_constant<int, SC + 3>{}), ld_k, false, ids);
      if constexpr (i == NB / 2 + 1) load_tile(Vg, Lk, vst(std::integral_constant<int, SC + 3>{}), ld_v, true, ids);
      if constexpr (i == NB / 2 + 2) {
        load_lim(Lk, lst(std::integral_constant<int, SC + 3>{}));
        advance(Lk);
      }
    });
  };
  for (int t = 0;;) {
    step(std::integral_constant<int, 0>{}, t);
    if (++t >= n_tiles) break;
    step(std::integral_constant<int, 1>{}, t);
    if (++t >= n_tiles) break;
    step(std::integral_constant<int, 2>{}, t);
    if (++t >= n_tiles) break;
    step(std::integral_constant<int, 3>{}, t);
    if (++t >= n_tiles) break;
  }
  __builtin_amdgcn_s_waitcnt(0);

  const float lt = l_run + __shfl_xor(l_run, 32);
  if (!valid) return;
  if constexpr (PAGED) {
    // split partial of column col: unnormalised O, reference maximum (log2
    // units), sum
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
    return;
  }
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

}  // namespace tile
}  // namespace padoc

// Q-block attention for bf16 KV caches on gfx950 (arxiv 2511.11581, Sec. 4.4
// Q-Blocks; Sec. 4.1 tiled softmax with online normalisation; Eq. 1-2).
//
// One workgroup = (Q-block, kv head g): 8 waves x 32 rows, BLOCK_M = 256
// rows = BLOCK_Q tokens x G query heads (row r is token r / G, head r % G).
// Only sequences with at least 2 query tokens come here.  Per wave and
// 64-key tile:
//   S^T[64 keys x 32 rows] = K Q^T          (v_mfma_f32_32x32x16_bf16)
//   online softmax, one lane per row (max / sum finish with permlane32)
//   O^T[d x 32 rows]      += V^T P^T         (P^T from S^T's registers)
//
// Per period t every wave runs one fixed sequence of matrix-core products:
// the scores of tile t + 1, then O += V^T P^T of tile t with the softmax of
// tile t + 1 (one exp, one pack and one dot2 per weight) placed between its
// products, so that the VALU work runs under the wave's own products; the
// second wave on the SIMD does the same.  Each weight takes one fma (c S -
// m, c = scale * log2(e)) before its exp; Q enters the products unchanged
// (rounding Q * c to bf16 would add a relative error of 2^-9 to every
// score, which grows with the logit).
//
// K/V tiles of 64 keys move from HBM into a ring of 4 LDS stages with
// global_load_lds_dwordx4 (no staging registers, no VALU), three tiles
// ahead of their use; each wave issues its share of a tile (whole 16-byte
// row chunks, 4 or 8 rows of one cache block per instruction, scalar page
// base) between its score products.  The waits are explicit vmcnt counts,
// so the tiles still in flight are never waited for.
//
// LDS layouts (rows of 2d bytes, 16-byte chunks XOR-swizzled by row; the
// swizzles were chosen with SQ_LDS_BANK_CONFLICT on the device, which reads
// 0 for every operand-read pattern below):
//   K: natural rows, chunk c of row r at slot c ^ fK(r), fK spreading the
//      16 rows that one 16-lane pass of ds_read_b128 reads over a 256-byte
//      bank window; read as MFMA A operands (32 keys x 8 d per lane group).
//   V: natural rows, chunk c at slot c ^ fV(r), fV a function of r mod 8
//      (the 8 rows one transposing read touches); read as V^T operands with
//      ds_read_b64_tr_b16, which hands each lane 4 consecutive keys of one d
//      column from the 16-lane group's 4 row pointers.
// The 32x32 score tile's lane l holds keys 8(i/4) + 4(l/32) + i%4 of its
// row, so the PV product takes its 16 keys in that order: V^T operand slots
// 0-3 come from keys 16u + 4(l/32) + 0..3 and slots 4-7 from 16u + 8 +
// 4(l/32) + 0..3.
//
// The reference m of a row is the first tile's row max and is only raised
// when a weight of the row exceeds 2^12 (the lane's 32-key weight sum tells):
// the final division uses the same reference, so the result is unchanged.
//
// The output goes through the K ring (free once the last scores are done)
// so that every store writes whole rows.
#include <type_traits>

#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kTile = kPrefillTileKeys;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16v2 __attribute__((ext_vector_type(2)));
#define LDS_AS __attribute__((address_space(3)))

constexpr uint32_t kOnesBf16x2 = 0x3f803f80u;   // bf16 pair (1, 1)

__device__ __forceinline__ uint32_t lds_addr(const uint8_t* p) {
  return (uint32_t)(uintptr_t)(const LDS_AS uint8_t*)p;
}

// Global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4): lane
// i's 16 bytes at g land at LDS byte lds + 16 i (lds wave-uniform).  Issued
// as inline asm, outside the compiler's view of LDS: otherwise every LDS
// read after it would first wait for all such copies in flight.  The
// kernel orders copies and reads itself, with explicit vmcnt waits before
// its barriers.
__device__ __forceinline__ void dma16(const uint8_t* g, uint32_t lds) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"   // (one wait state after the M0 write)
               :
               : "v"(g), "{m0}"(lds)
               : "memory");
}

// c + lo(a) lo(b) + hi(a) hi(b) for bf16 pairs, accumulated in fp32.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16v2, a), __builtin_bit_cast(bf16v2, b), c, false);
}

// Scalar-cache loads (wave-uniform address): a table entry, a Q-block record.
__device__ __forceinline__ int load_s32(const int* p) {
  return *(const __attribute__((address_space(4))) int*)p;
}
__device__ __forceinline__ int4 load_rec(const int4* p) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  const i32x4 v = *(const __attribute__((address_space(4))) i32x4*)p;
  return make_int4(v[0], v[1], v[2], v[3]);
}

// s_waitcnt with the vector-memory count bounded by N and every LDS
// operation drained (gfx9 encoding: vmcnt[3:0] and [15:14], expcnt[6:4],
// lgkmcnt[11:8]).
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0070);
}
// Vector-memory count bounded by N, LDS operations left in flight; a
// compiler memory barrier too, so that no LDS access moves across it.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
// Every LDS operation drained, vector-memory operations left in flight.
__device__ __forceinline__ void wait_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory");
}

// The Q-block record of rank wi in the plan kernel's order (decreasing
// key-tile count; ties in sequence, then block order), derived by the wave
// itself from the batch metadata, for launches without a plan kernel (at
// most kFusedPlanSeqs sequences; block_q a power of two).  Lane j holds
// sequence j.  Q-block b of a sequence with q query rows and ctx earlier
// keys needs ctx + min((b + 1) bq, q) keys, so the count C(K) of Q-blocks
// with at least K key tiles is a sum of closed forms; the rank's tile
// count K* is the largest K with C(K) > wi (C falls as K rises), found by
// a 64-way search with one candidate per lane, and the record is then the
// (wi - C(K* + 1))-th Q-block with K* tiles.  False if wi >= the count.
__device__ bool fused_record(const BatchArgs& a, const PrefillPlan& pp, int wi, int4& rec) {
  const int lane = __builtin_amdgcn_workitem_id_x() & 63, S = a.num_seqs;
  const int bq = pp.block_q, bsh = __builtin_ctz((unsigned)bq);
  const int cap = a.mb * a.block_size;
  int t0 = 0, ql = 0, ctx = 0, nqb = 0, kt = 0;
  if (lane < S) {
    t0 = a.qsl[lane];
    const int q = a.qsl[lane + 1] - t0, L = min(a.seq_lens[lane], cap);
    if (q >= pp.qmin && t0 >= 0 && t0 + q <= a.num_tokens && L >= q) {
      ql = q;
      ctx = L - q;
      nqb = (q + bq - 1) >> bsh;
      kt = (L + kTile - 1) / kTile;   // tiles of its last Q-block, the most
    }
  }
  // Q-blocks of sequence j (readlane'd) with at least K key tiles
  auto cnt = [&](int j, int K) {
    const int n = __builtin_amdgcn_readlane(nqb, j), q = __builtin_amdgcn_readlane(ql, j);
    const int x = kTile * (K - 1) - __builtin_amdgcn_readlane(ctx, j);   // need min((b+1) bq, q) > x
    return (n == 0 || q <= x) ? 0 : n - (x < 0 ? 0 : (x >> bsh));
  };
  int count = 0, kmax = 0;
  for (int j = 0; j < S; ++j) {
    count += __builtin_amdgcn_readlane(nqb, j);
    kmax = max(kmax, __builtin_amdgcn_readlane(kt, j));
  }
  count = min(count, pp.work_items);
  if (wi >= count) return false;
  // largest K in [1, kmax] with C(K) > wi: C(lo) > wi, C(hi) <= wi
  int lo = 1, hi = kmax + 1;
  while (hi - lo > 1) {
    const int step = (hi - lo + 63) / 64;
    const int K = lo + lane * step;
    int c = 0;
    for (int j = 0; j < S; ++j) c += cnt(j, K);
    const bool ok = K < hi && c > wi;
    lo += (63 - __builtin_clzll(__ballot(ok))) * step;
    hi = min(hi, lo + step);
  }
  int r = wi;
  for (int j = 0; j < S; ++j) r -= cnt(j, lo + 1);   // rank among the Q-blocks with lo tiles
  for (int j = 0; j < S; ++j) {
    const int hi_j = cnt(j, lo), e = hi_j - cnt(j, lo + 1);
    if (r < e) {
      const int b = __builtin_amdgcn_readlane(nqb, j) - hi_j + r;
      const int q = __builtin_amdgcn_readlane(ql, j);
      rec = make_int4(j, __builtin_amdgcn_readlane(t0, j) + b * bq, min(bq, q - b * bq),
                      __builtin_amdgcn_readlane(ctx, j) + b * bq);
      return true;
    }
    r -= e;
  }
  return false;   // (not reached: C(lo) > wi)
}

// GATHER: only the last Q-block of each sequence runs; it walks the block
// table and copies every tile into the ring with the same loads, then
// stores the bytes of every valid key into the dense outputs a.kd / a.vd:
// K read back at the matrix-core operand addresses, V through the loader's
// swizzle (pa_debug_gather).
//
// W waves of 32 rows: BLOCK_M = 32 W.  W = 8: one workgroup per CU (128 KB
// of LDS: K and V rings of 4 stages, tiles t + 1 .. t + 3 in flight).  W =
// 4: two workgroups per CU (80 KB each: a K ring of 3 stages and a V ring of
// 2; period t loads V of tile t + 1 and K of tile t + 3), so that one
// workgroup's barrier waits and start-up run under the other's products.
//
// FP8 (e4m3 caches; W = 8, d = 128 or 64): the copies land in a staging
// area private to each wave (3 stages of its 8 K rows and 8 V rows, 2 KB a
// stage; with d = 64 1 KB, K and V rows in one copy instruction, lanes
// 0..31 K and 32..63 V, and one read and widening), and the wave itself
// widens its rows to bf16 into the K and V rings (3 stages each), exactly: every e4m3 value is a bf16 value, and the
// per-tensor scales act on the scores (k_scale, folded into c) and on the
// output (v_scale).  Period t widens tile t + 2, which landed during
// periods t - 2 and t - 1, and copies tile t + 4 into the staging stage
// that tile t + 1 left; V rows at or past the end are widened to zeros.
// Since a wave widens only what it copied, its own vmcnt wait orders the
// two; the barrier of the next period publishes the bf16 rows.  The
// products are those of the bf16 kernel.
template <int D, int W, bool FP8, bool GATHER>
__global__ __launch_bounds__(64 * W, 8 / W) void qblock_kernel(BatchArgs a, PrefillPlan pp) {
  constexpr int RB = 2 * D;                        // bytes per row in the rings (bf16)
  constexpr int CPR = D / 8;                       // 16-byte chunks per row
  constexpr int TB = kTile * RB;                   // bytes per K (or V) tile
  constexpr int RPI = 1024 / RB;                   // rows per load instruction
  constexpr int NLD = kTile / (RPI * W);           // load instructions per wave, tile and tensor
  constexpr int KRW = 256 / RB;                    // K rows per 256-byte bank window
  constexpr int NT = D / 16;                       // k-steps of K Q^T
  constexpr int NDB = D / 32;                      // 32-row d blocks of O^T
  constexpr int KSTG = FP8 ? 3 : W == 8 ? 4 : 3;   // K ring stages
  constexpr int VSTG = FP8 ? 3 : W == 8 ? 4 : 2;   // V ring stages
  constexpr bool kSplit = W != 8;                  // K and V of one period from different tiles
  // fp8 staging: per wave and stage, its K rows then its V rows (kTile / W
  // rows of D bytes each, one 16-byte copy per lane and tensor)
  constexpr int SROW = kTile / W;                  // rows per wave and tile
  constexpr int SCH = D / 16;                      // 16-byte chunks per fp8 row
  constexpr int SSTG = 3;                          // staging stages
  // d = 64: a wave's K and V rows of a tile are one 16-byte copy per lane
  // (lanes 0..31 K, 32..63 V); d = 128: one copy per tensor
  constexpr bool KV1 = FP8 && SROW * SCH == 32;
  constexpr int SWB = KV1 ? 1024 : 2 * 1024;       // staging bytes per wave and stage
  constexpr int NCP = KV1 ? 1 : 2;                 // copy instructions per wave and tile
  constexpr int SBYTES = FP8 ? SSTG * W * SWB : 0;
  constexpr int SBASE = KSTG * TB;                 // staging after the K ring
  constexpr int VBASE = KSTG * TB + SBYTES;        // V ring after the K ring (and the staging)
  static_assert(kQblockWaveRows == 32 && (W == 8 || W == 4), "8 or 4 waves x 32 rows");
  static_assert(NLD >= 1 && NLD * RPI * W == kTile, "tile loads");
  static_assert(RPI <= 16, "one instruction stays inside one 16-key block");
  static_assert(!FP8 || (W == 8 && (SROW * SCH == 64 || SROW * SCH == 32)), "fp8: 8 waves, d = 64 or 128");
  static_assert(((KSTG + VSTG) * TB + SBYTES) * (8 / W) <= 160 * 1024, "workgroups per CU fit the LDS");
  static_assert(kQblockWaveRows * W * RB <= KSTG * TB + SBYTES, "output staging below the V ring");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[(KSTG + VSTG) * TB + SBYTES];
  auto kst = [](int t) { return t % KSTG; };   // ring stage of tile t's K
  auto vst = [](int t) { return t % VSTG; };   // ring stage of tile t's V

  const int tid = __builtin_amdgcn_workitem_id_x(), lane = tid & 63, wave = uniform(tid >> 6);
  const int n = lane & 31, hf = lane >> 5;
  const int Hkv = a.num_kv_heads;
  const int G = a.group;
  const BlockDiv bd = a.bdiv;   // block size: a multiple of 16
  const float c = a.sl2;   // scale * log2(e) (* k_scale)
  // One workgroup per (Q-block, kv head) unit, kv head fastest: with
  // round-robin dispatch over the 8 XCDs, the units of one kv head (Hkv =
  // 8) share an XCD and its L2, which serves the K/V re-reads of a
  // sequence's Q-blocks.
  const int wg = __builtin_amdgcn_workgroup_id_x();
  const int g = wg % Hkv;
  const int wi = wg / Hkv;
  // The Q-block's record (its sequence, first token, tokens, and the keys
  // before its first token): from the plan kernel, in one scalar load, or
  // derived here.
  int4 rec;
  if (!GATHER && pp.fused) {
    if (!fused_record(a, pp, wi, rec)) return;
  } else {
    if (wi >= load_s32(pp.count)) return;
    rec = load_rec(pp.rec + wi);
  }
  const int seq = rec.x;
  const int t0 = rec.y;        // token of the block's row 0 (rows are relative to it)
  const int tok_lo = 0;
  const int tok_hi = rec.z;    // the block's tokens (1 .. BLOCK_Q)
  const int ctx = rec.w;       // keys before the block's first token
  if (tok_hi <= 0) return;
  const int kv_len = ctx + tok_hi;                 // keys the block needs
  const int ntiles = (kv_len + kTile - 1) / kTile;
  const int last_blk = bd.block(kv_len - 1);
  const int32_t* bt_row = a.bt + (int64_t)seq * a.bt_row;

  // This lane's row and the wave's range of causal bounds.
  const int row = wave * 32 + n;
  const int tl = tok_lo + row / G;
  const bool rvalid = tl < tok_hi;
  const int pos = ctx + (rvalid ? tl : tok_hi - 1);
  const int pos_lo = ctx + min(tok_lo + (wave * 32) / G, tok_hi - 1);
  const int pos_hi = ctx + min(tok_lo + (wave * 32 + 31) / G, tok_hi - 1);
  const int nact = min(ntiles, pos_hi / kTile + 1);     // tiles this wave attends to
  const int nfull = min(ntiles, (pos_lo + 1) / kTile);  // tiles needing no causal mask

  // Q^T operands: d = 16t + 8hf + 0..7 of this row.
  bf16x8 qt[NT];
  if constexpr (!GATHER) {
    const uint8_t* qrow = a.q + (int64_t)(t0 + (rvalid ? tl : tok_hi - 1)) * a.q_tok +
                          (int64_t)(g * G + row % G) * a.q_head;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      qt[t] = __builtin_bit_cast(bf16x8, ld16_cached(qrow + 2 * (16 * t + 8 * hf)));
  }

  // ---- loader geometry.  A wave loads kTile / W = 8 or 16 consecutive rows
  //      of every tile, which lie in one cache block (block_size >= 16):
  //      instruction k covers rows wrow + RPI k .. + RPI - 1, lane i takes
  //      row wrow + RPI k + i / CPR and LDS slot i % CPR, i.e. logical chunk
  //      (i % CPR) ^ f(row).
  constexpr int kWaveRows = kTile / W;
  static_assert(kWaveRows * W == kTile && kWaveRows <= 16, "a wave's rows of a tile stay in one block");
  const int wrow = kWaveRows * wave;
  auto fK = [](int r) { return (r / KRW) & (CPR - 1); };
  auto fV = [](int r) { return (CPR / 4) * (r & 3) + (CPR / 8) * ((r >> 2) & 1); };
  int koff[NLD], voff[NLD];
  if constexpr (FP8) {
    // lane i copies chunk i % SCH of row wrow + i / SCH (16 fp8 values);
    // d = 64: lane i of 32..63 the same chunk of V as lane i - 32 of K
    const int l = KV1 ? (lane & 31) : lane;
    koff[0] = (l / SCH) * (int)a.kg.slot + 16 * (l % SCH);
    voff[0] = (l / SCH) * (int)a.vg.slot + 16 * (l % SCH);
  } else {
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
      const int rr = RPI * k + lane / CPR, r = wrow + rr, s = lane % CPR;
      koff[k] = rr * (int)a.kg.slot + 16 * (s ^ fK(r));
      voff[k] = rr * (int)a.vg.slot + 16 * (s ^ fV(r));
    }
  }
  const uint8_t* kbase = a.k + (int64_t)g * a.kg.head;
  const uint8_t* vbase = a.v + (int64_t)g * a.vg.head;
  const uint32_t kblk = (uint32_t)a.kg.blk, vblk = (uint32_t)a.vg.blk;   // < 2^32 (host check)

  // Page of this wave's rows in tile tb + j, lane j (tiles tb .. tb + 63),
  // clamped into the cache so that a corrupt table cannot address outside it.
  int twin;
  int tb = 0;
  auto load_twin = [&](int first) {
    const int p = bt_row[min(bd.block(kTile * (first + lane) + wrow), last_blk)];
    twin = p < 0 ? 0 : (p >= a.num_blocks ? a.num_blocks - 1 : p);
  };
  load_twin(0);
  __builtin_amdgcn_s_waitcnt(0);   // Q and the window (one latency for both)

  // Loads of tile t, in parts so that the address work can sit between
  // matrix-core products: issue_prep(t) finds the wave's page of tile t
  // (rare: moves the window, draining the loads in flight), issue_kpart /
  // issue_vpart(t, k) send instruction k of NLD of its K / V into the tile's
  // ring stage.  With split rings the V tiles asked for trail the K tiles by
  // two, so a moved window starts two tiles back.
  constexpr int ND = 2 * NLD;   // load instructions per wave and tile
  constexpr int kLag = kSplit ? 2 : 0;
  const uint8_t* kp = kbase;
  const uint8_t* vp = vbase;
  auto issue_prep = [&](int t) {
    if (t - tb >= 64) {
      tb = uniform(max(t - kLag, 0));
      load_twin(tb);
      __builtin_amdgcn_s_waitcnt(0);
    }
    const uint32_t pg = (uint32_t)__builtin_amdgcn_readlane(twin, t - tb);
    const int rb = bd.slot(kTile * t + wrow);   // first row inside the block
    kp = kbase + (uint64_t)pg * kblk + (uint32_t)(rb * (int)a.kg.slot);
    vp = vbase + (uint64_t)pg * vblk + (uint32_t)(rb * (int)a.vg.slot);
  };
  auto issue_kpart = [&](int t, int k) {
    dma16(kp + koff[k], lds_addr(lds + kst(t) * TB + (wave * NLD + k) * 1024));
  };
  auto issue_vpart = [&](int t, int k) {
    dma16(vp + voff[k], lds_addr(lds + VBASE + vst(t) * TB + (wave * NLD + k) * 1024));
  };
  auto issue_k = [&](int t) {
    issue_prep(t);
#pragma unroll
    for (int k = 0; k < NLD; ++k) issue_kpart(t, k);
  };
  auto issue_v = [&](int t) {
    issue_prep(t);
#pragma unroll
    for (int k = 0; k < NLD; ++k) issue_vpart(t, k);
  };
  auto issue = [&](int t) {   // K and V of tile t (K, V alternating)
    issue_prep(t);
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
      issue_kpart(t, k);
      issue_vpart(t, k);
    }
  };
  // fp8: the wave's staging stage of tile t (K rows, then V rows at + 1 KB)
  auto stg_s = [&](int sg) { return SBASE + (sg * W + wave) * SWB; };   // staging stage sg
  auto stg = [&](int t) { return stg_s(t % SSTG); };
  auto issue8_k_s = [&](int sg) { dma16(kp + koff[0], lds_addr(lds + stg_s(sg))); };
  auto issue8_v_s = [&](int sg) { dma16(vp + voff[0], lds_addr(lds + stg_s(sg) + 1024)); };
  auto issue8_kv_s = [&](int sg) {   // d = 64: K rows to bytes 0..511, V rows to 512..1023
    dma16(lane < 32 ? kp + koff[0] : vp + voff[0], lds_addr(lds + stg_s(sg)));
  };
  auto issue8 = [&](int t) {
    issue_prep(t);
    if constexpr (KV1) {
      issue8_kv_s(t % SSTG);
    } else {
      issue8_k_s(t % SSTG);
      issue8_v_s(t % SSTG);
    }
  };
  // fp8: widen the wave's staged rows of tile t to bf16 in the K and V
  // rings, at the places the bf16 copies would have put them (its copies
  // of tile t have landed).  Lane i: row r8 = wrow + i / SCH, fp8 chunk
  // c8 = i % SCH, i.e. bf16 chunks 2 c8 and 2 c8 + 1, whose swizzled
  // slots differ in bit 0 (both swizzles keep it or flip it for the pair).
  // read8 fetches the 16 codes, put8_k / put8_v write the bf16 values.
  const int l8 = KV1 ? (lane & 31) : lane;
  const int r8 = wrow + l8 / SCH;
  const int w8k = r8 * RB + 16 * ((2 * (l8 % SCH)) ^ fK(r8));
  const int w8v = r8 * RB + 16 * ((2 * (l8 % SCH)) ^ fV(r8));
  // (The _s forms take the ring and staging stages of tile t as given.)
  auto read8_s = [&](int sg, int tensor) -> u32x4 {
    return *(const u32x4*)(lds + stg_s(sg) + 1024 * tensor + 16 * lane);
  };
  auto put8_k_s = [&](int ksg, const u32x4& raw) {
    bf16x8 lo, hi;
    fp8x16_to_bf16(raw, lo, hi);
    uint8_t* base = lds + ksg * TB;
    *(bf16x8*)(base + w8k) = lo;
    *(bf16x8*)(base + (w8k ^ 16)) = hi;
  };
  auto put8_v_s = [&](int vsg, int t, const u32x4& raw) {
    bf16x8 lo, hi;
    fp8x16_to_bf16(raw, lo, hi);
    if (t * kTile + r8 >= kv_len) {   // past the end: zeros (the bytes may be NaN codes)
      lo = bf16x8{};
      hi = bf16x8{};
    }
    uint8_t* base = lds + VBASE + vsg * TB;
    *(bf16x8*)(base + w8v) = lo;
    *(bf16x8*)(base + (w8v ^ 16)) = hi;
  };
  // d = 64: lanes 0..31 widen K rows, 32..63 V rows, from one read
  auto put8_kv_s = [&](int ksg, int vsg, int t, const u32x4& raw) {
    bf16x8 lo, hi;
    fp8x16_to_bf16(raw, lo, hi);
    const bool isv = lane >= 32;
    if (isv && t * kTile + r8 >= kv_len) {   // past the end: zeros (the bytes may be NaN codes)
      lo = bf16x8{};
      hi = bf16x8{};
    }
    const int off = isv ? VBASE + vsg * TB : ksg * TB;
    const int w8 = isv ? w8v : w8k;
    *(bf16x8*)(lds + off + w8) = lo;
    *(bf16x8*)(lds + off + (w8 ^ 16)) = hi;
  };
  auto widen8 = [&](int t) {   // tile t's copies have landed
    if constexpr (KV1) {
      put8_kv_s(kst(t), vst(t), t, read8_s(t % SSTG, 0));
    } else {
      put8_k_s(kst(t), read8_s(t % SSTG, 0));
      put8_v_s(vst(t), t, read8_s(t % SSTG, 1));
    }
  };
  // V rows at or past kv_len (last tile only) may hold anything, NaN
  // included, and would poison P V even with zero weights: each lane zeroes
  // the chunks it loaded, after its own loads have landed.
  auto zero_tail = [&](int t) {
    const int st = vst(t);
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
      const int r = RPI * (wave * NLD + k) + lane / CPR;
      if (t * kTile + r >= kv_len)
        *(u32x4*)(lds + VBASE + st * TB + (wave * NLD + k) * 1024 + 16 * lane) = u32x4{0, 0, 0, 0};
    }
  };

  // ---- operand addresses inside a stage
  int kaddr[NT];   // K row n (+ 32 kb), chunk 2t + hf
#pragma unroll
  for (int t = 0; t < NT; ++t) kaddr[t] = n * RB + 16 * ((2 * t + hf) ^ fK(n));
  int vaddr[NDB];  // V^T operand of d block db: source row 4hf + j/4, 4 d values at 32db + 16cb + 4(j&3)
  {
    const int j = lane & 15, cb = (lane >> 4) & 1;
    const int r = 4 * hf + (j >> 2);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int col = 32 * db + 16 * cb + 4 * (j & 3);
      vaddr[db] = VBASE + r * RB + 16 * ((col >> 3) ^ fV(r)) + 2 * (col & 7);
    }
  }

  f32x16 o[NDB];     // O^T accumulators
  f32x16 s[2];       // S^T of one tile (two 32-key halves)
  bf16x8 pb[4];      // P^T operands (four 16-key steps)
  float m_run = 0.f, l_run = 0.f;
  float psum = 0.f;                   // row sum of the tile in progress
  float alpha = 1.f;                  // O rescale owed before the next products
  uint64_t resc = 0;                  // (wave-uniform) some lane's alpha != 1
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;

  // ---- softmax pieces.  s = S = q . k; with c = scale * log2(e) the
  //      weight is 2^(c S - m_run), one fma and one exp (the fma rounds
  //      once, after the exact product).  Element e is s[e / 16][e % 16],
  //      key 8(e % 16 / 4) + 4 hf + e % 4 + 32 (e / 16) of the tile.  Causal
  //      mask of tile t (tiles crossing a diagonal only):
  auto mask = [&](int t) {
    const int lim = pos - t * kTile - 4 * hf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        s[kb][i] = (32 * kb + 8 * (i >> 2) + (i & 3)) <= lim ? s[kb][i] : kNegInf;
  };
  // Weights of elements 8u .. 8u + 7, 2^(c s - m), to the bf16 operand
  // pb[u]; the row sum adds the rounded weights (the ones the products use)
  // with dot2.  (Used for the first tile and where the reference moves; the
  // products' schedule splits the work into exp_pair and pack_group below.)
  auto group = [&](int u, float m) {
    const int kb = u >> 1, i0 = 8 * (u & 1);
    u32x4 pw;
#pragma unroll
    for (int h = 0; h < 4; ++h)
      pw[h] = pack_bf16(fast_exp2(__builtin_fmaf(s[kb][i0 + 2 * h], c, -m)),
                        fast_exp2(__builtin_fmaf(s[kb][i0 + 2 * h + 1], c, -m)));
    pb[u] = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int h = 0; h < 4; ++h) psum = dot2_bf16(pw[h], kOnesBf16x2, psum);
  };
  // The same split for the products' schedule: exp_pair(u, h) computes the
  // weights of elements 8u + 2h, 8u + 2h + 1 into ex[], pack_group(u)
  // writes pb[u] and the row sum.
  float ex[8];
  auto exp_pair = [&](int u, int h) {
    const int kb = u >> 1, i0 = 8 * (u & 1);
    ex[2 * h] = fast_exp2(__builtin_fmaf(s[kb][i0 + 2 * h], c, -m_run));
    ex[2 * h + 1] = fast_exp2(__builtin_fmaf(s[kb][i0 + 2 * h + 1], c, -m_run));
  };
  auto pack_group = [&](int u) {
    u32x4 pw;
#pragma unroll
    for (int h = 0; h < 4; ++h) pw[h] = pack_bf16(ex[2 * h], ex[2 * h + 1]);
    pb[u] = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int h = 0; h < 4; ++h) psum = dot2_bf16(pw[h], kOnesBf16x2, psum);
  };
  // Row max of the tile in log2 units (c S), across the lane pair.
  auto tile_max = [&]() {
    float mA = kNegInf, mB = kNegInf;
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      mA = fmaxf(fmaxf(mA, s[0][i]), s[0][i + 1]);
      mB = fmaxf(fmaxf(mB, s[1][i]), s[1][i + 1]);
    }
    return xor32_max(fmaxf(mA, mB)) * c;
  };
  // End of a tile's softmax.  The reference is kept while every weight of
  // the row stays below 2^12 (the lane's 32-key sum tells); otherwise it
  // moves up to the row max and the weights are recomputed, and O and l
  // owe the factor 2^-d.  m_run thus stays within 12 of the running max
  // and never above it.
  auto finish = [&]() {
    if (__ballot(psum > 4096.f)) {
      const float d = fmaxf(tile_max() - m_run, 0.f);
      m_run += d;
      alpha = fast_exp2(-d);
      resc = 1;
      l_run *= alpha;
      psum = 0.f;
#pragma unroll
      for (int u = 0; u < 4; ++u) group(u, m_run);
    }
    l_run += psum;
    psum = 0.f;
  };
  // Softmax work placed after product step p of the P V sequence (NP steps;
  // operand pb[u] is read by steps NDB u .. NDB u + NDB - 1, so its next
  // value may only be written after them).  group(3) and finish() follow
  // the sequence.
  constexpr int NS = 2 * NT;       // score products: (k-step tt, key half kb)
  constexpr int NP = 4 * NDB;      // PV products: (16-key step u, d block db)
  // Group u's weights are computed over the NDB steps that read pb[u] and
  // packed after the last of them; group 3 is packed after the sequence.
  auto valu_step = [&](int p) {
    const int u = p / NDB, q = p % NDB;
#pragma unroll
    for (int h = q * (4 / NDB); h < (q + 1) * (4 / NDB); ++h) exp_pair(u, h);
    if (q == NDB - 1 && u < 3) pack_group(u);
  };

  // Products of period t as one fixed sequence: scores of tile t + 1 (if
  // this wave needs it) over the K stage, then O^T += V^T P^T of tile t over
  // the V stage with the softmax of tile t + 1 spread between its steps.
  // LDS operands are read kAhead products ahead into a small register ring;
  // a scheduling fence after every product keeps each step's work in place.
  constexpr int kAhead = 4;
  static_assert(!FP8 || 14 < NS + NP, "fp8: widening and copies between the products");
  static_assert(kSplit ? 3 + 4 * NLD <= NS + NP : 2 + 3 * ND <= NS + 1,
                "tile loads fit between the products");
  auto period = [&](int t, auto full_tag, auto stage_tag) {
    constexpr bool kFullP = decltype(full_tag)::value;
    // t mod the unroll length of the main loop (a multiple of every ring's
    // size) where the caller knows it, else -1: then the stages of tile t + x
    // are constants and the LDS offsets immediates.
    constexpr int S4 = decltype(stage_tag)::value;
    auto kst_at = [&](int x) { return S4 >= 0 ? (S4 + x) % KSTG : kst(t + x); };
    auto vst_at = [&](int x) { return S4 >= 0 ? (S4 + x) % VSTG : vst(t + x); };
    auto sst_at = [&](int x) { return S4 >= 0 ? (S4 + x) % SSTG : (t + x) % SSTG; };
    const uint8_t* ks = lds + kst_at(1) * TB;
    uint8_t* vs = lds + vst_at(0) * TB;
    auto rd = [&](int i) -> bf16x8 {   // operand of product i (i < NS: K, else V^T)
      if (i < NS) return *(const bf16x8*)(ks + kaddr[i >> 1] + 32 * RB * (i & 1));
      const int u = (i - NS) / NDB, db = (i - NS) % NDB;
      uint8_t* p0 = vs + vaddr[db] + 16 * u * RB;
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(p0));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(p0 + 8 * RB));
      const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
      const u32x4 vw = {l2[0], l2[1], h2[0], h2[1]};
      return __builtin_bit_cast(bf16x8, vw);
    };
    constexpr int I0 = kFullP ? 0 : NS;
    bf16x8 ring[kAhead];
    u32x4 raw8;   // fp8: staged codes between their read and their widening
#pragma unroll
    for (int i = 0; i < kAhead; ++i) ring[i] = rd(I0 + i);
#pragma unroll
    for (int i = I0; i < NS + NP; ++i) {
      const bf16x8 op = ring[(i - I0) % kAhead];
      if (i < NS) {
        s[i & 1] = mfma32(op, qt[i >> 1], (i >> 1) == 0 ? f32x16{} : s[i & 1]);
      } else {
        const int p = i - NS;
        o[p % NDB] = mfma32(op, pb[p / NDB], o[p % NDB]);
      }
      if (i + kAhead < NS + NP) ring[(i - I0) % kAhead] = rd(i + kAhead);
      if constexpr (kFullP && FP8) {
        // widen tile t + 2 (copied two periods ago; tile t + 3's copies may
        // still fly), then copy tile t + 4 into the staging stage of t + 1
        if (t + 2 < ntiles) {
          if (i == 0) {
            if (t + 3 < ntiles) wait_vm<NCP>();
            else wait_vm<0>();
            raw8 = read8_s(sst_at(2), 0);
          }
          if constexpr (KV1) {
            if (i == 3) put8_kv_s(kst_at(2), vst_at(2), t + 2, raw8);
          } else {
            if (i == 3) put8_k_s(kst_at(2), raw8);
            if (i == 6) raw8 = read8_s(sst_at(2), 1);
            if (i == 9) put8_v_s(vst_at(2), t + 2, raw8);
          }
        }
        if (t + 4 < ntiles) {
          if (i == 11) issue_prep(t + 4);
          if constexpr (KV1) {
            if (i == 12) issue8_kv_s(sst_at(4));
          } else {
            if (i == 12) issue8_k_s(sst_at(4));
            if (i == 14) issue8_v_s(sst_at(4));
          }
        }
      }
      if constexpr (kFullP && !kSplit && !FP8) {
        // K and V of tile t + 3 between the score products, alternating
        if (t + 3 < ntiles) {
          if (i == 1) issue_prep(t + 3);
          if (i >= 2 && i < 2 + 3 * ND && (i - 2) % 3 == 0) {
            const int j = (i - 2) / 3;
            if (j & 1) dma16(vp + voff[j >> 1], lds_addr(lds + VBASE + vst_at(3) * TB + (wave * NLD + (j >> 1)) * 1024));
            else dma16(kp + koff[j >> 1], lds_addr(lds + kst_at(3) * TB + (wave * NLD + (j >> 1)) * 1024));
          }
        }
      }
      if constexpr (kFullP && kSplit) {
        // V of tile t + 1, then K of tile t + 3, one instruction every
        // second product
        if (t + 1 < ntiles) {
          if (i == 1) issue_prep(t + 1);
          if (i >= 2 && i < 2 + 2 * NLD && (i & 1) == 0)
            dma16(vp + voff[(i - 2) / 2], lds_addr(lds + VBASE + vst_at(1) * TB + (wave * NLD + (i - 2) / 2) * 1024));
        }
        if (t + 3 < ntiles) {
          if (i == 2 + 2 * NLD) issue_prep(t + 3);
          if (i >= 3 + 2 * NLD && i < 3 + 4 * NLD && ((i - 3) & 1) == 0)
            dma16(kp + koff[(i - 3 - 2 * NLD) / 2], lds_addr(lds + kst_at(3) * TB + (wave * NLD + (i - 3 - 2 * NLD) / 2) * 1024));
        }
      }
      if constexpr (kFullP) {
        if (i == NS - 1 && t + 1 >= nfull) mask(t + 1);
        if (i >= NS) valu_step(i - NS);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (kFullP) {
      pack_group(3);
      finish();
    }
  };

  if constexpr (GATHER) {
    if (ctx + tok_hi != min(a.seq_lens[seq], a.mb * a.block_size)) return;   // not the last Q-block
    const int64_t kd0 = (int64_t)seq * a.d_seq + (int64_t)g * a.d_head;
    if constexpr (FP8) {
      // each wave stores the raw codes of its staged rows
      const int r = wrow + l8 / SCH, c8 = l8 % SCH;
      for (int t = 0; t < ntiles; ++t) {
        issue8(t);
        wait_vm<0>();
        const int key = t * kTile + r;
        const u32x4 w0 = *(const u32x4*)(lds + stg(t) + 16 * lane);
        if constexpr (KV1) {   // lanes 0..31 hold K codes, 32..63 V codes
          if (key < kv_len) *(u32x4*)((lane < 32 ? a.kd : a.vd) + kd0 + (int64_t)key * a.d_tok + 16 * c8) = w0;
        } else {
          const u32x4 vw = *(const u32x4*)(lds + stg(t) + 1024 + 16 * lane);
          if (key < kv_len) {
            *(u32x4*)(a.kd + kd0 + (int64_t)key * a.d_tok + 16 * c8) = w0;
            *(u32x4*)(a.vd + kd0 + (int64_t)key * a.d_tok + 16 * c8) = vw;
          }
        }
      }
      return;
    }
    for (int t = 0; t < ntiles; ++t) {
      issue(t);
      wait_vm_lds<0>();
      __builtin_amdgcn_s_barrier();   // every wave's rows of tile t have landed
      // K: waves 0 / 1 store keys 0..31 / 32..63 from the operand addresses
      // (lane (n, hf), k-step tt: key n (+ 32), d = 16 tt + 8 hf .. + 7)
      if (wave < 2) {
        const int key = t * kTile + 32 * wave + n;
        if (key < kv_len)
#pragma unroll
          for (int tt = 0; tt < NT; ++tt)
            *(u32x4*)(a.kd + kd0 + (int64_t)key * a.d_tok + 16 * (2 * tt + hf)) =
                *(const u32x4*)(lds + kst(t) * TB + kaddr[tt] + 32 * RB * wave);
      }
      // V: each wave its own rows, chunk slot s holding logical chunk s ^ fV(row)
#pragma unroll
      for (int k = 0; k < NLD; ++k) {
        const int r = wrow + RPI * k + lane / CPR, c = (lane % CPR) ^ fV(r);
        const int key = t * kTile + r;
        if (key < kv_len)
          *(u32x4*)(a.vd + kd0 + (int64_t)key * a.d_tok + 16 * c) =
              *(const u32x4*)(lds + VBASE + vst(t) * TB + (wave * NLD + k) * 1024 + 16 * lane);
      }
      wait_vm_lds<0>();
      __builtin_amdgcn_s_barrier();   // the stages read by every wave before they are reused
    }
    return;
  }

  // ---- prologue: tiles 0, 1, 2 in flight (split rings: K of tiles 0, 1,
  //      V of tile 0, K of tile 2, in that order); scores and weights of
  //      tile 0, whose row max becomes the first reference
  if constexpr (FP8) {
    // tiles 0 .. 2 copied; 0 and 1 widened (2 may still fly), then tile 3
    // copied over tile 0's staging once its reads are done
    issue8(0);
    if (ntiles > 1) issue8(1);
    if (ntiles > 2) issue8(2);
    if (ntiles > 2) wait_vm<2 * NCP>();
    else if (ntiles == 2) wait_vm<NCP>();
    else wait_vm<0>();
    widen8(0);
    if (ntiles > 1) {
      if (ntiles > 2) wait_vm<NCP>();
      else wait_vm<0>();
      widen8(1);
    }
    wait_lds();
    if (ntiles > 3) issue8(3);
  } else if constexpr (!kSplit) {
    issue(0);
    if (ntiles > 1) issue(1);
    if (ntiles > 2) issue(2);
  } else {
    issue_k(0);
    if (ntiles > 1) issue_k(1);
    issue_v(0);
    if (ntiles > 2) issue_k(2);
  }
  auto wait_first = [&]() {   // tile 0's K (and V) landed; later loads may still fly
    if constexpr (!kSplit) {
      if (ntiles > 2) wait_vm_lds<2 * ND>();
      else if (ntiles == 2) wait_vm_lds<ND>();
      else wait_vm_lds<0>();
    } else {
      if (ntiles > 2) wait_vm_lds<3 * NLD>();
      else if (ntiles == 2) wait_vm_lds<2 * NLD>();
      else wait_vm_lds<0>();
    }
  };
  if constexpr (FP8) {
    wait_lds();
  } else {
    wait_first();
    if (ntiles == 1) zero_tail(0);
    wait_first();
  }
  __builtin_amdgcn_s_barrier();
  {
    const uint8_t* ks = lds;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      s[0] = mfma32(*(const bf16x8*)(ks + kaddr[tt]), qt[tt], tt == 0 ? f32x16{} : s[0]);
      s[1] = mfma32(*(const bf16x8*)(ks + kaddr[tt] + 32 * RB), qt[tt], tt == 0 ? f32x16{} : s[1]);
    }
  }
  if (0 >= nfull) mask(0);
  m_run = tile_max();   // finite: key 0 is never masked
#pragma unroll
  for (int u = 0; u < 4; ++u) group(u, m_run);
  l_run = psum;
  psum = 0.f;

  // ---- tile periods.  sync(t): K of tile t + 1 and V of tile t have
  //      landed for every wave and every wave has finished period t - 1, so
  //      the stages that held tile t - 1 (K of tile t with split rings) take
  //      this period's loads.  The O rescale owed by the softmax of tile t is
  //      applied before the products of tile t.
  auto sync = [&](int t) {
    if constexpr (FP8) {
      wait_lds();   // the rows this wave widened are written
    } else if constexpr (!kSplit) {
      // this wave's loads of tile t + 1 have landed (those of t + 2, if it
      // exists, may still fly)
      auto wait_next = [&]() {
        if (t + 2 < ntiles) wait_vm_lds<ND>();
        else wait_vm_lds<0>();
      };
      wait_next();
      if (t + 1 == ntiles - 1) zero_tail(t + 1);
      wait_next();
    } else {
      // K of tile t + 1 and V of tile t have landed (K of tile t + 2, issued
      // after them, may still fly)
      auto wait_next = [&]() {
        if (t + 2 < ntiles) wait_vm_lds<NLD>();
        else wait_vm_lds<0>();
      };
      wait_next();
      if (t == ntiles - 1) zero_tail(t);
      wait_next();
    }
    __builtin_amdgcn_s_barrier();
  };
  auto load_next = [&](int t) {   // period t's loads, outside the products
    if constexpr (FP8) {
      if (t + 2 < ntiles) {
        if (t + 3 < ntiles) wait_vm<NCP>();
        else wait_vm<0>();
        widen8(t + 2);
      }
      if (t + 4 < ntiles) issue8(t + 4);
    } else if constexpr (!kSplit) {
      if (t + 3 < ntiles) issue(t + 3);
    } else {
      if (t + 1 < ntiles) issue_v(t + 1);
      if (t + 3 < ntiles) issue_k(t + 3);
    }
  };
  auto rescale = [&]() {
    if (resc) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= alpha;
      resc = 0;
    }
  };
  constexpr std::true_type kFull{};
  constexpr std::false_type kPvOnly{};
  int t = 0;
  // Full periods, unrolled by L (a multiple of every ring's size: 4, 3 + 2
  // or 3) so that the stages inside them are constants; the rest one by one.
  constexpr std::integral_constant<int, -1> sN{};
  constexpr int L = FP8 ? 3 : (KSTG == 4 && VSTG == 4 ? 4 : 6);
  static_assert(L % KSTG == 0 && L % VSTG == 0 && (!FP8 || L % SSTG == 0), "unroll length");
  auto full = [&](int tt, auto stage_tag) {
    sync(tt);
    rescale();
    period(tt, kFull, stage_tag);   // issues this period's loads as well
  };
  auto unrolled = [&](auto... stage_tags) {
    for (; t + L < nact; t += L) (full(t + decltype(stage_tags)::value, stage_tags), ...);
  };
  using std::integral_constant;
  if constexpr (L == 3)
    unrolled(integral_constant<int, 0>{}, integral_constant<int, 1>{}, integral_constant<int, 2>{});
  else if constexpr (L == 4)
    unrolled(integral_constant<int, 0>{}, integral_constant<int, 1>{}, integral_constant<int, 2>{},
             integral_constant<int, 3>{});
  else
    unrolled(integral_constant<int, 0>{}, integral_constant<int, 1>{}, integral_constant<int, 2>{},
             integral_constant<int, 3>{}, integral_constant<int, 4>{}, integral_constant<int, 5>{});
  for (; t + 1 < nact; ++t) full(t, sN);
  sync(t);
  load_next(t);
  rescale();
  period(t, kPvOnly, sN);
  for (++t; t < ntiles; ++t) {
    sync(t);
    load_next(t);
  }

  // ---- finalise: out = O / l, bf16, staged through the K ring so that
  //      the stores write whole rows.  Every wave has finished its K reads
  //      (the last were before the last sync barrier) and no copy is in
  //      flight, so each wave writes its own 32 rows there (row-major,
  //      16-byte chunk c of row r at slot c ^ (r mod CPR)) and reads them
  //      back as 1 KB runs: 1024 / RB rows per store, 16 bytes per lane.
  const float l_tot = xor32_sum(l_run);
  const float inv = a.v_scale / l_tot;
  {
    uint8_t* orow_l = lds + row * RB;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = 4 * db + q;   // 16-byte chunk of d 32db + 8q .. + 7
        u32x2 w = {pack_bf16(o[db][4 * q] * inv, o[db][4 * q + 1] * inv),
                   pack_bf16(o[db][4 * q + 2] * inv, o[db][4 * q + 3] * inv)};
        *(u32x2*)(orow_l + 16 * (c ^ (row & (CPR - 1))) + 8 * hf) = w;
      }
  }
  constexpr int RPS = 1024 / RB;   // rows per store instruction
#pragma unroll
  for (int j = 0; j < kQblockWaveRows / RPS; ++j) {
    const int r = wave * kQblockWaveRows + j * RPS + lane / CPR, c = lane % CPR;
    const u32x4 w = *(const u32x4*)(lds + r * RB + 16 * (c ^ (r & (CPR - 1))));
    const int tr = tok_lo + r / G;
    if (tr < tok_hi)
      *(u32x4*)(a.out + (int64_t)(t0 + tr) * a.o_tok + (int64_t)(g * G + r % G) * a.o_head + 16 * c) = w;
  }
}

}  // namespace

hipError_t launch_qblock(const BatchArgs& a, const PrefillPlan& p, int head_dim, bool fp8,
                         hipStream_t st, bool gather, KernelTiming* tm) {
  const int64_t blocks = (int64_t)p.work_items * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  const int W = p.block_m / kQblockWaveRows;
  const dim3 grid((unsigned)blocks), block(64 * W);
  if (fp8) {
    if (W != 8) return hipErrorInvalidValue;
    if (head_dim == 128) {
      if (gather) launch_k(qblock_kernel<128, 8, true, true>, grid, block, st, tm, a, p);
      else launch_k(qblock_kernel<128, 8, true, false>, grid, block, st, tm, a, p);
    } else if (head_dim == 64) {
      if (gather) launch_k(qblock_kernel<64, 8, true, true>, grid, block, st, tm, a, p);
      else launch_k(qblock_kernel<64, 8, true, false>, grid, block, st, tm, a, p);
    } else {
      return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
#define PA_QB(DD, WW, GG) launch_k(qblock_kernel<DD, WW, false, GG>, grid, block, st, tm, a, p)
  if (W == 8) {
    if (head_dim == 128) gather ? PA_QB(128, 8, true) : PA_QB(128, 8, false);
    else if (head_dim == 64) gather ? PA_QB(64, 8, true) : PA_QB(64, 8, false);
    else return hipErrorInvalidValue;
  } else if (W == 4) {
    if (head_dim == 128) gather ? PA_QB(128, 4, true) : PA_QB(128, 4, false);
    else if (head_dim == 64) gather ? PA_QB(64, 4, true) : PA_QB(64, 4, false);
    else return hipErrorInvalidValue;
  } else {
    return hipErrorInvalidValue;
  }
#undef PA_QB
  return hipGetLastError();
}

}  // namespace pa

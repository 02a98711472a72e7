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
// Ping-pong: waves 0-3 and 4-7 form two groups with one wave of each on
// every SIMD, and the groups work half a tile period apart, separated by a
// workgroup barrier at every half period.  In one half a wave runs its
// matrix-core phase (scores of tile t + 1 and O += V^T P^T of tile t, LDS
// operand reads only) while the other wave on the SIMD runs its VALU phase
// (mask, row max, rescale, weights 2^(S scale - m) packed to bf16 for tile
// t + 1); in the next half they swap.  The matrix cores of a SIMD thus see
// one wave's products while its VALU serves the other wave's softmax.
//
// K/V tiles of 64 keys move from HBM into a ring of 4 LDS stages with
// global_load_lds_dwordx4 (no staging registers, no VALU), three tiles
// ahead of their use; each wave issues its share of a tile (whole 16-byte
// row chunks, 4 or 8 rows of one cache block per instruction, scalar page
// base).  The waits are explicit vmcnt counts, so the two tiles still in
// flight are never waited for.
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
// The running max is only raised when a row's tile max exceeds it by more
// than 8 (log2 units): the weights then stay below 2^8 and the final
// division uses the same reference, so the result is unchanged.
#include <type_traits>

#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kWaves = kQblockWaves;
constexpr int kThreads = 64 * kWaves;
constexpr int kTile = kPrefillTileKeys;
constexpr int kStages = 4;
constexpr int kNWin = 4;   // block-id registers per lane (a window of 256 blocks)

typedef short s16x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

// s_waitcnt with the vector-memory count bounded by N and every LDS
// operation drained (gfx9 encoding: vmcnt[3:0] and [15:14], expcnt[6:4],
// lgkmcnt[11:8]).
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0070);
}

template <int D>
__global__ __launch_bounds__(kThreads, 1) void qblock_kernel(BatchArgs a, PrefillPlan pp) {
  constexpr int RB = 2 * D;                        // bytes per cached row
  constexpr int CPR = D / 8;                       // 16-byte chunks per row
  constexpr int TB = kTile * RB;                   // bytes per K (or V) tile
  constexpr int RPI = 1024 / RB;                   // rows per load instruction
  constexpr int NLD = kTile / (RPI * kWaves);      // load instructions per wave, tile and tensor
  constexpr int KRW = 256 / RB;                    // K rows per 256-byte bank window
  constexpr int NT = D / 16;                       // k-steps of K Q^T
  constexpr int NDB = D / 32;                      // 32-row d blocks of O^T
  constexpr int VBASE = kStages * TB;              // V ring after the K ring
  static_assert(kQblockWaveRows == 32 && kWaves == 8, "two groups of 4 waves x 32 rows");
  static_assert(NLD >= 1 && NLD * RPI * kWaves == kTile, "tile loads");
  static_assert(RPI <= 16, "one instruction stays inside one 16-key block");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * kStages * TB];

  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int grp = wave >> 2;                       // ping-pong group
  const int n = lane & 31, hf = lane >> 5;
  const int Hkv = a.num_kv_heads;
  const int g = blockIdx.x % Hkv;
  const int wi = blockIdx.x / Hkv;
  const int G = a.group, BQ = pp.block_q, bsl = a.bs_log2, bsm = a.block_size - 1;

  if (wi >= pp.count[0]) return;
  const int seq = uniform(pp.list_seq[wi]);
  const int qb = uniform(pp.list_qb[wi]);
  const int t0 = uniform(a.qsl[seq]);
  const int qlen = uniform(a.qsl[seq + 1]) - t0;
  const int L = min(uniform(a.seq_lens[seq]), a.mb * a.block_size);
  const int ctx = L - qlen;
  if (ctx < 0 || t0 < 0 || t0 + qlen > a.num_tokens) return;
  const int tok_lo = qb * BQ;
  const int tok_hi = min(tok_lo + BQ, qlen);
  if (tok_lo >= tok_hi) return;
  const int kv_len = ctx + tok_hi;                 // keys the block needs
  const int ntiles = (kv_len + kTile - 1) / kTile;
  const int last_blk = (kv_len - 1) >> bsl;
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
  {
    const uint8_t* qrow = a.q + (int64_t)(t0 + (rvalid ? tl : tok_hi - 1)) * a.q_tok +
                          (int64_t)(g * G + row % G) * a.q_head;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      qt[t] = __builtin_bit_cast(bf16x8, ld16_cached(qrow + 2 * (16 * t + 8 * hf)));
  }

  // ---- loader geometry: instruction k of this wave covers tile rows
  //      r0 .. r0 + RPI - 1 (one cache block); lane i takes row r0 + i / CPR
  //      and LDS slot i % CPR, i.e. logical chunk (i % CPR) ^ f(row).
  auto fK = [](int r) { return (r / KRW) & (CPR - 1); };
  auto fV = [](int r) { return (CPR / 4) * (r & 3) + (CPR / 8) * ((r >> 2) & 1); };
  int koff[NLD], voff[NLD];
#pragma unroll
  for (int k = 0; k < NLD; ++k) {
    const int r = RPI * (wave * NLD + k) + lane / CPR, s = lane % CPR;
    koff[k] = (r & bsm) * (int)a.kg.slot + 16 * (s ^ fK(r));
    voff[k] = (r & bsm) * (int)a.vg.slot + 16 * (s ^ fV(r));
  }
  const uint8_t* kbase = a.k + (int64_t)g * a.kg.head;
  const uint8_t* vbase = a.v + (int64_t)g * a.vg.head;

  // Block ids of blocks wb .. wb + 64 kNWin - 1, one per lane and register.
  int win[kNWin];
  int wb = 0;
  auto load_window = [&](int first) {
#pragma unroll
    for (int q = 0; q < kNWin; ++q) win[q] = bt_row[min(first + 64 * q + lane, a.mb - 1)];
  };
  load_window(0);
  __builtin_amdgcn_s_waitcnt(0);   // Q and the window; nothing else in flight

  // Issue the loads of tile t into ring stage st.  Callers clamp t to the
  // last tile but keep st = (unclamped tile) % kStages, so a clamped re-load
  // never lands in the stage that holds the real last tile.
  // issue_part(t, st, j): instruction j of this wave's 2 NLD for the tile
  // (row group j / 2, K if j is even, else V).
  auto issue_part = [&](int t, int st, int j) {
    const int tsl = (t * kTile) & bsm;   // tile start inside its block (block_size > 64)
    const int k = j >> 1;
    {
      const int r0 = RPI * (wave * NLD + k);
      const int bi = min((t * kTile + r0) >> bsl, last_blk);
      const int rel = bi - wb;   // inside the window (ensure_window ran for t)
      int pg = __builtin_amdgcn_readlane(win[0], rel & 63);
#pragma unroll
      for (int q = 1; q < kNWin; ++q) {
        const int c = __builtin_amdgcn_readlane(win[q], rel & 63);
        pg = (rel >> 6) == q ? c : pg;
      }
      pg = pg < 0 ? 0 : (pg >= a.num_blocks ? a.num_blocks - 1 : pg);
      const int ldo = (wave * NLD + k) * 1024;
      // (the source is passed as void*: a const pointer here makes the host
      // pass drop the kernel's launch stub without a diagnostic)
      if ((j & 1) == 0) {
        const uint8_t* kp = kbase + (int64_t)pg * a.kg.blk + (int64_t)tsl * a.kg.slot;
        __builtin_amdgcn_global_load_lds((void*)(kp + koff[k]), (LDS_AS void*)(lds + st * TB + ldo), 16, 0, 0);
      } else {
        const uint8_t* vp = vbase + (int64_t)pg * a.vg.blk + (int64_t)tsl * a.vg.slot;
        __builtin_amdgcn_global_load_lds((void*)(vp + voff[k]), (LDS_AS void*)(lds + VBASE + st * TB + ldo),
                                         16, 0, 0);
      }
    }
  };
  constexpr int ND = 2 * NLD;   // load instructions per wave and tile
  // Make the window hold every block id tile t's loads need (tiles are
  // loaded in increasing order; the window moves to the tile's first block).
  // Rare: drains the loads in flight.
  auto ensure_window = [&](int t) {
    const int bl = min((t * kTile + kTile - 1) >> bsl, last_blk);
    if (bl >= wb + 64 * kNWin) {
      wb = uniform(min((t * kTile) >> bsl, last_blk));
      load_window(wb);
      __builtin_amdgcn_s_waitcnt(0);
    }
  };
  auto issue = [&](int t, int st) {
    ensure_window(t);
#pragma unroll
    for (int j = 0; j < ND; ++j) issue_part(t, st, j);
  };
  // V rows at or past kv_len (last tile only) may hold anything, NaN
  // included, and would poison P V even with zero weights: each lane zeroes
  // the chunks it loaded, after its own loads have landed.
  auto zero_tail = [&](int t) {
    const int st = t & (kStages - 1);
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
  float m_run = kNegInf, l_run = 0.f;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;

  // Matrix-core phase of period t: scores of tile t + 1 (if this wave needs
  // it) and O^T += V^T P^T of tile t (if this wave attends to it), as one
  // fixed sequence of products whose LDS operands are read kAhead products
  // ahead into a small register ring (a scheduling fence after every
  // product keeps the compiler from hoisting all reads at once).
  constexpr int NS = 2 * NT;       // score products: (k-step tt, key half kb)
  constexpr int NP = 4 * NDB;      // PV products: (16-key step u, d block db)
  constexpr int kAhead = 4;
  // mfma_phase(t, full): full = scores of tile t + 1 as well (else PV only).
  auto mfma_phase = [&](int t, auto full_tag) {
    const uint8_t* ks = lds + ((t + 1) & (kStages - 1)) * TB;
    uint8_t* vs = lds + (t & (kStages - 1)) * TB;
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
    auto run = [&](auto first_tag) {
      constexpr int I0 = decltype(first_tag)::value;   // 0: scores and PV, NS: PV only
      bf16x8 ring[kAhead];
#pragma unroll
      for (int i = 0; i < kAhead; ++i) ring[i] = rd(I0 + i);
#pragma unroll
      for (int i = I0; i < NS + NP; ++i) {
        const bf16x8 op = ring[(i - I0) % kAhead];
        if (i < NS) {
          s[i & 1] = mfma32(op, qt[i >> 1], s[i & 1]);
        } else {
          const int u = (i - NS) / NDB, db = (i - NS) % NDB;
          o[db] = mfma32(op, pb[u], o[db]);
        }
        if (i + kAhead < NS + NP) ring[(i - I0) % kAhead] = rd(i + kAhead);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    if constexpr (decltype(full_tag)::value) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
      run(std::integral_constant<int, 0>{});
    } else {
      run(std::integral_constant<int, NS>{});
    }
  };
  // VALU phase for tile t: causal mask (tiles crossing a diagonal), row max,
  // rescale of O when the max rises, weights packed to P^T operands.
  auto valu_phase = [&](int t) {
    if (t >= nfull) {
      const int lim = pos - t * kTile - 4 * hf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          s[kb][i] = (32 * kb + 8 * (i >> 2) + (i & 3)) <= lim ? s[kb][i] : kNegInf;
    }
    float m = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) m = fmaxf(m, s[kb][i]);
    const float mx = xor32_max(m) * a.sl2;
    if (__ballot(mx > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = fast_exp2(__builtin_fmaf(s[kb][i], a.sl2, -m_run));
        s[kb][i] = p;
        psum += p;
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r0 = 8 * h;
        const u32x4 pw = {pack_bf16(s[kb][r0 + 0], s[kb][r0 + 1]), pack_bf16(s[kb][r0 + 2], s[kb][r0 + 3]),
                          pack_bf16(s[kb][r0 + 4], s[kb][r0 + 5]), pack_bf16(s[kb][r0 + 6], s[kb][r0 + 7])};
        pb[2 * kb + h] = __builtin_bit_cast(bf16x8, pw);
      }
    }
    l_run += psum;
  };

  // ---- prologue: tiles 0, 1, 2 in flight; scores of tile 0 for all waves,
  //      weights of tile 0 for group 0 (group 1 takes them in its first
  //      VALU half)
  issue(0, 0);
  issue(min(1, ntiles - 1), 1);
  issue(min(2, ntiles - 1), 2);
  wait_vm_lds<4 * NLD>();
  if (ntiles == 1) zero_tail(0);
  wait_vm_lds<4 * NLD>();
  __builtin_amdgcn_s_barrier();
  {
    const uint8_t* ks = lds;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      s[0] = mfma32(*(const bf16x8*)(ks + kaddr[tt]), qt[tt], s[0]);
      s[1] = mfma32(*(const bf16x8*)(ks + kaddr[tt] + 32 * RB), qt[tt], s[1]);
    }
  }

  // ---- tile periods.  First half: group 0 matrix cores (tile t + 1 scores,
  //      tile t products), group 1 VALU (tile t weights); second half: the
  //      reverse.  Loads of tile t + 3 go into the stage of tile t - 1,
  //      which both groups finished in the previous period.  The groups run
  //      separate loops with the same
  //      barriers (a barrier counts waves, not code addresses), so that
  //      neither loop merges the other's register state.
  auto sync = [&](int t) {
    wait_vm_lds<2 * NLD>();   // this wave's loads of tile t + 1 have landed
    if (t + 1 == ntiles - 1) zero_tail(t + 1);
    wait_vm_lds<2 * NLD>();
    __builtin_amdgcn_s_barrier();
  };
  // Loads of tile t + 3 (into the stage of tile t - 1, free in period t).
  // Each group issues them in its VALU half, next to the short softmax
  // work, so that the issue stalls stay out of the matrix-core phases.
  auto load_next = [&](int t) { issue(min(t + 3, ntiles - 1), (t + 3) & (kStages - 1)); };
  auto half = [&]() {
    __builtin_amdgcn_s_waitcnt(0xc07f);   // this half's LDS reads done (vmcnt untouched)
    __builtin_amdgcn_s_barrier();
  };
  // Each wave: full periods while it needs the next tile's scores, one
  // period with the products of its last tile, then barriers only.
  constexpr std::true_type kFull{};
  constexpr std::false_type kPvOnly{};
  int t = 0;
  if (grp == 0) {
    valu_phase(0);
    for (; t + 1 < nact; ++t) {
      sync(t);
      mfma_phase(t, kFull);
      half();
      valu_phase(t + 1);
      load_next(t);
    }
    sync(t);
    mfma_phase(t, kPvOnly);
    half();
    load_next(t);
  } else {
    for (; t + 1 < nact; ++t) {
      sync(t);
      load_next(t);
      valu_phase(t);
      half();
      mfma_phase(t, kFull);
    }
    sync(t);
    load_next(t);
    valu_phase(t);
    half();
    mfma_phase(t, kPvOnly);
  }
  for (++t; t < ntiles; ++t) {
    sync(t);
    load_next(t);
    half();
  }
  // Clamped re-loads of the last tile may still be in flight: they must
  // land before the workgroup's LDS can be handed to another workgroup.
  __builtin_amdgcn_s_waitcnt(0);

  // ---- finalise: out = O / l, bf16
  const float l_tot = xor32_sum(l_run);
  if (rvalid) {
    const float inv = a.v_scale / l_tot;
    uint8_t* orow = a.out + (int64_t)(t0 + tl) * a.o_tok + (int64_t)(g * G + row % G) * a.o_head;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int d0 = 32 * db + 8 * q + 4 * hf;
        u32x2 w = {pack_bf16(o[db][4 * q] * inv, o[db][4 * q + 1] * inv),
                   pack_bf16(o[db][4 * q + 2] * inv, o[db][4 * q + 3] * inv)};
        *(u32x2*)(orow + 2 * d0) = w;
      }
  }
}

}  // namespace

hipError_t launch_qblock(const BatchArgs& a, const PrefillPlan& p, int head_dim, hipStream_t st) {
  const int64_t blocks = (int64_t)p.work_items * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  dim3 grid((unsigned)blocks), block(kThreads);
  if (head_dim == 128) qblock_kernel<128><<<grid, block, 0, st>>>(a, p);
  else if (head_dim == 64) qblock_kernel<64><<<grid, block, 0, st>>>(a, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa

// Varlen / chunked-prefill attention over a paged KV cache
// (arxiv 2511.11581, Sec. 4.4 Q-Blocks, Sec. 4.1 tiled softmax, Eq. 1-2).
//
// One workgroup = (Q-block, kv head g), 4 waves, BLOCK_M = 128 rows.  A
// Q-block packs BLOCK_Q = 128 / G consecutive query tokens of one sequence
// times the G query heads of kv head g; row r is (token r / G, head r % G).
// Only sequences with at least 2 query tokens are handled here (single-token
// rows go to the decode kernel).  K/V tiles of 64 keys are gathered through
// the block table with 16-byte loads into registers (prefetching the next
// tile while the current one is computed) and staged in LDS: K in natural
// row layout, V transposed.  Each wave owns 32 rows:
//   S^T[64 keys x 32 rows] = K Q^T   (v_mfma_f32_32x32x16_bf16)
//   online softmax, one lane per row; max/sum finish with a permlane32 swap
//   O^T[d x 32 rows]  += V^T P^T     (P^T taken from the S^T registers)
// Keys run from 0 to the largest prefix of the block; only tiles that cross
// the diagonal are masked.
//
// Work order: the grid enumerates (work item, kv head) with the kv head
// fastest, so all workgroups of one kv head land on the same XCD when
// Hkv = 8 and share its L2 for K/V.  Work item w is the w-th entry of a
// Q-block list that a one-workgroup plan kernel builds on the device, sorted
// by decreasing key count (heaviest Q-blocks first).
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kTileN = kPrefillTileKeys;  // keys per tile
constexpr int kThreads = 256;

// GATHER: only the last Q-block of each sequence runs its tile loads, and
// the loaded registers (raw cache bytes) of every valid key are stored into
// the dense outputs a.kd / a.vd (pa_debug_gather).
template <int D, bool FP8, bool GATHER>
__global__ __launch_bounds__(kThreads, 2) void prefill_kernel(BatchArgs a, PrefillPlan pp) {
  constexpr int EB = FP8 ? 1 : 2;
  constexpr int CH = D * EB / 16;                 // 16-byte chunks per cached row
  constexpr int KLD = kTileN * CH / kThreads;     // K loads per thread
  constexpr int VTASKS = 16 * CH;                 // (4-key group, chunk) pairs
  constexpr int DPC = 16 / EB;                    // d values per chunk
  constexpr int KROW = 2 * D + 16;                // LDS bytes per K row (bf16 + pad)
  constexpr int VROW = 2 * kTileN + 16;           // LDS bytes per V^T row
  constexpr int NT = D / 16;                      // 16-wide d steps of Q K^T
  constexpr int NDB = D / 32;                     // 32-row d blocks of O^T
  static_assert(KLD >= 1, "tile too small");

  // Two stages of (K tile, V^T tile): tile t lives in stage t & 1, so the
  // next tile is written while the current one is read (one barrier a tile).
  constexpr int KS_BYTES = kTileN * KROW, VT_BYTES = D * VROW;
  __shared__ __attribute__((aligned(16))) uint8_t stage_mem[2 * (KS_BYTES + VT_BYTES)];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hf = lane >> 5;
  const int Hkv = a.num_kv_heads;
  const int g = blockIdx.x % Hkv;
  const int wi = blockIdx.x / Hkv;
  const int G = a.group, BQ = pp.block_q;
  const BlockDiv bd = a.bdiv;   // block size: a multiple of 16

  if (wi >= pp.count[0]) return;
  const int seq = uniform(pp.list_seq[wi]);
  const int qb = uniform(pp.list_qb[wi]);

  const int t0 = a.qsl[seq];
  const int qlen = a.qsl[seq + 1] - t0;
  const int L = min(a.seq_lens[seq], a.mb * a.block_size);
  const int ctx = L - qlen;
  if (ctx < 0 || t0 < 0 || t0 + qlen > a.num_tokens) return;
  const int tok_lo = qb * BQ;                              // first token of the block
  const int tok_hi = min(tok_lo + BQ, qlen);               // one past the last
  const int kv_len = ctx + tok_hi;                         // keys needed by the block
  const int ntiles = (kv_len + kTileN - 1) / kTileN;
  const int32_t* bt_row = a.bt + (int64_t)seq * a.bt_row;

  // This lane's row.
  const int row = wave * 32 + n;
  const int tl = tok_lo + row / G;                         // token index inside the query
  const int hh = row % G;
  const bool rvalid = tl < tok_hi;
  const int pos = ctx + (rvalid ? tl : tok_hi - 1);        // absolute position (causal bound)
  const int wave_pos_max = ctx + min(tok_lo + (wave * 32 + 31) / G, tok_hi - 1);
  const int blk_pos_min = ctx + tok_lo;

  // Q^T B operands: d = 16t + 8hf + j of this row.
  bf16x8 qt[NT];
  if constexpr (!GATHER) {
    const uint8_t* qrow = a.q + (int64_t)(t0 + (rvalid ? tl : tok_hi - 1)) * a.q_tok +
                          (int64_t)(g * G + hh) * a.q_head;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      qt[t] = __builtin_bit_cast(bf16x8, ld16_cached(qrow + 2 * (16 * t + 8 * hf)));
  }

  // ---- loader geometry.  Tile t covers keys [64t, 64t + 64).  K load i of
  // this thread reads key kk_i = (tid + 256 i) / CH, 16-byte chunk tid % CH;
  // all keys of one wave's K load fall in one 16-key block, so its block-table
  // lookup is wave-uniform (scalar): the page and the slot of the group's
  // first key, the lanes' rows at fixed offsets from it.  V: thread (m = vt &
  // 15, c = vt >> 4) reads keys 4m..4m+3, chunk c (one lookup per thread).
  // Keys past kv_len read clamped block-table entries (at in-block slots) and
  // are zeroed when written to LDS.
  const int vtask = tid % VTASKS;
  const int vm = vtask & 15, vc = vtask >> 4;
  // (Offsets inside one block fit in 32 bits: the host checks
  // block_size * slot stride < 2^31.)
  int koff[KLD];
  int kkw[KLD];
#pragma unroll
  for (int i = 0; i < KLD; ++i) {
    const int kk = (tid + kThreads * i) / CH;
    kkw[i] = uniform(kk);   // the wave's first key of load i (lane 0's)
    koff[i] = (kk - kkw[i]) * (int)a.kg.slot + 16 * ((tid + kThreads * i) % CH);
  }
  const int voff = 16 * vc;
  const uint8_t* kbase = a.k + (int64_t)g * a.kg.head;
  const uint8_t* vbase = a.v + (int64_t)g * a.vg.head;
  const int last_blk = bd.block(kv_len - 1);
  auto page = [&](int bi) {   // table entry bi (<= the last needed block), clamped into the cache
    const int b = bt_row[min(bi, last_blk)];
    return b < 0 ? 0 : (b >= a.num_blocks ? a.num_blocks - 1 : b);
  };

  // Pages and in-block slots of the first keys of this thread's loads.
  int pg_k[KLD], sl_k[KLD], pg_v, sl_v;
  auto load_pages = [&](int tile) {
    const int tb = tile * kTileN;
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int key0 = uniform(tb + kkw[i]), bi = uniform(bd.block(key0));
      pg_k[i] = uniform(page(bi));
      sl_k[i] = uniform(key0 - a.block_size * bi);
    }
    const int kv0 = tb + 4 * vm, bv = bd.block(kv0);
    pg_v = page(bv);
    sl_v = kv0 - a.block_size * bv;
  };
  u32x4 kreg[KLD];
  u32x4 vreg[4];
  auto load_tile = [&]() {   // the tile whose pages load_pages found last
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const uint8_t* base = kbase + (int64_t)pg_k[i] * a.kg.blk + (int64_t)sl_k[i] * a.kg.slot;
      kreg[i] = ld16_cached(base + koff[i]);   // K/V are reused by other Q-blocks
    }
    const uint8_t* vb = vbase + (int64_t)pg_v * a.vg.blk + (int64_t)sl_v * a.vg.slot + voff;
#pragma unroll
    for (int r = 0; r < 4; ++r) vreg[r] = ld16_cached(vb + r * (int)a.vg.slot);
  };
  // ---- registers -> LDS (K natural bf16 rows, V transposed bf16)
  auto store_tile = [&](int tile) {
    const int tb = tile * kTileN;
    uint8_t* ks = stage_mem + (tile & 1) * (KS_BYTES + VT_BYTES);
    uint8_t* vts = ks + KS_BYTES;
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int flat = tid + kThreads * i;
      const int c = flat % CH, key = flat / CH;
      const u32x4 kw = tb + key < kv_len ? kreg[i] : u32x4{0, 0, 0, 0};
      uint8_t* dst = ks + key * KROW + 2 * DPC * c;
      if constexpr (FP8) {
        bf16x8 lo, hi;
        fp8x16_to_bf16(kw, lo, hi);
        *(bf16x8*)dst = lo;
        *(bf16x8*)(dst + 16) = hi;
      } else {
        *(u32x4*)dst = kw;
      }
    }
    if (tid < VTASKS) {
      // 16 consecutive threads share a chunk c and cover the 16 key groups,
      // so each 8-byte transposing write of a 16-lane group fills one
      // 128-byte V^T row segment without bank conflicts.
      u32x4 v4[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v4[r] = tb + 4 * vm + r < kv_len ? vreg[r] : u32x4{0, 0, 0, 0};
      // keys 4m..4m+3 -> V^T positions: bits 2 and 3 of the key swapped
      const int pb = 16 * (vm >> 2) + 8 * (vm & 1) + 4 * ((vm >> 1) & 1);
      uint8_t* wp = vts + (vc * DPC) * VROW + 2 * pb;
      if constexpr (FP8) {
        uint32_t w[4][8];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            u32x2 cv = fp8x4_to_bf16x4(v4[r][q]);
            w[r][2 * q] = cv[0];
            w[r][2 * q + 1] = cv[1];
          }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int dw = e >> 1;
          uint32_t lo, hi;
          if (e & 1) {
            lo = (w[0][dw] >> 16) | (w[1][dw] & 0xFFFF0000u);
            hi = (w[2][dw] >> 16) | (w[3][dw] & 0xFFFF0000u);
          } else {
            lo = (w[0][dw] & 0xFFFFu) | (w[1][dw] << 16);
            hi = (w[2][dw] & 0xFFFFu) | (w[3][dw] << 16);
          }
          *(u32x2*)(wp + e * VROW) = u32x2{lo, hi};
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int dw = e >> 1;
          uint32_t lo, hi;
          if (e & 1) {
            lo = (v4[0][dw] >> 16) | (v4[1][dw] & 0xFFFF0000u);
            hi = (v4[2][dw] >> 16) | (v4[3][dw] & 0xFFFF0000u);
          } else {
            lo = (v4[0][dw] & 0xFFFFu) | (v4[1][dw] << 16);
            hi = (v4[2][dw] & 0xFFFFu) | (v4[3][dw] << 16);
          }
          *(u32x2*)(wp + e * VROW) = u32x2{lo, hi};
        }
      }
    }
  };

  float m_run = kNegInf, l_run = 0.f;
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;

  // One tile of attention from LDS.  MASKED: the tile crosses the diagonal
  // of some row of the block (keys above a row's position are dropped).
  // The running max m_run is kept in scaled log2 units and only raised when
  // some row's tile max exceeds it by more than 8; otherwise the tile is
  // exponentiated against the stale max (weights stay below 2^8, and the
  // final division uses the same reference, so the result is unchanged).
  auto attend = [&](int tile, bool masked) {
    const int tb = tile * kTileN;
    const uint8_t* ks = stage_mem + (tile & 1) * (KS_BYTES + VT_BYTES);
    const uint8_t* vts = ks + KS_BYTES;
    // ---- S^T = K Q^T for 2 blocks of 32 keys; all K operands of a block are
    //      read before its MFMA chain so the LDS latency is paid once.
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 kop[NT];
      const uint8_t* kr = ks + (32 * kb + n) * KROW + 16 * hf;
#pragma unroll
      for (int t = 0; t < NT; ++t) kop[t] = *(const bf16x8*)(kr + 32 * t);
      __builtin_amdgcn_sched_barrier(0);
      f32x16 acc;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t) acc = mfma32(kop[t], qt[t], acc);
      sacc[kb] = acc;
    }
    if (masked) {
      // key (tb + 32kb + 8(i/4) + 4hf + i%4) is dropped when it exceeds pos
      const int lim = pos - tb - 4 * hf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          sacc[kb][i] = (32 * kb + 8 * (i >> 2) + (i & 3)) <= lim ? sacc[kb][i] : kNegInf;
    }
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kb][i]);
    mx = xor32_max(mx) * a.sl2;
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
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float pv = fast_exp2(__builtin_fmaf(sacc[kb][i], a.sl2, -m_run));
        sacc[kb][i] = pv;
        psum += pv;
      }
    l_run += psum;
    // ---- O^T += V^T P^T over 4 steps of 16 keys
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const f32x16& sp = sacc[u >> 1];
      const int r0 = 8 * (u & 1);
      u32x4 pw = {pack_bf16(sp[r0 + 0], sp[r0 + 1]), pack_bf16(sp[r0 + 2], sp[r0 + 3]),
                  pack_bf16(sp[r0 + 4], sp[r0 + 5]), pack_bf16(sp[r0 + 6], sp[r0 + 7])};
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
      bf16x8 vop[NDB];
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        vop[db] = *(const bf16x8*)(vts + (32 * db + n) * VROW + 2 * (16 * u + 8 * hf));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] = mfma32(vop[db], pb, o[db]);
    }
  };

  if constexpr (GATHER) {
    if (tok_hi != qlen) return;   // not the sequence's last Q-block
    const int64_t d0 = (int64_t)seq * a.d_seq + (int64_t)g * a.d_head;
    for (int tile = 0; tile < ntiles; ++tile) {
      const int tb = tile * kTileN;
      load_pages(tile);
      load_tile();
#pragma unroll
      for (int i = 0; i < KLD; ++i) {
        const int flat = tid + kThreads * i;
        const int key = tb + flat / CH;
        if (key < kv_len) *(u32x4*)(a.kd + d0 + (int64_t)key * a.d_tok + 16 * (flat % CH)) = kreg[i];
      }
      if (tid < VTASKS)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = tb + 4 * vm + r;
          if (key < kv_len) *(u32x4*)(a.vd + d0 + (int64_t)key * a.d_tok + 16 * vc) = vreg[r];
        }
    }
    return;
  }

  load_pages(0);
  load_tile();
  load_pages(min(1, ntiles - 1));
  store_tile(0);
  __syncthreads();

  // Tiles below every row's diagonal need no mask.  Per iteration: issue
  // the loads of tile + 1, attend to tile (stage tile & 1), write tile + 1
  // into the other stage, one barrier.
  const int nfull = min(ntiles, (blk_pos_min + 1) / kTileN);
  for (int tile = 0; tile < ntiles; ++tile) {
    const int tb = tile * kTileN;
    // Unconditional (clamped) prefetch keeps the waits exact: the store of
    // tile + 1 waits only for its own loads, not the younger page lookups.
    load_tile();                              // tile + 1 (clamped): pages found last iteration
    load_pages(min(tile + 2, ntiles - 1));
    __builtin_amdgcn_sched_barrier(0);
    if (tb <= wave_pos_max) attend(tile, uniform(tile >= nfull) != 0);
    if (tile + 1 < ntiles) store_tile(tile + 1);
    __syncthreads();
  }

  // ---- finalise: out = O / l, bf16
  const float l_tot = xor32_sum(l_run);
  if (rvalid) {
    const float inv = a.v_scale / l_tot;
    uint8_t* orow = a.out + (int64_t)(t0 + tl) * a.o_tok + (int64_t)(g * G + hh) * a.o_head;
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


hipError_t launch_prefill(const BatchArgs& a, const PrefillPlan& p, int head_dim, bool fp8,
                          hipStream_t st, bool gather) {
  if (!fp8 || head_dim == 128) return launch_qblock(a, p, head_dim, fp8, st, gather);
  const int64_t blocks = (int64_t)p.work_items * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  dim3 grid((unsigned)blocks), block(kThreads);
  if (head_dim == 128 && !gather) prefill_kernel<128, true, false><<<grid, block, 0, st>>>(a, p);
  else if (head_dim == 64 && !gather) prefill_kernel<64, true, false><<<grid, block, 0, st>>>(a, p);
  else if (head_dim == 128) prefill_kernel<128, true, true><<<grid, block, 0, st>>>(a, p);
  else if (head_dim == 64) prefill_kernel<64, true, true><<<grid, block, 0, st>>>(a, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa

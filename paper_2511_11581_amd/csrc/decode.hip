// Decode attention over a paged KV cache: persistent workers over an even
// split of the batch's key tiles, plus the log-sum-exp merge
// (arxiv 2511.11581, Sec. 4.4 GQA packing, Sec. 4.5 parallel tiled softmax,
// Sec. 4.7 static launch grid; Eq. 1-2 for what is computed).
//
// Only sequences whose query length is 1 are handled here.  The plan kernel
// lists them (j = 0..J-1) with the prefix P(j) of their step counts
// nt(j) = ceil(L_j / KS) (KS keys per step).  The kv heads are taken in
// units of HU adjacent heads (HU = 1 for 256-byte cache rows, 2 for 128-byte
// rows, 4 for 64-byte rows, as Hkv allows) that one wave computes together,
// so that its loads of one token cover a contiguous run of 256 bytes: HBM
// serves 128-byte rows at a 1 KB stride at little more than half the rate
// of 256-byte runs, even when two waves read the two halves at the same
// time.  The (sequence, unit) pairs, sequence-major, lay out a space of
// (Hkv / HU) P(J) steps: pair (j, gu) occupies
// [(Hkv / HU) P(j) + gu nt(j), + nt(j)).  Worker w of the W active workers
// (one wave each, launched as a fixed grid of 4-wave workgroups, one per
// CU) takes the contiguous range [worker_begin(w), worker_begin(w + 1)) of
// that space, so every worker streams the same number of K/V bytes
// whatever the lengths.  The part of one (sequence, kv head) pair inside one
// worker is a piece, i.e. a segment of the parallel tiled softmax: a piece
// covering its whole pair writes bf16 output; a piece cut at the worker's
// start (head) or end (tail) stores its unnormalised partials (acc, m, l),
// and merge_kernel combines the pieces of every pair that spans several
// workers.  A worker has at most one head and one tail unit piece, so
// partial slot (w, 0) holds the head pieces and (w, 1) tail-only pieces.
// Batches of short sequences (every pair within a few steps, known from the
// table width) take whole pairs instead: worker w computes pairs
// [w U / W, (w + 1) U / W) of the U pairs, W = min(U, workers), every piece
// covers its pair, and no merge follows (one launch fewer where the launch,
// not the keys, sets the time).
//
// Per wave and step: the G query heads of kv head g are the columns of one
// 16-wide MFMA tile, so every K/V row is read from HBM once.  K and V rows
// are read with whole-row coalesced loads (16 lanes per 256-byte row; lane l
// reads key 4r + (l & 3), bytes (l >> 2) * LB of the row), the next step's
// loads in flight while the current one is consumed.  Through the wave's
// private LDS area:
//   K  -> natural bf16 rows, read back as MFMA A operands (key rows),
//   V  -> V^T rows (one row per d), 16-byte transposing writes,
//   S^T[16 keys x 16 heads] = K Q^T, P = online softmax (log2 domain),
//   O^T[d x heads] += V^T P^T      (v_mfma_f32_16x16x32_bf16).
// MFMA row m of key block kb holds key 16kb + (m >> 2) + 4(m & 3), so the 8
// keys of one lane's P^T / V^T operand slots are exactly the 8 keys that one
// loading lane holds (all keys of the sub-tile congruent to l & 3 mod 4).
// A step is one sub-tile of 32 keys, or two for head_dim 64 (shorter rows:
// more keys per step keep the bytes in flight per wave up).
#include <type_traits>

#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kSub = 32;       // keys per sub-tile (one pass of the matrix cores)

// V^T row r (a d index), 16-byte column group cg (8 keys): rows are 64 bytes,
// 64 bytes of padding follow every 2^PSH rows (PSH = log2 of the d values a
// lane writes per row) and the column group is XOR-swizzled with bits 2..3
// of the row, so the transposing writes (8- and 16-lane groups) and the
// operand reads (32-lane groups) hit distinct LDS banks.
template <int PSH>
__device__ __forceinline__ int vt_off(int r, int cg) {
  return 16 * (4 * r + 4 * (r >> PSH) + (cg ^ ((r >> 2) & 3)));
}

template <int LB> struct LoadT;
template <> struct LoadT<16> { typedef u32x4 T; };
template <> struct LoadT<8> { typedef u32x2 T; };
template <> struct LoadT<4> { typedef uint32_t T; };

template <int LB>
__device__ __forceinline__ typename LoadT<LB>::T ldn(const uint8_t* p) {
  return __builtin_nontemporal_load((const typename LoadT<LB>::T*)p);
}
template <int LB>
__device__ __forceinline__ uint32_t dw(const typename LoadT<LB>::T& v, int i) {
  if constexpr (LB == 4) return v;
  else return v[i];
}

__device__ __forceinline__ int lane_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

// A contiguous range of steps of one (sequence, unit) pair (wave-uniform).
struct Piece {
  int j, s, t0, L, g;  // decode-list index, sequence, token row, length, first kv head
  int gu;              // unit (its heads are g = HU gu .. HU gu + HU - 1)
  int k0, k1;          // steps [k0, k1) of the pair
  int head, tail;      // the pair starts before / continues after this worker
};

// The log-sum-exp merge of one query head's n pieces (Sec. 4.5), by one
// wave: M = max_k m_k, out = sum_k 2^(m_k - M) acc_k / sum_k 2^(m_k - M) l_k,
// lanes over d; the result goes to row `tok`, query head g G + hh.  Piece k
// is read through ml_of(k) (its (m, l)) and po_of(k) (its d partials).  Up
// to 8 pieces are read in one round (every lane reads their (m, l)); more
// are read 64 (m, l) at a time, one per lane, their weights reaching the
// lanes by readlane.
template <int D, class MlOf, class PoOf>
__device__ __forceinline__ void merge_rows(const BatchArgs& a, int n, int hh, int tok, int g,
                                           MlOf ml_of, PoOf po_of) {
  constexpr int DPT = D / 64;   // d values per lane
  const int lane = threadIdx.x & 63;
  const int G = a.group;
  uint8_t* orow = a.out + (int64_t)tok * a.o_tok + (int64_t)(g * G + hh) * a.o_head + 2 * lane * DPT;
  auto store = [&](const float (&num)[DPT], float den) {
    const float inv = a.v_scale / den;
    if constexpr (DPT == 2) *(uint32_t*)orow = pack_bf16(num[0] * inv, num[1] * inv);
    else *(__bf16*)orow = (__bf16)(num[0] * inv);
  };
  if (n <= 8) {
    // Up to 8 pieces: their (m, l) (the same for every lane) and their
    // partials in one round of loads.
    f32x2 ml[8];
    float v[8][DPT];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = min(i, n - 1);
      ml[i] = ml_of(k);
      const float* po = po_of(k) + lane * DPT;
#pragma unroll
      for (int x = 0; x < DPT; ++x) v[i][x] = po[x];
    }
    float M = ml[0][0];
#pragma unroll
    for (int i = 1; i < 8; ++i) M = i < n ? fmaxf(M, ml[i][0]) : M;
    float num[DPT] = {}, den = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float wi = i < n ? fast_exp2(ml[i][0] - M) : 0.f;
      den += wi * ml[i][1];
#pragma unroll
      for (int x = 0; x < DPT; ++x) num[x] += wi * v[i][x];
    }
    store(num, den);
    return;
  }
  float M = kNegInf;
  for (int k0 = 0; k0 < n; k0 += 64) {
    const int k = k0 + lane;
    const float m = k < n ? ml_of(k)[0] : kNegInf;
    M = fmaxf(M, m);
  }
  M = xor16_max(M);
  M = xor32_max(M);
  M = fmaxf(M, __shfl_xor(M, 8));
  M = fmaxf(M, __shfl_xor(M, 4));
  M = fmaxf(M, __shfl_xor(M, 2));
  M = fmaxf(M, __shfl_xor(M, 1));
  float num[DPT] = {}, den = 0.f;
  for (int k0 = 0; k0 < n; k0 += 64) {
    const int k = k0 + lane;
    f32x2 ml = {kNegInf, 0.f};
    if (k < n) ml = ml_of(k);
    const float wk = k < n ? fast_exp2(ml[0] - M) : 0.f;
    den += wk * ml[1];
    const int kn = min(64, n - k0);
    // 8 pieces per round: their loads are independent and in flight together
    for (int i0 = 0; i0 < kn; i0 += 8) {
      float v[8][DPT];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int kk = min(i0 + i, kn - 1);
        const float* po = po_of(k0 + kk) + lane * DPT;
#pragma unroll
        for (int x = 0; x < DPT; ++x) v[i][x] = po[x];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float wi = i0 + i < kn ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wk), i0 + i)) : 0.f;
#pragma unroll
        for (int x = 0; x < DPT; ++x) num[x] += wi * v[i][x];
      }
    }
  }
  den = xor16_sum(den);
  den = xor32_sum(den);
  den += __shfl_xor(den, 8);
  den += __shfl_xor(den, 4);
  den += __shfl_xor(den, 2);
  den += __shfl_xor(den, 1);
  store(num, den);
}

// Pieces in the workspace: piece k sits with worker w0 + k (slot 1 for the
// pair's first worker, slot 0 for the others), head hu of its unit, query
// head hh of the group.
template <int D>
__device__ __forceinline__ void merge_pieces(const BatchArgs& a, const DecodePlan& p, int w0, int n,
                                             int hu, int hh, int tok, int g) {
  const int HU = p.unit_heads, G = a.group;
  auto row_of = [&](int k) { return (((int64_t)(w0 + k) * 2 + (k == 0 ? 1 : 0)) * HU + hu) * G + hh; };
  merge_rows<D>(
      a, n, hh, tok, g, [&](int k) { return *(const f32x2*)(p.part_ml + row_of(k) * 2); },
      [&](int k) { return (const float*)(p.part_o + row_of(k) * D); });
}

// GATHER: the same partition, block-table walk and loads, but every loaded
// row chunk of a valid key is stored into the dense outputs a.kd / a.vd
// instead of being computed with (pa_debug_gather).
template <int D, bool FP8, int HU, bool GATHER>
__global__ __launch_bounds__(64 * kDecodeWaves, 1) void decode_kernel(BatchArgs a, DecodePlan p) {
  constexpr int EB = FP8 ? 1 : 2;          // bytes per cached element
  constexpr int UB = HU * D * EB;          // bytes of one token's unit row (HU heads)
  constexpr int LB = UB / 16;              // bytes one lane loads per unit row
  constexpr int LPH = 16 / HU;             // lanes per head row
  constexpr int DPL = LB / EB;             // d values one lane loads per row
  constexpr int PSH = DPL == 16 ? 4 : (DPL == 8 ? 3 : 2);   // log2(DPL)
  constexpr int NW = DPL / 2;              // bf16 dwords per lane per row
  constexpr int NSTEP = D / 32;            // MFMA k-steps over d
  constexpr int NDB = D / 16;              // 16-row d blocks of O^T
  constexpr int KRB = 2 * D + 32;          // LDS bytes per K row (bf16 + pad)
  constexpr int KT = kSub * KRB;           // K sub-tile bytes
  constexpr int VT = 16 * (4 * D + 4 * (D >> PSH));  // V^T sub-tile bytes
  constexpr int HT = KT + VT;              // LDS bytes per head of the unit
  constexpr int WB = HU * HT;              // LDS bytes per wave
  constexpr int NSUB = decode_subtiles(UB, EB);  // sub-tiles per step
  constexpr int KS = kSub * NSUB;          // keys per step
  constexpr int R = 8 * NSUB;              // rows one lane loads per step (K and V each)
  constexpr int BPS = KS / 16;             // 16-key blocks per step
  typedef typename LoadT<LB>::T LT;
  static_assert(DPL == 16 || DPL == 8 || DPL == 4, "head_dim 64 or 128");
  static_assert(LPH * DPL == D, "lanes of one head row cover it");
  constexpr int NWIN = 4;                  // block-id registers per lane (window of 64 NWIN blocks)
  static_assert(64 % BPS == 0, "steps must not straddle block-id registers");

  // LDS sized so that one workgroup fills a CU (a second would not fit),
  // the rest of the CU's LDS for a decode list built here (fused launches).
  constexpr int kLdsBytes = decode_tile_lds(D, EB, HU);
  constexpr int kListCap = decode_list_cap(D, EB, HU);
  static_assert(WB == decode_wave_lds(D, EB, HU) && kLdsBytes >= kDecodeWaves * WB, "tile LDS");
  static_assert(HU * 16 * (4 * D + 8) <= WB, "a whole pair's partials (G <= 16) fit the wave's LDS");
  static_assert(kLdsBytes <= 160 * 1024 && 2 * kLdsBytes > 160 * 1024, "one workgroup per CU");
  __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsBytes];
  __shared__ int4 list_lds[GATHER ? 1 : kListCap + 1];

  const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
  const int q4 = lane >> 4, c16 = lane & 15;   // MFMA operand coordinates
  const int lq = lane & 3, lc = lane >> 2;     // loading coordinates
  const int hl = lc / LPH, ci = lc % LPH;      // head of the unit and chunk of its row this lane loads
  const int Hkv = a.num_kv_heads, G = a.group;
  const BlockDiv bd = a.bdiv;   // block size: a multiple of 16, so no 16-key block straddles two

  const int w = blockIdx.x * kDecodeWaves + wave;
  const int Hu = Hkv / HU;                     // units per sequence
  // The decode list: built by the plan kernel, or (fused launches, decode-
  // only batches) by this workgroup in LDS, the same pass over the
  // sequences as the plan kernel's.
  int J, Wn;
  const int4* dec = p.dec;
  if (!GATHER && p.fused) {
    const int tid = threadIdx.x, S = a.num_seqs, cap = a.mb * a.block_size;
    int nj = 0, nsteps = 0;
    for (int b0 = 0; b0 < S; b0 += 64 * kDecodeWaves) {
      const int i = b0 + tid;
      int v[2] = {0, 0}, t0 = 0, L = 0;
      if (i < S) {
        t0 = a.qsl[i];
        const int q = a.qsl[i + 1] - t0;
        L = min(a.seq_lens[i], cap);
        if (q == 1 && t0 >= 0 && t0 < a.num_tokens && L >= 1) {
          v[0] = 1;
          v[1] = (L + p.step_keys - 1) / p.step_keys;
        }
      }
      int ex[2], tot[2];
      block_scan<2, 64 * kDecodeWaves>(v, ex, tot);
      if (v[0] && nj + ex[0] < kListCap) list_lds[nj + ex[0]] = make_int4(i, t0, L, nsteps + ex[1]);
      nj += tot[0];
      nsteps += tot[1];
    }
    nj = min(nj, kListCap);   // (the host launches fused only for S < kListCap)
    if (tid == 0) list_lds[nj] = make_int4(0, 0, 0, nsteps);
    __syncthreads();
    J = nj;
    Wn = active_workers((int64_t)Hu * nsteps, p.min_steps, p.workers);
    dec = list_lds;
    if (blockIdx.x == 0 && !p.whole_units) {   // the merge kernel, launched next, reads the list from the workspace
      for (int i = tid; i <= nj; i += 64 * kDecodeWaves) p.dec[i] = list_lds[i];
      if (tid == 0) {
        p.meta[0] = J;
        p.meta[1] = Wn;
        p.meta[2] = nsteps;
      }
    }
  } else {
    J = p.meta[0];
    Wn = p.meta[1];
  }
  if (J <= 0) return;
  const int64_t Ttot = (int64_t)Hu * dec[J].w;

  // Steps [t, t_end) of the step space, piece by piece.
  auto run = [&](int64_t t, const int64_t t_end) {

    // ---- first unit: largest j with Hu * P(j) <= t, by a 64-ary search; the
    //      wave then holds entries base .. base + 63 of the list, one per lane.
    int lo = 0, hi = J;
    while (hi - lo > 63) {
      const int step = (hi - lo + 63) / 64;
      const int idx = lo + lane * step;
      const int64_t P = (int64_t)Hu * dec[min(idx, J)].w;
      const bool ok = idx < hi && P <= t;
      lo += (63 - __builtin_clzll(__ballot(ok))) * step;
      hi = min(hi, lo + step);
    }
    int base = lo;
    int4 ent = dec[min(base + lane, J)];
    {
      const bool ok = base + lane < hi && (int64_t)Hu * ent.w <= t;
      lo = base + (63 - __builtin_clzll(__ballot(ok)));
    }
    // Entry jj of the list (jj + 1 - base <= 63 must hold): fields by readlane.
    auto reload = [&](int jj) {   // rare: the wait below drains everything in flight
      base = jj;
      ent = dec[min(base + lane, J)];
      __builtin_amdgcn_s_waitcnt(0);
    };

    // Block-table entries of the 64 * NWIN 16-key blocks starting at `first`
    // (register i, lane l: block first + 64 i + l), loaded from clamped
    // indices; entries past the sequence end are never used for a valid key,
    // and every entry is clamped into [0, num_blocks) at its use.
    auto load_window = [&](const Piece& pc, int first, int (&win)[NWIN]) {
      const int32_t* bt_row = a.bt + (int64_t)pc.s * a.bt_row;
  #pragma unroll
      for (int i = 0; i < NWIN; ++i) win[i] = bt_row[min(bd.block((first + 64 * i + lane) * 16), a.mb - 1)];
    };
    auto make_piece = [&](int jj, int gu, int k0, int64_t budget) {
      if (jj + 1 - base > 63) reload(jj);
      Piece pc;
      jj = uniform(jj);
      pc.j = jj;
      pc.gu = uniform(gu);
      pc.s = lane_i(ent.x, jj - base);
      pc.t0 = lane_i(ent.y, jj - base);
      pc.L = min(lane_i(ent.z, jj - base), a.mb * a.block_size);
      const int nt = lane_i(ent.w, jj + 1 - base) - lane_i(ent.w, jj - base);
      pc.g = uniform(gu * HU);
      pc.k0 = uniform(k0);
      pc.k1 = uniform((int)min((int64_t)nt, (int64_t)k0 + budget));
      pc.head = pc.k0 > 0;
      pc.tail = pc.k1 < nt;
      return pc;
    };
    // Q^T of a piece as MFMA B operands, per head hu of the unit: column c16
    // = query head (g + hu) G + c16 (zero if c16 >= G), k-step st covers
    // d = 32 st + 8 q4 + j.
    auto load_q = [&](const Piece& pc, bf16x8 (&qt)[HU][NSTEP]) {
      const bool hv = c16 < G;
  #pragma unroll
      for (int hu = 0; hu < HU; ++hu) {
        const uint8_t* qrow = a.q + (int64_t)pc.t0 * a.q_tok + (int64_t)((pc.g + hu) * G + (hv ? c16 : 0)) * a.q_head;
  #pragma unroll
        for (int st = 0; st < NSTEP; ++st) {
          u32x4 v = hv ? ld16_cached(qrow + 2 * (32 * st + 8 * q4)) : u32x4{0, 0, 0, 0};
          qt[hu][st] = __builtin_bit_cast(bf16x8, v);
        }
      }
    };

    Piece cur;
    {
      const int64_t Pj = lane_i(ent.w, lo - base);
      const int nt = lane_i(ent.w, lo + 1 - base) - (int)Pj;
      const int64_t off = t - (int64_t)Hu * Pj;
      cur = make_piece(lo, (int)(off / nt), (int)(off % nt), t_end - t);
    }
    bf16x8 qc[HU][NSTEP];
    int win[NWIN];
    int cb = 0;   // first 16-key block of the window held in win

    float m_run[HU], l_run[HU];
    f32x4 o[HU][NDB];
  #pragma unroll
    for (int hu = 0; hu < HU; ++hu) {
      m_run[hu] = kNegInf;
      l_run[hu] = 0.f;
  #pragma unroll
      for (int db = 0; db < NDB; ++db) o[hu][db] = f32x4{0, 0, 0, 0};
    }
    // Per head of the unit: a K tile (natural rows) and a V^T tile.
    uint8_t* const wl = lds + wave * WB;
    auto kl = [&](int hu) { return wl + hu * HT; };
    auto vt = [&](int hu) { return wl + hu * HT + KT; };

    // Issue the K/V loads of step k of a pair (kv head g, block cache `cache`
    // starting at 16-key block cb); live = 0 issues harmless loads of one row.
    // Addresses: a wave-uniform (scalar) base per 4-row group and a fixed
    // 32-bit per-lane offset (row lq of the group, head hl of the unit, chunk
    // ci of that head's row).
    const uint32_t koff = (uint32_t)(lq * a.kg.slot + hl * a.kg.head + ci * LB);
    const uint32_t voff = (uint32_t)(lq * a.vg.slot + hl * a.vg.head + ci * LB);
    // Issue the K (or V) loads of step k of the current piece (block ids from
    // the window registers; refill() must have made the step's blocks resident).
    auto issue = [&](const uint8_t* base, const KvGeom& geo, uint32_t off, int k, LT (&rows)[R]) {
      const int blk0 = uniform(k * BPS - cb);
  #pragma unroll
      for (int b = 0; b < BPS; ++b) {
        const int bi = blk0 + b;   // never straddles registers: 64 % BPS == 0
        int pg = lane_i(win[0], bi & 63);
  #pragma unroll
        for (int i = 1; i < NWIN; ++i) pg = (bi >> 6) == i ? lane_i(win[i], bi & 63) : pg;
        pg = pg < 0 ? 0 : (pg >= a.num_blocks ? a.num_blocks - 1 : pg);
        const int sb = bd.slot(k * KS + 16 * b);   // slot of the 16-key block's first key
        const uint8_t* bp = base + (int64_t)pg * geo.blk + (int64_t)cur.g * geo.head + (int64_t)sb * geo.slot;
  #pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) rows[4 * b + r4] = ldn<LB>(bp + 4 * r4 * geo.slot + off);
      }
    };
    // bf16 words of one loaded row chunk (DPL values of one key).
    auto to_bf16 = [&](const LT& v, uint32_t (&wd)[NW]) {
      if constexpr (FP8) {
  #pragma unroll
        for (int q = 0; q < LB / 4; ++q) {
          const u32x2 cv = fp8x4_to_bf16x4(dw<LB>(v, q));
          wd[2 * q] = cv[0];
          wd[2 * q + 1] = cv[1];
        }
      } else {
  #pragma unroll
        for (int q = 0; q < NW; ++q) wd[q] = dw<LB>(v, q);
      }
    };
    // Scores and online-softmax update for step k of the current piece; the
    // probabilities P^T of sub-tile u (as MFMA B operands) go to pt[u].
    auto consume_k = [&](int k, LT (&kr)[R], bf16x8 (&pt)[HU][NSUB]) {
      f32x4 sacc[HU][NSUB][2];
  #pragma unroll
      for (int u = 0; u < NSUB; ++u) {
        // ---- K rows -> LDS (bf16, natural layout), into the tile of head hl
  #pragma unroll
        for (int r = 0; r < 8; ++r) {
          uint32_t wd[NW];
          to_bf16(kr[8 * u + r], wd);
          uint8_t* dst = kl(hl) + (4 * r + lq) * KRB + ci * (2 * DPL);
          if constexpr (NW == 8) {
            *(u32x4*)dst = u32x4{wd[0], wd[1], wd[2], wd[3]};
            *(u32x4*)(dst + 16) = u32x4{wd[4], wd[5], wd[6], wd[7]};
          } else if constexpr (NW == 4) {
            *(u32x4*)dst = u32x4{wd[0], wd[1], wd[2], wd[3]};
          } else {
            *(u32x2*)dst = u32x2{wd[0], wd[1]};
          }
        }
        // ---- S^T = K Q^T per head; MFMA row c16 of block kb is key 16kb + (c16>>2) + 4(c16&3)
  #pragma unroll
        for (int hu = 0; hu < HU; ++hu)
  #pragma unroll
          for (int kb = 0; kb < 2; ++kb) {
            f32x4 acc = {0, 0, 0, 0};
            const uint8_t* kp = kl(hu) + (16 * kb + (c16 >> 2) + 4 * (c16 & 3)) * KRB + 16 * q4;
  #pragma unroll
            for (int st = 0; st < NSTEP; ++st)
              acc = mfma16(*(const bf16x8*)(kp + 64 * st), qc[hu][st], acc);
            sacc[hu][u][kb] = acc;
          }
      }
      // ---- online softmax (log2 domain); lane holds keys 32u + 16kb + q4 + 4r of head c16
      const int kend = uniform(cur.L - k * KS);   // keys of this step inside the sequence
      if (kend < KS) {   // last step of the pair: mask keys >= L (compare with immediates)
        const int lim = kend - q4;
  #pragma unroll
        for (int hu = 0; hu < HU; ++hu)
  #pragma unroll
          for (int u = 0; u < NSUB; ++u)
  #pragma unroll
            for (int kb = 0; kb < 2; ++kb)
  #pragma unroll
              for (int r = 0; r < 4; ++r)
                sacc[hu][u][kb][r] = kSub * u + 16 * kb + 4 * r < lim ? sacc[hu][u][kb][r] : kNegInf;
      }
  #pragma unroll
      for (int hu = 0; hu < HU; ++hu) {
        float mx = kNegInf;
  #pragma unroll
        for (int u = 0; u < NSUB; ++u)
  #pragma unroll
          for (int kb = 0; kb < 2; ++kb)
  #pragma unroll
            for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sacc[hu][u][kb][r]);
        mx = xor16_max(mx);
        mx = xor32_max(mx) * a.sl2;
        // The reference max m_run is only raised when some query head's step
        // max exceeds it by more than 8 (log2 units): the weights then stay
        // below 2^8, and l, O and the stored partials all use the same
        // reference, so the result is unchanged while O is rescaled on few
        // steps only.
        if (__ballot(mx > m_run[hu] + 8.f)) {
          const float m_new = fmaxf(m_run[hu], mx);
          const float alpha = fast_exp2(m_run[hu] - m_new);
          m_run[hu] = m_new;
          l_run[hu] *= alpha;
  #pragma unroll
          for (int db = 0; db < NDB; ++db) o[hu][db] *= alpha;
        }
        float psum = 0.f;
  #pragma unroll
        for (int u = 0; u < NSUB; ++u) {
          float x[2][4];
  #pragma unroll
          for (int kb = 0; kb < 2; ++kb)
  #pragma unroll
            for (int r = 0; r < 4; ++r) {
              x[kb][r] = fast_exp2(__builtin_fmaf(sacc[hu][u][kb][r], a.sl2, -m_run[hu]));
              psum += x[kb][r];
            }
          const u32x4 pw = {pack_bf16(x[0][0], x[0][1]), pack_bf16(x[0][2], x[0][3]),
                            pack_bf16(x[1][0], x[1][1]), pack_bf16(x[1][2], x[1][3])};
          pt[hu][u] = __builtin_bit_cast(bf16x8, pw);
        }
        l_run[hu] += psum;
      }
    };
    // V^T column group of sub-tile u for d value e of this lane's chunk: the
    // bf16 pairs (row 2jj, row 2jj + 1) for jj = 0..3, taken straight from the
    // loaded row chunks (v_perm pairs the 16-bit halves, or the fp8 bytes,
    // which one conversion then widens); with MASK, rows of keys >= kend
    // (lim = kend - lq) read as zero, as their slots may hold NaN.
    auto vt_col = [&](LT (&vr)[R], int u, int e, int lim, auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      u32x4 col;
  #pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int r0 = 8 * u + 2 * jj, r1 = r0 + 1;
        uint32_t w0, w1;
        if constexpr (FP8) {
          w0 = dw<LB>(vr[r0], e >> 2);
          w1 = dw<LB>(vr[r1], e >> 2);
        } else {
          w0 = dw<LB>(vr[r0], e >> 1);
          w1 = dw<LB>(vr[r1], e >> 1);
        }
        if constexpr (MASK) {
          w0 = kSub * u + 4 * (2 * jj) < lim ? w0 : 0u;
          w1 = kSub * u + 4 * (2 * jj + 1) < lim ? w1 : 0u;
        }
        if constexpr (FP8) {
          const uint32_t bsel = (uint32_t)(e & 3);
          const uint32_t pair = __builtin_amdgcn_perm(w1, w0, bsel | ((4u + bsel) << 8) | 0x0C0C0000u);
          col[jj] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(pair, 1.0f, false));
        } else {
          col[jj] = __builtin_amdgcn_perm(w1, w0, (e & 1) ? 0x07060302u : 0x05040100u);
        }
      }
      return col;
    };
    // O^T += V^T P^T for step k of the current piece.
    auto consume_v = [&](int k, LT (&vr)[R], const bf16x8 (&pt)[HU][NSUB]) {
      const int kend = uniform(cur.L - k * KS);
      const int lim = kend - lq;
  #pragma unroll
      for (int u = 0; u < NSUB; ++u) {
        // ---- V -> V^T: this lane's 8 keys (4r + lq, r = 0..7) are the 8
        //      consecutive positions of column group lq.
        if (kend < KS) {
  #pragma unroll
          for (int e = 0; e < DPL; ++e)
            *(u32x4*)(vt(hl) + vt_off<PSH>(ci * DPL + e, lq)) = vt_col(vr, u, e, lim, std::true_type{});
        } else {
  #pragma unroll
          for (int e = 0; e < DPL; ++e)
            *(u32x4*)(vt(hl) + vt_off<PSH>(ci * DPL + e, lq)) = vt_col(vr, u, e, lim, std::false_type{});
        }
        // ---- O^T += V^T P^T per head
  #pragma unroll
        for (int hu = 0; hu < HU; ++hu)
  #pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const u32x4 va = *(const u32x4*)(vt(hu) + vt_off<PSH>(16 * db + c16, q4));
            o[hu][db] = mfma16(__builtin_bit_cast(bf16x8, va), pt[hu][u], o[hu][db]);
          }
      }
    };
    // End of a piece: bf16 output if the piece is its whole pair, else
    // partials (rows [wave, slot, head of the unit, query head]).
    auto finalize = [&]() {
  #pragma unroll
      for (int hu = 0; hu < HU; ++hu) {
        float l_tot = xor16_sum(l_run[hu]);
        l_tot = xor32_sum(l_tot);
        if (c16 < G) {
          if (!cur.head && !cur.tail) {
            const float inv = a.v_scale / l_tot;
            uint8_t* orow = a.out + (int64_t)cur.t0 * a.o_tok + (int64_t)((cur.g + hu) * G + c16) * a.o_head;
  #pragma unroll
            for (int db = 0; db < NDB; ++db) {
              const u32x2 v2 = {pack_bf16(o[hu][db][0] * inv, o[hu][db][1] * inv),
                                pack_bf16(o[hu][db][2] * inv, o[hu][db][3] * inv)};
              *(u32x2*)(orow + 2 * (16 * db + 4 * q4)) = v2;
            }
          } else if (!GATHER && p.whole_units) {
            // the workgroup merges this pair: the partials stay in this
            // wave's LDS ([HU G][d] floats, then [HU G] (m, l)), free since
            // the piece's last products read their operands
            float* po = (float*)wl + (hu * G + c16) * D;
  #pragma unroll
            for (int db = 0; db < NDB; ++db) *(f32x4*)(po + 16 * db + 4 * q4) = o[hu][db];
            if (q4 == 0) *(f32x2*)((float*)wl + HU * G * D + (hu * G + c16) * 2) = f32x2{m_run[hu], l_tot};
          } else {
            const int64_t row = (((int64_t)w * 2 + (cur.head ? 0 : 1)) * HU + hu) * G + c16;
            float* po = p.part_o + row * D;
  #pragma unroll
            for (int db = 0; db < NDB; ++db) *(f32x4*)(po + 16 * db + 4 * q4) = o[hu][db];
            if (q4 == 0) *(f32x2*)(p.part_ml + row * 2) = f32x2{m_run[hu], l_tot};
          }
        }
        m_run[hu] = kNegInf;
        l_run[hu] = 0.f;
  #pragma unroll
        for (int db = 0; db < NDB; ++db) o[hu][db] = f32x4{0, 0, 0, 0};
      }
    };

    // Software pipeline over the worker's steps (two register sets, loop
    // unrolled by two).  Every half issues the loads of the next step (of the
    // current piece, else the first step of the next piece) unconditionally,
    // so that each wait covers only the older set; sched_barrier keeps the
    // compiler from hoisting the consumer's first instructions above them.
    // Make the blocks of step k resident in the window registers (a new window
    // starts at the step's first block; the load is waited for at its use).
    auto refill = [&](int k) {
      if (k * BPS >= cb + 64 * NWIN) {   // rare: drains the loads in flight
        cb = uniform(k * BPS);
        load_window(cur, cb, win);
        __builtin_amdgcn_s_waitcnt(0);
      }
    };

    // Per piece: block ids and query rows, then a software pipeline over its
    // steps with one step in flight, skewed by half a step: while step k is
    // consumed, the K loads of step k + 1 are issued before its scores and the
    // V loads before its P V product, so that step k's K registers are free
    // before step k + 1's V registers fill.  Two register sets, loop unrolled
    // by two with an exact tail; every issue in the loop body is
    // unconditional so that each wait covers only the older set, and
    // sched_barrier keeps the compiler from hoisting consumers above the loads.
    LT krA[R], vrA[R], krB[R], vrB[R];
    auto step = [&](int k, bool more, LT (&kx)[R], LT (&vx)[R], LT (&kz)[R], LT (&vz)[R]) {
      bf16x8 pt[HU][NSUB];
      if (more) {
        refill(k + 1);
        issue(a.k, a.kg, koff, k + 1, kz);
        __builtin_amdgcn_sched_barrier(0);
      }
      consume_k(k, kx, pt);
      if (more) {
        __builtin_amdgcn_sched_barrier(0);
        issue(a.v, a.vg, voff, k + 1, vz);
        __builtin_amdgcn_sched_barrier(0);
      }
      consume_v(k, vx, pt);
    };
    // Gather-only: the rows of step k go straight from the load registers
    // to the dense outputs (keys < L only).
    auto store_rows = [&](int k, LT (&kx)[R], LT (&vx)[R]) {
      const int64_t base = (int64_t)cur.s * a.d_seq + (int64_t)(cur.g + hl) * a.d_head + ci * LB;
  #pragma unroll
      for (int b = 0; b < BPS; ++b)
  #pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int key = k * KS + 16 * b + 4 * r4 + lq;
          if (key < cur.L) {
            *(LT*)(a.kd + base + (int64_t)key * a.d_tok) = kx[4 * b + r4];
            *(LT*)(a.vd + base + (int64_t)key * a.d_tok) = vx[4 * b + r4];
          }
        }
    };
    for (;;) {
      cb = uniform(cur.k0 * BPS);
      load_window(cur, cb, win);
      if constexpr (GATHER) {
        __builtin_amdgcn_s_waitcnt(0);
        for (int k = cur.k0; k < cur.k1; ++k) {
          refill(k);
          issue(a.k, a.kg, koff, k, krA);
          issue(a.v, a.vg, voff, k, vrA);
          store_rows(k, krA, vrA);
        }
      } else {
      load_q(cur, qc);
      __builtin_amdgcn_s_waitcnt(0);
      int k = cur.k0;
      const int k1 = cur.k1;
      issue(a.k, a.kg, koff, k, krA);
      issue(a.v, a.vg, voff, k, vrA);
      for (; k + 2 < k1; k += 2) {   // A holds step k
        step(k, true, krA, vrA, krB, vrB);
        step(k + 1, true, krB, vrB, krA, vrA);
      }
      if (k + 1 < k1) {
        step(k, true, krA, vrA, krB, vrB);
        step(k + 1, false, krB, vrB, krB, vrB);
      } else {
        step(k, false, krA, vrA, krA, vrA);
      }
      finalize();
      }
      t += cur.k1 - cur.k0;
      if (t >= t_end) break;
      const int jj = cur.gu + 1 < Hu ? cur.j : cur.j + 1;
      const int gu = cur.gu + 1 < Hu ? cur.gu + 1 : 0;
      cur = make_piece(jj, gu, 0, t_end - t);
    }
  };

  if (p.whole_units) {
    // Whole pairs: workgroup b takes pairs [b U / B, (b + 1) U / B), B =
    // min(U, workgroups); the n = min(4, nt) waves split each pair's nt
    // steps evenly, store their pieces' partials (slot 1 for the first, 0
    // for the others) and, after a workgroup barrier, merge them (one wave
    // per (unit head, query head)).  A pair of one step is one piece and
    // writes its rows itself.
    const int64_t U = (int64_t)J * Hu;
    const int B = (int)min(U, (int64_t)gridDim.x);
    if ((int)blockIdx.x >= B) return;
    const int64_t ua = U * blockIdx.x / B, ub = U * (blockIdx.x + 1) / B;
    for (int64_t u = ua; u < ub; ++u) {
      const int j = (int)(u / Hu), gu = (int)(u % Hu);
      const int64_t Pj = dec[j].w;
      const int nt = dec[j + 1].w - (int)Pj;
      const int n = min(kDecodeWaves, nt);
      const int64_t s0 = (int64_t)Hu * Pj + (int64_t)gu * nt;
      if (wave < n) run(s0 + (int64_t)wave * nt / n, s0 + (int64_t)(wave + 1) * nt / n);
      if constexpr (!GATHER) {
        if (n > 1) {
          __syncthreads();   // the pieces' partials are stored
          const int tok = dec[j].y;
          for (int x = wave; x < HU * G; x += kDecodeWaves)   // piece k: wave k's LDS
            merge_rows<D>(
                a, n, x % G, tok, gu * HU + x / G,
                [&](int k) { return *(const f32x2*)((const float*)(lds + k * WB) + HU * G * D + x * 2); },
                [&](int k) { return (const float*)(lds + k * WB) + x * D; });
          __syncthreads();   // read before the next pair's pieces reuse the slots
        }
      }
    }
    return;
  }
  if (w >= Wn) return;
  {
    const int64_t t = worker_begin(w, Ttot, Wn), t_end = worker_begin(w + 1, Ttot, Wn);
    if (t < t_end) run(t, t_end);
  }
}

// Log-sum-exp merge of the pieces of every (sequence, kv head) pair that
// spans several workers (Sec. 4.5), for launches without fused merges.  One
// wave per (pair, query head of the group); pairs one worker finished exit.
template <int D>
__global__ __launch_bounds__(256) void merge_kernel(BatchArgs a, DecodePlan p) {
  const int jj = blockIdx.x, G = a.group;
  const int hh = uniform(blockIdx.y * 4 + (threadIdx.x >> 6));   // head within the group
  const int g = blockIdx.z;
  // The counters and the pair's two list entries in one round of loads
  // (entries jj, jj + 1 <= S exist whatever J is).
  const int J = p.meta[0], Wn = p.meta[1], PJ = p.meta[2];
  const int4 e = p.dec[jj];
  const int4 e1 = p.dec[jj + 1];
  if (jj >= J || hh >= G) return;
  const int HU = p.unit_heads, Hu = a.num_kv_heads / HU;
  const int gu = g / HU, hu = g - gu * HU;
  const int nt = e1.w - e.w;
  const int64_t Ttot = (int64_t)Hu * PJ;
  const int64_t ta = (int64_t)Hu * e.w + (int64_t)gu * nt;
  const int w0 = worker_of(ta, Ttot, Wn), w1 = worker_of(ta + nt - 1, Ttot, Wn);
  if (w0 == w1) return;
  merge_pieces<D>(a, p, w0, w1 - w0 + 1, hu, hh, e.y, g);
}

template <bool GATHER>
hipError_t launch_decode_t(const BatchArgs& a, const DecodePlan& p, int head_dim, bool fp8,
                           hipStream_t st, KernelTiming* tm) {
  const dim3 grid((unsigned)((p.workers + kDecodeWaves - 1) / kDecodeWaves)), block(64 * kDecodeWaves);
  const int hu = p.unit_heads;
  if (head_dim == 128 && !fp8 && hu == 1) launch_k(decode_kernel<128, false, 1, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 128 && fp8 && hu == 2) launch_k(decode_kernel<128, true, 2, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 128 && fp8 && hu == 1) launch_k(decode_kernel<128, true, 1, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 64 && !fp8 && hu == 2) launch_k(decode_kernel<64, false, 2, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 64 && !fp8 && hu == 1) launch_k(decode_kernel<64, false, 1, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 64 && fp8 && hu == 4) launch_k(decode_kernel<64, true, 4, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 64 && fp8 && hu == 2) launch_k(decode_kernel<64, true, 2, GATHER>, grid, block, st, tm, a, p);
  else if (head_dim == 64 && fp8 && hu == 1) launch_k(decode_kernel<64, true, 1, GATHER>, grid, block, st, tm, a, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const BatchArgs& a, const DecodePlan& p, int head_dim, bool fp8,
                         hipStream_t st, bool gather, KernelTiming* tm) {
  return gather ? launch_decode_t<true>(a, p, head_dim, fp8, st, tm)
                : launch_decode_t<false>(a, p, head_dim, fp8, st, tm);
}

hipError_t launch_merge(const BatchArgs& a, const DecodePlan& p, int head_dim, hipStream_t st,
                        KernelTiming* tm) {
  const dim3 grid(a.num_seqs, (a.group + 3) / 4, a.num_kv_heads), block(256);
  if (head_dim == 128) launch_k(merge_kernel<128>, grid, block, st, tm, a, p);
  else if (head_dim == 64) launch_k(merge_kernel<64>, grid, block, st, tm, a, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa

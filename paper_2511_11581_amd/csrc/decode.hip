// Decode attention over a paged KV cache with split-KV segments
// (arxiv 2511.11581, Sec. 4.4 GQA packing and Sec. 4.5 parallel tiled
// softmax; Eq. 1-2 for what is computed).
//
// One workgroup = (kv head g, segment k, sequence s), 4 waves.  Only
// sequences whose query length is 1 are handled here.  All G = Hq/Hkv query
// heads of kv head g are packed into the columns of one 16-wide MFMA tile,
// so each K/V row of the segment is read from HBM exactly once.  The segment
// [k*seg_len, min((k+1)*seg_len, L)) is cut into 32-key tiles dealt to the 4
// waves round-robin; each wave keeps its own running max / sum / output and
// the waves are merged through LDS at the end.  A sequence that needs one
// segment writes bf16 output directly; otherwise the segment stores its
// unnormalised partials for the log-sum-exp merge kernel.
//
// Memory path per wave and tile: K and V rows are read with whole-row
// coalesced loads (16 lanes per row, 4 rows per instruction: lane l reads
// key 4r + (l & 3), bytes (l >> 2) * LB of the row, r = 0..7), the next
// tile's loads in flight while the current one is consumed.  Through the
// wave's private LDS area they are rearranged for the matrix cores:
//   K  -> natural bf16 rows, read back as MFMA A operands (key rows),
//   V  -> V^T rows (one row per d), 16-byte transposing writes,
//   S^T[16 keys x 16 heads] = K Q^T, P = online softmax (log2 domain),
//   O^T[d x heads] += V^T P^T      (v_mfma_f32_16x16x32_bf16).
// MFMA row m of key block kb holds key 16kb + (m >> 2) + 4(m & 3), so the 8
// keys of one lane's P^T / V^T operand slots are exactly the 8 keys that one
// loading lane holds (all keys of the tile congruent to l & 3 mod 4).
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kWaves = 4;
constexpr int kTile = 32;      // keys per wave iteration

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

template <int D, bool FP8>
__global__ __launch_bounds__(256, 2) void decode_kernel(BatchArgs a, DecodePlan p) {
  constexpr int EB = FP8 ? 1 : 2;          // bytes per cached element
  constexpr int LB = D * EB / 16;          // bytes one lane loads per row
  constexpr int DPL = LB / EB;             // d values one lane loads per row
  constexpr int PSH = DPL == 8 ? 3 : 2;    // log2(DPL)
  constexpr int NW = DPL / 2;              // bf16 dwords per lane per row
  constexpr int NSTEP = D / 32;            // MFMA k-steps over d
  constexpr int NDB = D / 16;              // 16-row d blocks of O^T
  constexpr int KRB = 2 * D + 32;          // LDS bytes per K row (bf16 + pad)
  constexpr int KT = kTile * KRB;          // K tile bytes
  constexpr int VT = 16 * (4 * D + 4 * (D >> PSH));  // V^T tile bytes
  constexpr int WB = KT + VT;              // LDS bytes per wave
  constexpr int RED = D + 2;               // floats per (wave, head) in the merge area
  typedef typename LoadT<LB>::T LT;
  static_assert(DPL == 8 || DPL == 4, "head_dim 64 or 128");
  static_assert(kWaves * 16 * RED * 4 <= kWaves * WB, "merge area must fit");

  __shared__ __attribute__((aligned(16))) uint8_t lds[kWaves * WB];

  const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
  const int q4 = lane >> 4, c16 = lane & 15;   // MFMA operand coordinates
  const int lq = lane & 3, lc = lane >> 2;     // loading coordinates
  int g, ks, s;
  if (p.head_major == 2) {
    // XCD-grouped: workgroups are dealt round-robin to the 8 XCDs; the j-th
    // workgroup of XCD x handles head j % Hkv of unit (j / Hkv) * 8 + x, so
    // the Hkv heads of one (sequence, segment) run together on one XCD.
    const int i = blockIdx.x, x = i & 7, j = i >> 3;
    const int u = (j / a.num_kv_heads) * 8 + x;
    if (u >= a.num_seqs * p.max_splits) return;
    g = j % a.num_kv_heads;
    s = u / p.max_splits;
    ks = u % p.max_splits;
  } else {
    g = p.head_major ? blockIdx.x : blockIdx.y;
    ks = p.head_major ? blockIdx.y : blockIdx.x;
    s = blockIdx.z;
  }

  const int t0 = a.qsl[s];
  if (a.qsl[s + 1] - t0 != 1 || t0 < 0 || t0 >= a.num_tokens) return;
  const int L = min(a.seq_lens[s], a.mb * a.block_size);
  if (L <= 0) return;
  const int nsplit = (L + p.seg_len - 1) / p.seg_len;
  if (ks >= nsplit) return;
  const int kbeg = ks * p.seg_len;
  const int kend = min(L, kbeg + p.seg_len);
  const int ntiles = (kend - kbeg + kTile - 1) / kTile;
  const int32_t* bt_row = a.bt + (int64_t)s * a.bt_row;
  const int G = a.group, bsl = a.bs_log2, bsm = a.block_size - 1;

  // Q^T as MFMA B operands: column c16 = head g*G + c16 (zero if c16 >= G),
  // k-step st covers d = 32 st + 8 q4 + j.
  bf16x8 qt[NSTEP];
  {
    const bool hv = c16 < G;
    const uint8_t* qrow = a.q + (int64_t)t0 * a.q_tok + (int64_t)(g * G + (hv ? c16 : 0)) * a.q_head;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      u32x4 w = hv ? ld16_cached(qrow + 2 * (32 * st + 8 * q4)) : u32x4{0, 0, 0, 0};
      qt[st] = __builtin_bit_cast(bf16x8, w);
    }
  }

  float m_run = kNegInf, l_run = 0.f;
  f32x4 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4{0, 0, 0, 0};
  uint8_t* kl = lds + wave * WB;
  uint8_t* vt = kl + KT;
  const uint8_t* kbase = a.k + (int64_t)g * a.kg.head + lc * LB;
  const uint8_t* vbase = a.v + (int64_t)g * a.vg.head + lc * LB;

  // This wave's tiles are wave, wave + 4, ...; it holds the physical block
  // of each of their 16-key blocks in a per-lane page cache (lane j: tile
  // number cache_base + j/2, half j%2), refilled every 32 tiles.
  const int nt = wave < ntiles ? (ntiles - wave + kWaves - 1) / kWaves : 0;
  int cache = 0, cache_base = -1000000;
  auto refill = [&](int i0) {
    const int blk16 = (kbeg + (wave + kWaves * (i0 + (lane >> 1))) * kTile) / 16 + (lane & 1);
    const int key = blk16 * 16;
    cache = key < kend ? page_of(bt_row, key, bsl, a.num_blocks) : 0;
    cache_base = i0;
  };
  // Issue the loads of the i-th tile of this wave: lane holds keys 4r + lq.
  auto issue = [&](int i, LT (&kr)[8], LT (&vr)[8]) {
    if (i - cache_base >= 32) refill(i);
    const int tb = kbeg + (wave + kWaves * i) * kTile;
    const int pg0 = __builtin_amdgcn_readlane(cache, 2 * (i - cache_base));
    int pg1 = __builtin_amdgcn_readlane(cache, 2 * (i - cache_base) + 1);
    pg1 = (tb + 16 < kend) ? pg1 : pg0;
    const int sl0 = tb & bsm, sl1 = (tb + 16) & bsm;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int kb = r >> 2;
      const int slot = (kb ? sl1 : sl0) + 4 * (r & 3) + lq;
      const int64_t pg = kb ? pg1 : pg0;
      kr[r] = ldn<LB>(kbase + pg * a.kg.blk + (int64_t)slot * a.kg.slot);
      vr[r] = ldn<LB>(vbase + pg * a.vg.blk + (int64_t)slot * a.vg.slot);
    }
  };
  // bf16 words of one loaded row chunk (DPL values of one key).
  auto to_bf16 = [&](const LT& v, uint32_t (&w)[NW]) {
    if constexpr (FP8) {
#pragma unroll
      for (int q = 0; q < LB / 4; ++q) {
        const u32x2 cv = fp8x4_to_bf16x4(dw<LB>(v, q));
        w[2 * q] = cv[0];
        w[2 * q + 1] = cv[1];
      }
    } else {
#pragma unroll
      for (int q = 0; q < NW; ++q) w[q] = dw<LB>(v, q);
    }
  };
  // Attention update with the i-th tile of this wave.
  auto consume = [&](int i, LT (&kr)[8], LT (&vr)[8]) {
    const int tb = kbeg + (wave + kWaves * i) * kTile;
    // ---- K rows -> LDS (bf16, natural layout)
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      uint32_t w[NW];
      to_bf16(kr[r], w);
      uint8_t* dst = kl + (4 * r + lq) * KRB + lc * (2 * DPL);
      if constexpr (NW == 4) *(u32x4*)dst = u32x4{w[0], w[1], w[2], w[3]};
      else *(u32x2*)dst = u32x2{w[0], w[1]};
    }
    // ---- S^T = K Q^T; MFMA row c16 of block kb is key 16kb + (c16>>2) + 4(c16&3)
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x4 acc = {0, 0, 0, 0};
      const uint8_t* kp = kl + (16 * kb + (c16 >> 2) + 4 * (c16 & 3)) * KRB + 16 * q4;
#pragma unroll
      for (int st = 0; st < NSTEP; ++st)
        acc = mfma16(*(const bf16x8*)(kp + 64 * st), qt[st], acc);
      sacc[kb] = acc;
    }
    // ---- online softmax (log2 domain); lane holds keys 16kb + q4 + 4r of head c16
    float x[2][4];
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = tb + 16 * kb + q4 + 4 * r;
        x[kb][r] = key < kend ? sacc[kb][r] : kNegInf;
        mx = fmaxf(mx, x[kb][r]);
      }
    mx = xor16_max(mx);
    mx = xor32_max(mx) * a.sl2;
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        x[kb][r] = fast_exp2(__builtin_fmaf(x[kb][r], a.sl2, -m_new));
        psum += x[kb][r];
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] *= alpha;
    u32x4 pw = {pack_bf16(x[0][0], x[0][1]), pack_bf16(x[0][2], x[0][3]),
                pack_bf16(x[1][0], x[1][1]), pack_bf16(x[1][2], x[1][3])};
    const bf16x8 pt = __builtin_bit_cast(bf16x8, pw);

    // ---- V -> V^T: this lane's 8 keys (4r + lq, r = 0..7) are the 8
    //      consecutive positions of column group lq; keys past the segment end
    //      are zeroed (their slots may hold NaN).
    uint32_t vw[8][NW];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      to_bf16(vr[r], vw[r]);
      if (tb + 4 * r + lq >= kend) {
#pragma unroll
        for (int q = 0; q < NW; ++q) vw[r][q] = 0u;
      }
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      const int wi = e >> 1;
      u32x4 col;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t lo = vw[2 * j][wi], hi = vw[2 * j + 1][wi];
        col[j] = (e & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
      }
      *(u32x4*)(vt + vt_off<PSH>(lc * DPL + e, lq)) = col;
    }
    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const u32x4 va = *(const u32x4*)(vt + vt_off<PSH>(16 * db + c16, q4));
      o[db] = mfma16(__builtin_bit_cast(bf16x8, va), pt, o[db]);
    }
  };

  // Software pipeline: the loads of tile i+1 are in flight while tile i is
  // consumed (two register sets, loop unrolled by two).  The steady-state
  // body issues unconditionally so that each wait covers only the older set;
  // sched_barrier keeps the compiler from hoisting the consumer's first
  // instructions above the new loads (which would force a full wait).
  LT krA[8], vrA[8], krB[8], vrB[8];
  int i = 0;
  if (nt > 0) issue(0, krA, vrA);
  for (; i + 2 < nt; i += 2) {
    issue(i + 1, krB, vrB);
    __builtin_amdgcn_sched_barrier(0);
    consume(i, krA, vrA);
    issue(i + 2, krA, vrA);
    __builtin_amdgcn_sched_barrier(0);
    consume(i + 1, krB, vrB);
  }
  if (i + 1 < nt) {
    issue(i + 1, krB, vrB);
    __builtin_amdgcn_sched_barrier(0);
    consume(i, krA, vrA);
    consume(i + 1, krB, vrB);
  } else if (i < nt) {
    consume(i, krA, vrA);
  }

  // ---- merge the 4 waves through LDS
  float l_tot = xor16_sum(l_run);
  l_tot = xor32_sum(l_tot);
  __syncthreads();
  float* red = (float*)lds;
  {
    float* rw = red + (wave * 16 + c16) * RED;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) rw[16 * db + 4 * q4 + i] = o[db][i];
    if (q4 == 0) {
      rw[D] = m_run;
      rw[D + 1] = l_tot;
    }
  }
  __syncthreads();
  const int hq = a.num_q_heads;
  for (int idx = threadIdx.x; idx < G * D; idx += 256) {
    const int hh = idx / D, dd = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red[(w * 16 + hh) * RED + D]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float* rw = red + (w * 16 + hh) * RED;
      const float sc = fast_exp2(rw[D] - M);
      num += sc * rw[dd];
      den += sc * rw[D + 1];
    }
    const int h = g * G + hh;
    if (nsplit == 1) {
      __bf16 r = (__bf16)(num / den * a.v_scale);
      *(__bf16*)(a.out + (int64_t)t0 * a.o_tok + (int64_t)h * a.o_head + 2 * dd) = r;
    } else {
      const int64_t row = ((int64_t)s * p.max_splits + ks) * hq + h;
      p.part_o[row * D + dd] = num;
      if (dd == 0) {
        p.part_ml[row * 2] = M;
        p.part_ml[row * 2 + 1] = den;
      }
    }
  }
}

// Log-sum-exp merge of the segment partials of one (sequence, query head):
// M = max_k m_k, out = sum_k 2^(m_k - M) acc_k / sum_k 2^(m_k - M) l_k.
// One thread per output element d; m_k and l_k are uniform per workgroup.
template <int D>
__global__ __launch_bounds__(D) void merge_kernel(BatchArgs a, DecodePlan p) {
  const int h = blockIdx.x, s = blockIdx.y;
  const int t0 = a.qsl[s];
  if (a.qsl[s + 1] - t0 != 1 || t0 < 0 || t0 >= a.num_tokens) return;
  const int L = min(a.seq_lens[s], a.mb * a.block_size);
  if (L <= 0) return;
  const int nsplit = min((L + p.seg_len - 1) / p.seg_len, p.max_splits);
  if (nsplit <= 1) return;
  const int hq = a.num_q_heads, dd = threadIdx.x;
  const int64_t row0 = (int64_t)s * p.max_splits * hq + h;
  float M = kNegInf;
  for (int k = 0; k < nsplit; ++k) M = fmaxf(M, p.part_ml[(row0 + (int64_t)k * hq) * 2]);
  float num = 0.f, den = 0.f;
  for (int k = 0; k < nsplit; ++k) {
    const int64_t row = row0 + (int64_t)k * hq;
    const float sc = fast_exp2(p.part_ml[row * 2] - M);
    num += sc * p.part_o[row * D + dd];
    den += sc * p.part_ml[row * 2 + 1];
  }
  __bf16 r = (__bf16)(num / den * a.v_scale);
  *(__bf16*)(a.out + (int64_t)t0 * a.o_tok + (int64_t)h * a.o_head + 2 * dd) = r;
}

}  // namespace

hipError_t launch_decode(const BatchArgs& a, const DecodePlan& p, int head_dim, bool fp8,
                         hipStream_t st) {
  // kv head fastest: the workgroups reading the same cache blocks run together
  dim3 grid(p.head_major ? a.num_kv_heads : p.max_splits,
            p.head_major ? p.max_splits : a.num_kv_heads, a.num_seqs), block(256);
  if (p.head_major == 2) {
    const int64_t units = (int64_t)a.num_seqs * p.max_splits;
    grid = dim3((unsigned)(((units + 7) / 8) * 8 * a.num_kv_heads), 1, 1);
  }
  if (head_dim == 128) {
    if (fp8) decode_kernel<128, true><<<grid, block, 0, st>>>(a, p);
    else decode_kernel<128, false><<<grid, block, 0, st>>>(a, p);
  } else if (head_dim == 64) {
    if (fp8) decode_kernel<64, true><<<grid, block, 0, st>>>(a, p);
    else decode_kernel<64, false><<<grid, block, 0, st>>>(a, p);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_merge(const BatchArgs& a, const DecodePlan& p, int head_dim, hipStream_t st) {
  dim3 grid(a.num_q_heads, a.num_seqs);
  if (head_dim == 128) merge_kernel<128><<<grid, dim3(128), 0, st>>>(a, p);
  else if (head_dim == 64) merge_kernel<64><<<grid, dim3(64), 0, st>>>(a, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa

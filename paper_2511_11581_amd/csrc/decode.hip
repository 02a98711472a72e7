// Decode attention over a paged KV cache with split-KV segments
// (arxiv 2511.11581, Sec. 4.4 GQA packing and Sec. 4.5 parallel tiled
// softmax; Eq. 1-2 for what is computed).
//
// One workgroup = (segment k, sequence s, kv head g), 4 waves.  Only
// sequences whose query length is 1 are handled here.  All G = Hq/Hkv query
// heads of kv head g are packed into the columns of one 16-wide MFMA tile,
// so each K/V row of the segment is read from HBM exactly once.  The segment
// [k*seg_len, min((k+1)*seg_len, L)) is cut into 32-key tiles dealt to the 4
// waves round-robin; each wave keeps its own running max / sum / output and
// the waves are merged through LDS at the end.  A sequence that needs one
// segment writes bf16 output directly; otherwise the segment stores its
// unnormalised partials for the log-sum-exp merge kernel.
//
// Per tile and wave:
//   S^T[16 keys x 16 heads] = K Q^T  (v_mfma_f32_16x16x32_bf16, 2 key blocks)
//   online softmax in the log2 domain (one lane = one head column)
//   O^T[d x heads] += V^T P^T         (V transposed through LDS)
// K is loaded straight into MFMA A-operand registers with 16-byte loads:
// lane (q4 = l/16, c16 = l%16) reads key c16 of a 16-key block, 16 bytes at
// byte offset 64*i + 16*q4 of the row.  The d-permutation this implies is
// applied identically to Q, so the dot products are unchanged.
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kWaves = 4;
constexpr int kTile = 32;      // keys per wave iteration

// Keys of a 32-key tile sit in a V^T row so that the 8 keys feeding one
// lane's MFMA A-operand slots (keys 16j + 4*q4 + r, j = 0..1, r = 0..3) are
// contiguous: key kk is at position 8*((kk >> 2) & 3) + 4*(kk >> 4) + (kk & 3).
//
// Byte offset of 16-byte column group cg (0..3) of V^T row r in a wave's LDS
// area.  Rows are 64 bytes, 64 bytes of padding follow every 2^PS rows and the
// column group is XOR-swizzled with bits 2..3 of the row.  With PS = log2 of
// the d rows one lane writes (8 for bf16, 16 for fp8) both the transposing
// 8-byte writes (16-lane groups) and the 16-byte operand reads (32-lane
// groups) hit distinct LDS banks.
template <int PS>
__device__ __forceinline__ int vt_off(int r, int cg) {
  return 16 * (4 * r + 4 * (r >> PS) + (cg ^ ((r >> 2) & 3)));
}
template <int D, int PS>
constexpr int vt_bytes() { return 16 * (4 * D + 4 * (D >> PS)); }

template <int D, bool FP8>
__global__ __launch_bounds__(256, 2) void decode_kernel(BatchArgs a, DecodePlan p) {
  constexpr int EB = FP8 ? 1 : 2;          // bytes per cached element
  constexpr int NSTEP = D / 32;            // MFMA k-steps over d
  constexpr int NKLD = D * EB / 64;        // 16-byte K loads per lane per key block
  constexpr int NDB = D / 16;              // 16-row d blocks of O^T
  constexpr int CH = D * EB / 16;          // 16-byte chunks per cached row
  constexpr int TASKS = 8 * CH;            // (4-key group, chunk) pairs per tile
  constexpr int NT = (TASKS + 63) / 64;    // tasks per lane
  constexpr int DPC = 16 / EB;             // d values per chunk
  constexpr int RED = D + 2;               // floats per (wave, head) in the merge area
  constexpr int PS = FP8 ? 4 : 3;          // log2(DPC)
  constexpr int VT = vt_bytes<D, PS>();    // LDS bytes per wave
  static_assert(kWaves * 16 * RED * 4 <= kWaves * VT, "merge area must fit");

  __shared__ __attribute__((aligned(16))) uint8_t lds[kWaves * VT];

  const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
  const int q4 = lane >> 4, c16 = lane & 15;
  const int g = blockIdx.x, ks = blockIdx.y, s = blockIdx.z;

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

  // Q^T as MFMA B operands: column c16 = head g*G + c16 (zero if c16 >= G).
  bf16x8 qt[NSTEP];
  {
    const bool hv = c16 < G;
    const uint8_t* qrow = a.q + (int64_t)t0 * a.q_tok + (int64_t)(g * G + (hv ? c16 : 0)) * a.q_head;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      const int dbase = FP8 ? (64 * (st >> 1) + 16 * q4 + 8 * (st & 1)) : (32 * st + 8 * q4);
      u32x4 w = hv ? ld16_cached(qrow + dbase * 2) : u32x4{0, 0, 0, 0};
      qt[st] = __builtin_bit_cast(bf16x8, w);
    }
  }

  float m_run = kNegInf, l_run = 0.f;
  f32x4 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4{0, 0, 0, 0};
  uint8_t* vt = lds + wave * VT;
  const uint8_t* kbase = a.k + (int64_t)g * a.kg.head;
  const uint8_t* vbase = a.v + (int64_t)g * a.vg.head;

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
  // Issue the loads of the i-th tile of this wave into (kr, vr).
  auto issue = [&](int i, u32x4 (&kr)[2][NKLD], u32x4 (&vr)[NT][4]) {
    if (i - cache_base >= 32) refill(i);
    const int tb = kbeg + (wave + kWaves * i) * kTile;
    const int pg0 = __builtin_amdgcn_readlane(cache, 2 * (i - cache_base));
    int pg1 = __builtin_amdgcn_readlane(cache, 2 * (i - cache_base) + 1);
    pg1 = (tb + 16 < kend) ? pg1 : pg0;
    const int sl0 = tb & bsm, sl1 = (tb + 16) & bsm;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const uint8_t* rp = kbase + (int64_t)(kb ? pg1 : pg0) * a.kg.blk +
                          (int64_t)((kb ? sl1 : sl0) + c16) * a.kg.slot + 16 * q4;
#pragma unroll
      for (int j = 0; j < NKLD; ++j) kr[kb][j] = ld16(rp + 64 * j);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int task = min(lane + 64 * t, TASKS - 1);
      const int m = task & 7, c = task >> 3;
      const int kb = m >> 2;
      const uint8_t* rp = vbase + (int64_t)(kb ? pg1 : pg0) * a.vg.blk +
                          (int64_t)((kb ? sl1 : sl0) + 4 * (m & 3)) * a.vg.slot + 16 * c;
#pragma unroll
      for (int r = 0; r < 4; ++r) vr[t][r] = ld16(rp + (int64_t)r * a.vg.slot);
    }
  };
  // Attention update with the i-th tile of this wave held in (kr, vr).
  auto consume = [&](int i, u32x4 (&kr)[2][NKLD], u32x4 (&vr)[NT][4]) {
    const int tb = kbeg + (wave + kWaves * i) * kTile;
    // ---- S^T = K Q^T
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x4 acc = {0, 0, 0, 0};
      if constexpr (FP8) {
#pragma unroll
        for (int j = 0; j < NKLD; ++j) {
          bf16x8 lo, hi;
          fp8x16_to_bf16(kr[kb][j], lo, hi);
          acc = mfma16(lo, qt[2 * j], acc);
          acc = mfma16(hi, qt[2 * j + 1], acc);
        }
      } else {
#pragma unroll
        for (int st = 0; st < NSTEP; ++st)
          acc = mfma16(__builtin_bit_cast(bf16x8, kr[kb][st]), qt[st], acc);
      }
      sacc[kb] = acc;
    }
    // ---- online softmax (log2 domain); lane holds keys 16kb + 4q4 + r of head c16
    float x[2][4];
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = tb + 16 * kb + 4 * q4 + r;
        x[kb][r] = key < kend ? sacc[kb][r] * a.sl2 : kNegInf;
        mx = fmaxf(mx, x[kb][r]);
      }
    mx = xor16_max(mx);
    mx = xor32_max(mx);
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        x[kb][r] = fast_exp2(x[kb][r] - m_new);
        psum += x[kb][r];
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] *= alpha;
    u32x4 pw = {pack_bf16(x[0][0], x[0][1]), pack_bf16(x[0][2], x[0][3]),
                pack_bf16(x[1][0], x[1][1]), pack_bf16(x[1][2], x[1][3])};
    const bf16x8 pt = __builtin_bit_cast(bf16x8, pw);

    // ---- V -> V^T in this wave's LDS area (bf16), 8 bytes = 4 keys per d row;
    //      rows of keys past the segment end are zeroed (their slots may hold NaN).
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int task = lane + 64 * t;
      if (task < TASKS) {
        const int m = task & 7, c = task >> 3;
        // keys 4m..4m+3 occupy 8 bytes (half m>>2 of column group m&3) of row DPC*c + e
        const int cg = m & 3, half8 = 8 * (m >> 2);
        u32x4 v4[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          v4[r] = (tb + 4 * m + r < kend) ? vr[t][r] : u32x4{0, 0, 0, 0};
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
            *(u32x2*)(vt + vt_off<PS>(DPC * c + e, cg) + half8) = u32x2{lo, hi};
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
            *(u32x2*)(vt + vt_off<PS>(DPC * c + e, cg) + half8) = u32x2{lo, hi};
          }
        }
      }
    }
    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const u32x4 va = *(const u32x4*)(vt + vt_off<PS>(16 * db + c16, q4));
      o[db] = mfma16(__builtin_bit_cast(bf16x8, va), pt, o[db]);
    }
  };

  // Software pipeline: the loads of tile i+1 are in flight while tile i is
  // consumed (two register sets, loop unrolled by two).  The steady-state
  // body issues unconditionally so that each wait covers only the older set.
  u32x4 krA[2][NKLD], vrA[NT][4], krB[2][NKLD], vrB[NT][4];
  int i = 0;
  if (nt > 0) issue(0, krA, vrA);
  // sched_barrier keeps the compiler from hoisting the consumer's first
  // instructions above the new loads (which would force a full wait).
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
  dim3 grid(a.num_kv_heads, p.max_splits, a.num_seqs), block(256);
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

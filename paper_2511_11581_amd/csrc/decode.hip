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
constexpr int kVRow = 80;      // LDS bytes per d-row of the V^T tile (64 + 16 pad)

// Position of key kk (0..31 in a tile) inside the V^T row: keys are stored so
// that the 8 keys feeding one lane's MFMA A-operand slots are contiguous.
__device__ __forceinline__ int vt_pos(int kk) {
  return (((kk >> 2) & 3) << 3) | ((kk >> 4) << 2) | (kk & 3);
}

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
  static_assert(kWaves * 16 * RED * 4 <= kWaves * D * kVRow, "merge area must fit");

  __shared__ __attribute__((aligned(16))) uint8_t lds[kWaves * D * kVRow];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q4 = lane >> 4, c16 = lane & 15;
  const int ks = blockIdx.x, s = blockIdx.y, g = blockIdx.z;

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
  const int G = a.group, bs = a.block_size;

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
  uint8_t* vt = lds + wave * D * kVRow;
  const uint8_t* kbase = a.k + (int64_t)g * a.kg.head;
  const uint8_t* vbase = a.v + (int64_t)g * a.vg.head;

  for (int tile = wave; tile < ntiles; tile += kWaves) {
    const int tb = kbeg + tile * kTile;
    const int pg0 = page_of(bt_row, tb, bs, a.num_blocks);
    const int pg1 = (tb + 16 < kend) ? page_of(bt_row, tb + 16, bs, a.num_blocks) : pg0;
    const int sl0 = tb % bs, sl1 = (tb + 16) % bs;

    // ---- K rows -> A operands
    u32x4 kr[2][NKLD];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int key = tb + 16 * kb + c16;
      const uint8_t* rp = kbase + (int64_t)(kb ? pg1 : pg0) * a.kg.blk +
                          (int64_t)((kb ? sl1 : sl0) + c16) * a.kg.slot + 16 * q4;
#pragma unroll
      for (int i = 0; i < NKLD; ++i)
        kr[kb][i] = key < kend ? ld16(rp + 64 * i) : u32x4{0, 0, 0, 0};
    }
    // ---- V rows (natural layout), 4 consecutive keys x one chunk per task
    u32x4 vr[NT][4];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int task = lane + 64 * t;
      const int c = task % CH, m = task / CH;
      const int kb = m >> 2;
      const uint8_t* rp = vbase + (int64_t)(kb ? pg1 : pg0) * a.vg.blk +
                          (int64_t)((kb ? sl1 : sl0) + 4 * (m & 3)) * a.vg.slot + 16 * c;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool ok = task < TASKS && tb + 4 * m + r < kend;
        vr[t][r] = ok ? ld16(rp + (int64_t)r * a.vg.slot) : u32x4{0, 0, 0, 0};
      }
    }

    // ---- S^T = K Q^T
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x4 acc = {0, 0, 0, 0};
      if constexpr (FP8) {
#pragma unroll
        for (int i = 0; i < NKLD; ++i) {
          bf16x8 lo, hi;
          fp8x16_to_bf16(kr[kb][i], lo, hi);
          acc = mfma16(lo, qt[2 * i], acc);
          acc = mfma16(hi, qt[2 * i + 1], acc);
        }
      } else {
#pragma unroll
        for (int st = 0; st < NSTEP; ++st)
          acc = mfma16(__builtin_bit_cast(bf16x8, kr[kb][st]), qt[st], acc);
      }
      sacc[kb] = acc;
    }

    // ---- online softmax (log2 domain); lane holds keys 16kb + 4q4 + i of head c16
    float x[2][4];
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = tb + 16 * kb + 4 * q4 + i;
        x[kb][i] = key < kend ? sacc[kb][i] * a.sl2 : kNegInf;
        mx = fmaxf(mx, x[kb][i]);
      }
    mx = xor16_max(mx);
    mx = xor32_max(mx);
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[kb][i] = fast_exp2(x[kb][i] - m_new);
        psum += x[kb][i];
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] *= alpha;
    u32x4 pw = {pack_bf16(x[0][0], x[0][1]), pack_bf16(x[0][2], x[0][3]),
                pack_bf16(x[1][0], x[1][1]), pack_bf16(x[1][2], x[1][3])};
    const bf16x8 pt = __builtin_bit_cast(bf16x8, pw);

    // ---- V -> V^T in this wave's LDS area (bf16), 8 bytes = 4 keys per d row
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int task = lane + 64 * t;
      if (task < TASKS) {
        const int c = task % CH, m = task / CH;
        const int pos = vt_pos(4 * m);
        uint8_t* wp = vt + (c * DPC) * kVRow + 2 * pos;
        if constexpr (FP8) {
          // 16 fp8 values per key -> 8 dwords of bf16 pairs per key
          uint32_t w[4][8];
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              u32x2 cv = fp8x4_to_bf16x4(vr[t][r][q]);
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
            *(u32x2*)(wp + e * kVRow) = u32x2{lo, hi};
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int dw = e >> 1;
            uint32_t lo, hi;
            if (e & 1) {
              lo = (vr[t][0][dw] >> 16) | (vr[t][1][dw] & 0xFFFF0000u);
              hi = (vr[t][2][dw] >> 16) | (vr[t][3][dw] & 0xFFFF0000u);
            } else {
              lo = (vr[t][0][dw] & 0xFFFFu) | (vr[t][1][dw] << 16);
              hi = (vr[t][2][dw] & 0xFFFFu) | (vr[t][3][dw] << 16);
            }
            *(u32x2*)(wp + e * kVRow) = u32x2{lo, hi};
          }
        }
      }
    }
    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const u32x4 va = *(const u32x4*)(vt + (16 * db + c16) * kVRow + 16 * q4);
      o[db] = mfma16(__builtin_bit_cast(bf16x8, va), pt, o[db]);
    }
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

// Log-sum-exp merge of the segment partials of one (sequence, kv head):
// M = max_k m_k, out = sum_k 2^(m_k - M) acc_k / sum_k 2^(m_k - M) l_k.
template <int D>
__global__ __launch_bounds__(256) void merge_kernel(BatchArgs a, DecodePlan p) {
  const int s = blockIdx.x, g = blockIdx.y;
  const int t0 = a.qsl[s];
  if (a.qsl[s + 1] - t0 != 1 || t0 < 0 || t0 >= a.num_tokens) return;
  const int L = min(a.seq_lens[s], a.mb * a.block_size);
  if (L <= 0) return;
  const int nsplit = min((L + p.seg_len - 1) / p.seg_len, p.max_splits);
  if (nsplit <= 1) return;
  const int G = a.group, hq = a.num_q_heads;
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int hh = idx / D, dd = idx % D;
    const int h = g * G + hh;
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
}

}  // namespace

hipError_t launch_decode(const BatchArgs& a, const DecodePlan& p, int head_dim, bool fp8,
                         hipStream_t st) {
  dim3 grid(p.max_splits, a.num_seqs, a.num_kv_heads), block(256);
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
  dim3 grid(a.num_seqs, a.num_kv_heads), block(256);
  if (head_dim == 128) merge_kernel<128><<<grid, block, 0, st>>>(a, p);
  else if (head_dim == 64) merge_kernel<64><<<grid, block, 0, st>>>(a, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa

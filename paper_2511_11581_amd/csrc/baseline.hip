// The paper's baseline decomposition, kept as the first rung of the
// optimisation-ladder ablation (arxiv 2511.11581, Sec. 4 and App. A; the
// ladder of Sec. 7): one workgroup (one wave) per (query token, query head).
// It finds its sequence by binary search over query_start_loc, walks the
// sequence's pages one tile (= one page) at a time and keeps the online
// softmax of Eq. 2 in registers.  No GQA packing (every query head re-reads
// its kv head's K/V), no split of long rows, no matrix cores: the reference
// point of the ablation, not a fast path.
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

template <bool FP8>
__device__ __forceinline__ float kv_elem(const uint8_t* row, int i) {
  if constexpr (FP8) return __builtin_amdgcn_cvt_f32_fp8((int)row[i], 0);
  else return __uint_as_float((uint32_t)((const uint16_t*)row)[i] << 16);
}

template <int D, bool FP8>
__global__ __launch_bounds__(64) void baseline_kernel(BatchArgs a) {
  constexpr int PER = D / 64;   // d values per lane
  const int t = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  if (t >= a.qsl[a.num_seqs]) return;
  int lo = 0, hi = a.num_seqs - 1;   // the last sequence s with qsl[s] <= t
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.qsl[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  const int s = lo, t0 = a.qsl[s], qlen = a.qsl[s + 1] - t0;
  const int L = min(a.seq_lens[s], a.mb * a.block_size);
  const int ctx = L - qlen;
  if (ctx < 0 || qlen < 1) return;
  const int nkeys = ctx + (t - t0) + 1;   // causal: keys 0 .. ctx + j
  const int g = h / a.group;
  float q[PER], o[PER];
  const uint16_t* qrow = (const uint16_t*)(a.q + (int64_t)t * a.q_tok + (int64_t)h * a.q_head);
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    q[e] = __uint_as_float((uint32_t)qrow[lane * PER + e] << 16) * a.sl2;   // log2 units
    o[e] = 0.f;
  }
  float m = -__builtin_inff(), l = 0.f;
  const int32_t* btr = a.bt + (int64_t)s * a.bt_row;
  for (int p0 = 0; p0 < nkeys; p0 += a.block_size) {   // one page per tile
    const int blk = page_of(btr, p0, a.bdiv, a.num_blocks);
    const int nk = min(a.block_size, nkeys - p0);
    const uint8_t* kb = a.k + (int64_t)blk * a.kg.blk + (int64_t)g * a.kg.head;
    const uint8_t* vb = a.v + (int64_t)blk * a.vg.blk + (int64_t)g * a.vg.head;
    for (int i = 0; i < nk; ++i) {
      const uint8_t* kr = kb + (int64_t)i * a.kg.slot;
      const uint8_t* vr = vb + (int64_t)i * a.vg.slot;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < PER; ++e) dot += q[e] * kv_elem<FP8>(kr, lane * PER + e);
      dot = wave_sum(dot);
      const float mn = fmaxf(m, dot);
      const float alpha = fast_exp2(m - mn), p = fast_exp2(dot - mn);
      l = l * alpha + p;
#pragma unroll
      for (int e = 0; e < PER; ++e) o[e] = o[e] * alpha + p * kv_elem<FP8>(vr, lane * PER + e);
      m = mn;
    }
  }
  const float inv = a.v_scale / l;
  uint16_t* orow = (uint16_t*)(a.out + (int64_t)t * a.o_tok + (int64_t)h * a.o_head);
#pragma unroll
  for (int e = 0; e < PER; ++e) orow[lane * PER + e] = (uint16_t)(pack_bf16(o[e] * inv, 0.f) & 0xffffu);
}

}  // namespace

hipError_t launch_baseline(const BatchArgs& a, int head_dim, bool fp8, hipStream_t st) {
  if (a.num_tokens <= 0 || a.num_seqs <= 0) return hipSuccess;
  dim3 grid((unsigned)a.num_tokens, (unsigned)a.num_q_heads), block(64);
  if (head_dim == 128 && !fp8) baseline_kernel<128, false><<<grid, block, 0, st>>>(a);
  else if (head_dim == 128) baseline_kernel<128, true><<<grid, block, 0, st>>>(a);
  else if (head_dim == 64 && !fp8) baseline_kernel<64, false><<<grid, block, 0, st>>>(a);
  else if (head_dim == 64) baseline_kernel<64, true><<<grid, block, 0, st>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa

// Per-batch work lists, built on the device by one workgroup so that the
// host never reads the batch metadata (arxiv 2511.11581, Sec. 6.1: count the
// decodes and accumulate the Q-blocks of the batch; Sec. 4.4 Q-blocks;
// Sec. 4.5 split of decode work).
//
// Decode list: the sequences with one query token, in batch order, with the
// prefix P(j) of their step counts ceil(L_j / KS) and the number of decode
// workers given work (every worker streams at least min_steps steps when the
// batch has that many).
//
// Q-block list: prefix sums of ceil(q_i / BLOCK_Q) over sequences with two or
// more query tokens, and the list of (sequence, Q-block) items ordered by
// decreasing number of key tiles (longest first), which evens out the
// causal triangle's very unequal work items across the CUs.
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPlanSortCap = 8192;   // larger Q-block lists keep the natural order
constexpr int kPlanBuckets = 2048;   // key-tile counts are clamped to this

// Number of Q-blocks of sequence i (0 for single-token or empty rows, and
// for rows whose metadata is out of range).
__device__ __forceinline__ int nqb_of(const BatchArgs& a, int i, int bq) {
  const int t0 = a.qsl[i], q = a.qsl[i + 1] - t0;
  if (q < 2 || t0 < 0 || t0 + q > a.num_tokens) return 0;
  const int L = min(a.seq_lens[i], a.mb * a.block_size);
  if (L < q) return 0;
  return (q + bq - 1) / bq;
}

// Block-wide exclusive scan of one value per thread (kPlanThreads threads).
__device__ int block_exclusive_scan(int v, int& total) {
  __shared__ int wsum[kPlanThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  if (w == 0) {
    int t = lane < kPlanThreads / 64 ? wsum[lane] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(t, o);
      if (lane >= o) t += y;
    }
    if (lane < kPlanThreads / 64) wsum[lane] = t;
  }
  __syncthreads();
  const int before = (w > 0 ? wsum[w - 1] : 0) + x - v;
  total = wsum[kPlanThreads / 64 - 1];
  __syncthreads();
  return before;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(BatchArgs a, DecodePlan dp, PrefillPlan pp,
                                                            int with_prefill) {
  __shared__ int hist[kPlanBuckets];
  __shared__ int keys[kPlanSortCap];
  const int tid = threadIdx.x, S = a.num_seqs;
  const int cap = a.mb * a.block_size;

  // ---- decode list
  {
    int njs = 0, nsteps = 0;
    for (int base = 0; base < S; base += kPlanThreads) {
      const int i = base + tid;
      int is_dec = 0, nt = 0, t0 = 0, L = 0;
      if (i < S) {
        t0 = a.qsl[i];
        L = min(a.seq_lens[i], cap);
        if (a.qsl[i + 1] - t0 == 1 && t0 >= 0 && t0 < a.num_tokens && L >= 1) {
          is_dec = 1;
          nt = (L + dp.step_keys - 1) / dp.step_keys;
        }
      }
      int tot_j, tot_s;
      const int ej = block_exclusive_scan(is_dec, tot_j);
      const int es = block_exclusive_scan(nt, tot_s);
      if (is_dec) dp.dec[njs + ej] = make_int4(i, t0, L, nsteps + es);
      njs += tot_j;
      nsteps += tot_s;
    }
    if (tid == 0) {
      dp.dec[njs] = make_int4(0, 0, 0, nsteps);
      dp.meta[0] = njs;
      dp.meta[1] = active_workers((int64_t)a.num_kv_heads * nsteps, dp.min_steps, dp.workers);
    }
  }
  if (!with_prefill) return;

  // ---- Q-block list: 1. prefix sums of Q-blocks per sequence
  const int bq = pp.block_q;
  int carry = 0;
  for (int base = 0; base < S; base += kPlanThreads) {
    const int i = base + tid;
    const int n = i < S ? nqb_of(a, i, bq) : 0;
    int tot;
    const int ex = block_exclusive_scan(n, tot);
    if (i < S) pp.seq_start[i] = carry + ex;
    carry += tot;
  }
  const int N = min(carry, pp.work_items);
  if (tid == 0) {
    pp.seq_start[S] = carry;
    pp.count[0] = N;
  }
  __threadfence();
  __syncthreads();
  // item -> (sequence, Q-block index): binary search in seq_start (device-
  // coherent loads: the array was just written by other threads)
  auto start_of = [&](int i) {
    return __hip_atomic_load(pp.seq_start + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  auto locate = [&](int idx, int& seq, int& qb) {
    int lo = 0, hi = S - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (start_of(mid) <= idx) lo = mid; else hi = mid - 1;
    }
    seq = lo;
    qb = idx - start_of(lo);
  };
  if (N > kPlanSortCap) {
    for (int idx = tid; idx < N; idx += kPlanThreads) {
      int seq, qb;
      locate(idx, seq, qb);
      pp.list_seq[idx] = seq;
      pp.list_qb[idx] = qb;
    }
    return;
  }
  // 2. counting sort by decreasing key-tile count
  for (int k = tid; k < kPlanBuckets; k += kPlanThreads) hist[k] = 0;
  __syncthreads();
  for (int idx = tid; idx < N; idx += kPlanThreads) {
    int seq, qb;
    locate(idx, seq, qb);
    const int t0 = a.qsl[seq], q = a.qsl[seq + 1] - t0;
    const int L = min(a.seq_lens[seq], cap);
    const int kv = (L - q) + min((qb + 1) * bq, q);
    const int key = min((kv + kPrefillTileKeys - 1) / kPrefillTileKeys, kPlanBuckets - 1);
    keys[idx] = key;
    atomicAdd(&hist[key], 1);
  }
  __syncthreads();
  // exclusive scan of the histogram in decreasing key order: bucket offsets
  int hcarry = 0;
  for (int base = 0; base < kPlanBuckets; base += kPlanThreads) {
    const int b = kPlanBuckets - 1 - (base + tid);
    const int n = hist[b];
    int tot;
    const int ex = block_exclusive_scan(n, tot);
    hist[b] = hcarry + ex;  // bucket b is read and written by this thread only
    hcarry += tot;
  }
  __syncthreads();
  for (int idx = tid; idx < N; idx += kPlanThreads) {
    int seq, qb;
    locate(idx, seq, qb);
    const int pos = atomicAdd(&hist[keys[idx]], 1);
    pp.list_seq[pos] = seq;
    pp.list_qb[pos] = qb;
  }
}

}  // namespace

hipError_t launch_plan(const BatchArgs& a, const DecodePlan& dp, const PrefillPlan& pp,
                       bool with_prefill, hipStream_t st) {
  if (a.num_seqs <= 0) return hipSuccess;
  plan_kernel<<<dim3(1), dim3(kPlanThreads), 0, st>>>(a, dp, pp, with_prefill ? 1 : 0);
  return hipGetLastError();
}

}  // namespace pa

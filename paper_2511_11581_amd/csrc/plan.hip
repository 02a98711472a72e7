// Per-batch work lists, built on the device by one workgroup so that the
// host never reads the batch metadata (arxiv 2511.11581, Sec. 6.1: count the
// decodes and accumulate the Q-blocks of the batch; Sec. 4.4 Q-blocks;
// Sec. 4.5 split of decode work).
//
// Decode list: the sequences with one query token, in batch order, with the
// prefix P(j) of their step counts ceil(L_j / KS) and the number of decode
// workers given work (every worker streams at least min_steps steps of its
// units when the batch has that many).
//
// Q-block list: prefix sums of ceil(q_i / BLOCK_Q) over sequences with two or
// more query tokens, and the list of (sequence, Q-block) items ordered by
// decreasing number of key tiles (longest first), which evens out the
// causal triangle's very unequal work items across the CUs.
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

// 256 threads: the work is a few passes over the sequences and Q-blocks,
// and each block-wide scan costs fewer barrier rounds than with 1024
// (measured 6.7 against 7.6 us per call on a 4-sequence prefill batch).
constexpr int kPlanThreads = 256;
constexpr int kPlanSortCap = 8192;   // larger Q-block lists keep the natural order
// Key-tile counts are clamped to the last bucket: Q-blocks of more than
// 32K keys all sort first, in batch order among themselves.
constexpr int kPlanBuckets = 512;


// Exclusive scan of NV values per thread with the block totals: one wave
// (NT = 64) scans with lane shuffles alone, larger blocks with block_scan.
template <int NV, int NT>
__device__ __forceinline__ void plan_scan(const int (&v)[NV], int (&ex)[NV], int (&tot)[NV]) {
  if constexpr (NT == 64) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int x = v[i];
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
      }
      ex[i] = x - v[i];
      tot[i] = __shfl(x, 63);
    }
  } else {
    block_scan<NV, NT>(v, ex, tot);
  }
}

template <int NT>
__global__ __launch_bounds__(NT) void plan_kernel(BatchArgs a, DecodePlan dp, PrefillPlan pp,
                                                            int with_prefill) {
  __shared__ int hist[kPlanBuckets];
  __shared__ int keys[kPlanSortCap];
  __shared__ int start_l[kPlanSortCap + 1];   // seq_start when S < kPlanSortCap
  const int tid = threadIdx.x, S = a.num_seqs;
  const int cap = a.mb * a.block_size;
  const int bq = pp.block_q;
  const bool local = S < kPlanSortCap;

  // ---- one pass over the sequences: decode flag, decode steps, Q-blocks
  int njs = 0, nsteps = 0, nqb = 0;
  for (int base = 0; base < S; base += NT) {
    const int i = base + tid;
    int v[3] = {0, 0, 0};
    int t0 = 0, L = 0;
    if (i < S) {
      t0 = a.qsl[i];
      const int q = a.qsl[i + 1] - t0;
      L = min(a.seq_lens[i], cap);
      if (q == 1 && pp.qmin == 2 && t0 >= 0 && t0 < a.num_tokens && L >= 1) {
        v[0] = 1;
        v[1] = (L + dp.step_keys - 1) / dp.step_keys;
      } else if (with_prefill && q >= pp.qmin && t0 >= 0 && t0 + q <= a.num_tokens && L >= q) {
        v[2] = (q + bq - 1) / bq;
      }
    }
    int ex[3], tot[3];
    plan_scan<3, NT>(v, ex, tot);
    if (v[0]) dp.dec[njs + ex[0]] = make_int4(i, t0, L, nsteps + ex[1]);
    if (with_prefill && i < S) {
      pp.seq_start[i] = nqb + ex[2];
      if (local) start_l[i] = nqb + ex[2];
    }
    njs += tot[0];
    nsteps += tot[1];
    nqb += tot[2];
  }
  if (tid == 0) {
    dp.dec[njs] = make_int4(0, 0, 0, nsteps);
    dp.meta[0] = njs;
    dp.meta[1] = active_workers((int64_t)(a.num_kv_heads / dp.unit_heads) * nsteps, dp.min_steps, dp.workers);
    dp.meta[2] = nsteps;
    if (with_prefill) {
      pp.seq_start[S] = nqb;
      pp.count[0] = min(nqb, pp.work_items);
    }
  }
  if (!with_prefill || nqb == 0) return;

  // ---- Q-block list: item -> (sequence, Q-block index) by binary search
  //      in the prefix sums (from LDS, or device-coherent global loads)
  if (local && tid == 0) start_l[S] = nqb;
  const int N = min(nqb, pp.work_items);
  if (!local) __threadfence();
  __syncthreads();
  auto start_of = [&](int i) {
    return local ? start_l[i]
                 : __hip_atomic_load(pp.seq_start + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
  // The record of a Q-block: its sequence, its first token, its row count
  // and the keys before its first token.
  auto place = [&](int at, int seq, int qb) {
    const int t0 = a.qsl[seq], q = a.qsl[seq + 1] - t0;
    const int L = min(a.seq_lens[seq], cap);
    pp.list_seq[at] = seq;
    pp.list_qb[at] = qb;
    pp.rec[at] = make_int4(seq, t0 + qb * bq, min(bq, q - qb * bq), (L - q) + qb * bq);
  };
  if (N > kPlanSortCap) {
    for (int idx = tid; idx < N; idx += NT) {
      int seq, qb;
      locate(idx, seq, qb);
      place(idx, seq, qb);
    }
    return;
  }
  // counting sort by decreasing key-tile count
  for (int k = tid; k < kPlanBuckets; k += NT) hist[k] = 0;
  __syncthreads();
  for (int idx = tid; idx < N; idx += NT) {
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
  for (int base = 0; base < kPlanBuckets; base += NT) {
    const int b = kPlanBuckets - 1 - (base + tid);
    const int v[1] = {hist[b]};
    int ex[1], tot[1];
    plan_scan<1, NT>(v, ex, tot);
    hist[b] = hcarry + ex[0];  // bucket b is read and written by this thread only
    hcarry += tot[0];
  }
  __syncthreads();
  for (int idx = tid; idx < N; idx += NT) {
    int seq, qb;
    locate(idx, seq, qb);
    place(atomicAdd(&hist[keys[idx]], 1), seq, qb);
  }
}

}  // namespace

hipError_t launch_plan(const BatchArgs& a, const DecodePlan& dp, const PrefillPlan& pp,
                       bool with_prefill, hipStream_t st, KernelTiming* tm) {
  if (a.num_seqs <= 0) return hipSuccess;
  // Small batches (at most 64 sequences and 64 Q-block slots): one wave,
  // whose scans need no workgroup barriers (0.3 us shorter on a 128-token
  // prompt; with a hundred Q-blocks the block's 256 threads are faster).
  if (a.num_seqs <= 64 && (!with_prefill || pp.work_items <= 64))
    launch_k(plan_kernel<64>, dim3(1), dim3(64), st, tm, a, dp, pp, with_prefill ? 1 : 0);
  else
    launch_k(plan_kernel<kPlanThreads>, dim3(1), dim3(kPlanThreads), st, tm, a, dp, pp, with_prefill ? 1 : 0);
  return hipGetLastError();
}

}  // namespace pa

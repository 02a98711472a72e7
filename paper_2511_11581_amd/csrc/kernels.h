// Argument blocks and launchers shared by the host API and the HIP kernels.
// All strides are in bytes unless named otherwise.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

constexpr int kPrefillTileKeys = 64;   // keys per tile of the Q-block kernels
// Q-block kernel: waves of 32 rows.  bf16 caches: 8 waves (BLOCK_M = 256,
// one workgroup per CU, two waves per SIMD) or 4 waves (BLOCK_M = 128, two
// workgroups per CU), tiles copied straight into LDS; fp8 caches: 8 waves,
// tiles copied into per-wave staging and widened to bf16 in LDS.
constexpr int kQblockWaveRows = 32;
// Decode workgroup: 4 waves, one workgroup per CU (its LDS use keeps a
// second one out), so one wave per SIMD.  With two waves on a SIMD the
// memory system serves the first wave slot first and the second finishes
// ~1.5x later, which a static split of the steps cannot absorb; deeper
// per-wave pipelines (three register sets) and two workgroups per CU
// measured no faster than one wave per SIMD with one step in flight.
constexpr int kDecodeWaves = 4;

// Division of a key position (0 <= p < 2^31) by the block size, any
// multiple of 16 up to 2^20: floor(p / bs) = mulhi(p, mul) >> shr with
// l = ceil(log2 bs), mul = ceil(2^(31 + l) / bs) < 2^32, shr = l - 1
// (division by invariant integers using multiplication, Granlund and
// Montgomery 1994, Thm. 4.2 for 31-bit numerators).
struct BlockDiv {
  uint32_t mul;
  int32_t shr;
  int32_t bs;
  __host__ __device__ int block(int p) const { return (int)(__umulhi_u32((uint32_t)p, mul) >> shr); }
  __host__ __device__ int slot(int p) const { return p - bs * block(p); }
  // mulhi of 32-bit operands on host and device
  __host__ __device__ static uint32_t __umulhi_u32(uint32_t a, uint32_t b) {
    return (uint32_t)(((uint64_t)a * b) >> 32);
  }
};

struct KvGeom {
  int64_t blk;   // bytes between physical blocks
  int64_t slot;  // bytes between token slots of one block
  int64_t head;  // bytes between kv heads of one slot
};

struct BatchArgs {
  const uint8_t* q;
  int64_t q_tok, q_head;        // q strides (bytes)
  const uint8_t* k;
  const uint8_t* v;
  KvGeom kg, vg;
  const int32_t* bt;            // block table
  int64_t bt_row;               // elements between table rows
  int32_t mb;                   // entries per table row
  const int32_t* seq_lens;
  const int32_t* qsl;           // query_start_loc
  uint8_t* out;
  int64_t o_tok, o_head;        // out strides (bytes)
  int32_t num_seqs, num_tokens, num_blocks, block_size;
  BlockDiv bdiv;                // key position -> (block, slot)
  int32_t num_q_heads, num_kv_heads, group;  // group = Hq / Hkv
  float sl2;                    // softmax scale * log2(e) * k_scale
  float v_scale;
  // Gather-only launches (pa_debug_gather): dense [S, MB * bs, Hkv, d]
  // outputs that receive the cache bytes the attention loaders read.
  uint8_t* kd;
  uint8_t* vd;
  int64_t d_seq, d_tok, d_head;  // dense strides (bytes)
};

// LDS of the decode kernel (kDecodeWaves waves of HU heads of head size d,
// cache element bytes eb): per wave and head a K tile of 32 rows of 2d + 32
// bytes and a V^T tile of d rows of 64 bytes plus 64 bytes of padding every
// 2^dpl rows (dpl = log2 of the d values one lane loads per row); at least
// 81 KB, so that one workgroup fills a CU.  Fused launches build the decode
// list in the rest of the CU's 160 KB, decode_list_cap entries.
__host__ __device__ constexpr int decode_dpl_log2(int d, int eb, int hu) {
  return (hu * d * eb / 16) / eb == 16 ? 4 : ((hu * d * eb / 16) / eb == 8 ? 3 : 2);
}
__host__ __device__ constexpr int decode_wave_lds(int d, int eb, int hu) {
  return hu * (32 * (2 * d + 32) + 16 * (4 * d + 4 * (d >> decode_dpl_log2(d, eb, hu))));
}
__host__ __device__ constexpr int decode_tile_lds(int d, int eb, int hu) {
  return kDecodeWaves * decode_wave_lds(d, eb, hu) > 81 * 1024 ? kDecodeWaves * decode_wave_lds(d, eb, hu)
                                                                : 81 * 1024;
}
__host__ __device__ constexpr int decode_list_cap(int d, int eb, int hu) {
  return (160 * 1024 - decode_tile_lds(d, eb, hu) - 1024) / 16 - 1;
}

struct DecodePlan {
  int32_t workers;     // decode waves in the static grid
  int32_t step_keys;   // keys per decode step (KS)
  int32_t min_steps;   // fewest steps per active worker when the batch allows
  // whole_units = 1 (short sequences): worker w takes the whole units
  // [w U / W, (w + 1) U / W) of the U = J Hu units, W = min(U, workers);
  // no unit is split and no merge follows.
  int32_t whole_units;
  int32_t unit_heads;  // HU: adjacent kv heads one worker computes together
  int32_t* meta;       // [3] written by the plan kernel: decode sequences J, active workers, P(J)
  int4* dec;           // [J + 1] {sequence, token row, length, prefix P(j) of step counts}
  // fused = 1 (decode-only batches): each workgroup builds the decode list
  // in LDS itself, the plan kernel's pass over the sequences, and workgroup
  // 0 also stores it (and meta) for the merge kernel: no plan launch.
  int32_t fused;
  float* part_o;       // [workers, 2, HU, G, head_dim] unnormalised piece results
  float* part_ml;      // [workers, 2, HU, G, 2] (max in log2 units, sum)
};

// Keys per decode step, for units whose rows of one token are unit_bytes
// long (HU heads x head_dim x elem_bytes): one lane loads unit_bytes / 16
// bytes of 8 rows per 32-key sub-tile.  A step is one sub-tile when a lane
// loads 16 bytes (or 8 bytes of fp8), else two, so that a step moves 8-16 KB
// per wave within the register budget of the workgroup shape.
__host__ __device__ constexpr int decode_subtiles(int unit_bytes, int elem_bytes) {
  return unit_bytes / 16 >= (elem_bytes == 1 ? 8 : 16) ? 1 : 2;
}
__host__ __device__ constexpr int decode_step_keys(int unit_bytes, int elem_bytes) {
  return 32 * decode_subtiles(unit_bytes, elem_bytes);
}

// Even split of the decode tile space (total steps over all (sequence, kv
// head) pairs) over W workers: worker w takes [worker_begin(w), worker_begin(w + 1)).
__host__ __device__ inline int64_t worker_begin(int64_t w, int64_t total, int64_t W) {
  return w * total / W;
}
// The worker whose range holds step t (0 <= t < total).
__host__ __device__ inline int worker_of(int64_t t, int64_t total, int64_t W) {
  return (int)(((t + 1) * W - 1) / total);
}
// Workers given work: every worker gets at least min_steps steps when the
// batch has that many, at most W, none for an empty batch.
__host__ __device__ inline int active_workers(int64_t total, int64_t min_steps, int64_t W) {
  if (total <= 0) return 0;
  const int64_t want = (total + min_steps - 1) / min_steps;
  return (int)(want < W ? want : W);
}

struct PrefillPlan {
  int32_t block_m;     // rows per Q-block (BLOCK_M; bf16: 256 or 128, i.e. 8 or 4 waves)
  int32_t block_q;     // query tokens per Q-block (BLOCK_M / group)
  int32_t qmin;        // fewest query tokens of a Q-block row (2; 1: no split-KV decode rows)
  int32_t work_items;  // Q-block slots in the grid (upper bound)
  int32_t* seq_start;  // [num_seqs + 1] prefix sums of Q-blocks per sequence
  int32_t* list_seq;   // [work_items] sequence of the w-th Q-block (planned order)
  int32_t* list_qb;    // [work_items] Q-block index inside that sequence
  int32_t* count;      // [1] number of Q-blocks
  int4* rec;           // [work_items] (sequence, first token, rows, keys before the first row)
  // fused = 1 (batches of at most kFusedPlanSeqs sequences with no split-KV
  // decode launch, whose Q-blocks fit two rounds of workgroups): no plan
  // launch; each Q-block workgroup derives its own record, the one of its
  // rank in the plan kernel's order.
  int32_t fused;
};
constexpr int kFusedPlanSeqs = 16;

struct ValidateArgs {
  const int32_t* bt;
  int64_t bt_row;
  int32_t mb;
  const int32_t* seq_lens;
  const int32_t* qsl;
  int32_t num_seqs, num_tokens, num_blocks, block_size;
  int32_t hint_no_decode;   // 1: no sequence may have query length 1
  int32_t hint_max_q;       // >= 0: no query length may exceed it
  uint32_t* error_word;
};

// Start and end stamps of one launch (PA_FLAG_PROFILE).  A launcher given
// one launches through hipExtLaunchKernel, so that the runtime stamps the
// kernel's dispatch itself: the duration is the kernel's own, without the
// dispatch latency that event markers recorded around the launch add.
// `used` tells whether a kernel was launched (an empty batch launches none).
struct KernelTiming {
  hipEvent_t start;
  hipEvent_t stop;
  bool used;
};

// Launch `kernel` on `st` (no dynamic LDS), timed into *tm when tm is given.
template <typename F, typename... Args>
inline void launch_k(F kernel, dim3 grid, dim3 block, hipStream_t st, KernelTiming* tm, Args... args) {
  if (tm) {
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, tm->start, tm->stop, 0, args...);
    tm->used = true;
  } else {
    kernel<<<grid, block, 0, st>>>(args...);
  }
}

// Launchers (return hipGetLastError() of the launch).  With gather = true
// the attention kernels run their K/V loaders only and store the loaded
// bytes of every valid key into a.kd / a.vd (pa_debug_gather).
hipError_t launch_decode(const BatchArgs& a, const DecodePlan& p, int head_dim, bool fp8,
                         hipStream_t st, bool gather = false, KernelTiming* tm = nullptr);
hipError_t launch_merge(const BatchArgs& a, const DecodePlan& p, int head_dim, hipStream_t st,
                        KernelTiming* tm = nullptr);
hipError_t launch_plan(const BatchArgs& a, const DecodePlan& dp, const PrefillPlan& pp,
                       bool with_prefill, hipStream_t st, KernelTiming* tm = nullptr);
hipError_t launch_qblock(const BatchArgs& a, const PrefillPlan& p, int head_dim, bool fp8,
                         hipStream_t st, bool gather = false, KernelTiming* tm = nullptr);

// KV-cache write (csrc/cache.hip).
struct CacheWriteArgs {
  const uint8_t* key;      // bf16 [T, Hkv, d], last dim contiguous
  const uint8_t* value;
  int64_t k_tok, k_head, v_tok, v_head;   // input strides (bytes)
  const int32_t* slots;    // [T] block * block_size + offset; outside the cache: skipped
  uint8_t* kc;             // caches [NB, bs, Hkv, d] (bf16 or fp8 e4m3fn)
  uint8_t* vc;
  KvGeom kg, vg;
  int64_t num_slots;       // NB * block_size
  int32_t num_tokens, num_kv_heads, head_dim, block_size;
  BlockDiv bdiv;
  int32_t fp8;
  float k_scale, v_scale;  // fp8: stored code = e4m3fn(value / scale)
};
hipError_t launch_cache_write(const CacheWriteArgs& a, hipStream_t st);
// The paper's baseline decomposition, for the ablation (csrc/baseline.hip).
hipError_t launch_baseline(const BatchArgs& a, int head_dim, bool fp8, hipStream_t st);
hipError_t launch_validate(const ValidateArgs& a, hipStream_t st);

}  // namespace pa

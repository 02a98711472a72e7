// Argument blocks and launchers shared by the host API and the HIP kernels.
// All strides are in bytes unless named otherwise.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

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
  int32_t bs_log2;              // block_size = 1 << bs_log2
  int32_t num_q_heads, num_kv_heads, group;  // group = Hq / Hkv
  float sl2;                    // softmax scale * log2(e) * k_scale
  float v_scale;
};

struct DecodePlan {
  int32_t seg_len;     // keys per segment (multiple of 128)
  int32_t max_splits;  // segments per sequence at most
  int32_t head_major;  // grid order: kv head fastest (1) or segment fastest (0)
  float* part_o;       // [num_seqs, max_splits, Hq, head_dim] unnormalised
  float* part_ml;      // [num_seqs, max_splits, Hq, 2] (max in log2 units, sum)
};

struct PrefillPlan {
  int32_t block_q;     // query tokens per Q-block (BLOCK_M / group)
  int32_t work_items;  // Q-block slots in the grid (upper bound)
  int32_t* seq_start;  // [num_seqs + 1] prefix sums of Q-blocks per sequence
  int32_t* list_seq;   // [work_items] sequence of the w-th Q-block (planned order)
  int32_t* list_qb;    // [work_items] Q-block index inside that sequence
  int32_t* count;      // [1] number of Q-blocks
};

struct GatherArgs {
  const uint8_t* k;
  const uint8_t* v;
  KvGeom kg, vg;
  const int32_t* bt;
  int64_t bt_row;
  int32_t mb;
  const int32_t* seq_lens;
  uint8_t* kd;
  uint8_t* vd;
  int64_t d_seq, d_tok, d_head;  // dense output strides (bytes)
  int32_t num_seqs, num_blocks, block_size, num_kv_heads;
  int32_t bs_log2;
  int32_t row_bytes;             // bytes of one head's row (head_dim * elem)
};

struct ValidateArgs {
  const int32_t* bt;
  int64_t bt_row;
  int32_t mb;
  const int32_t* seq_lens;
  const int32_t* qsl;
  int32_t num_seqs, num_tokens, num_blocks, block_size;
  uint32_t* error_word;
};

// Launchers (return hipGetLastError() of the launch).
hipError_t launch_decode(const BatchArgs& a, const DecodePlan& p, int head_dim, bool fp8,
                         hipStream_t st);
hipError_t launch_merge(const BatchArgs& a, const DecodePlan& p, int head_dim, hipStream_t st);
hipError_t launch_prefill_plan(const BatchArgs& a, const PrefillPlan& p, hipStream_t st);
hipError_t launch_prefill(const BatchArgs& a, const PrefillPlan& p, int head_dim, bool fp8,
                          hipStream_t st);
hipError_t launch_gather(const GatherArgs& a, hipStream_t st);
hipError_t launch_validate(const ValidateArgs& a, hipStream_t st);

}  // namespace pa

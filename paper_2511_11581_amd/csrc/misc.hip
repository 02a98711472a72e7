// Debug gather and device-side metadata validation.
//
// gather_kernel walks the block table exactly as the attention kernels do
// (page_of + slot offset, 16-byte loads) and stores the bytes of every valid
// key/value row in logical order into dense [S, MB*bs, Hkv, row] buffers, so
// block-table addressing can be checked bit for bit (Sec. 4.3).
//
// validate_kernel checks the preconditions of a well-formed paged batch
// (Sec. 4.2 terminology, Sec. 4.3 block table) and ORs an error code into a
// device word.
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

// grid: (ceil(MB*bs / 4), S, Hkv); block 256 = 4 keys x 64 lanes of 16 B.
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  const int s = blockIdx.y, g = blockIdx.z;
  const int key = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int L = min(a.seq_lens[s], a.mb * a.block_size);
  if (key >= L) return;
  const int32_t* bt_row = a.bt + (int64_t)s * a.bt_row;
  const int pg = page_of(bt_row, key, a.bs_log2, a.num_blocks);
  const int slot = key & (a.block_size - 1);
  for (int c = lane; c * 16 < a.row_bytes; c += 64) {
    const u32x4 kw = ld16(a.k + (int64_t)pg * a.kg.blk + (int64_t)slot * a.kg.slot +
                          (int64_t)g * a.kg.head + 16 * c);
    const u32x4 vw = ld16(a.v + (int64_t)pg * a.vg.blk + (int64_t)slot * a.vg.slot +
                          (int64_t)g * a.vg.head + 16 * c);
    const int64_t off = (int64_t)s * a.d_seq + (int64_t)key * a.d_tok + (int64_t)g * a.d_head + 16 * c;
    *(u32x4*)(a.kd + off) = kw;
    *(u32x4*)(a.vd + off) = vw;
  }
}

// Error bits written by validate_kernel.
enum : uint32_t {
  kErrQsl0 = 1u,          // query_start_loc[0] != 0
  kErrQslOrder = 2u,      // query_start_loc decreasing
  kErrQLen = 4u,          // query length > seq_len or seq_len < 0
  kErrCapacity = 8u,      // seq_len > table width * block_size
  kErrBlock = 16u,        // block id outside [0, num_blocks)
  kErrTokens = 32u,       // query_start_loc[S] > num_tokens
};

// grid: (S), block 256.
__global__ __launch_bounds__(256) void validate_kernel(ValidateArgs a) {
  const int s = blockIdx.x;
  uint32_t err = 0;
  const int q0 = a.qsl[s], q1 = a.qsl[s + 1];
  const int L = a.seq_lens[s];
  if (threadIdx.x == 0) {
    if (s == 0 && q0 != 0) err |= kErrQsl0;
    if (q1 < q0) err |= kErrQslOrder;
    if (L < 0 || q1 - q0 > L) err |= kErrQLen;
    if ((int64_t)L > (int64_t)a.mb * a.block_size) err |= kErrCapacity;
    if (s == a.num_seqs - 1 && q1 > a.num_tokens) err |= kErrTokens;
  }
  const int64_t nb = min((int64_t)(L > 0 ? L : 0), (int64_t)a.mb * a.block_size);
  const int nblk = (int)((nb + a.block_size - 1) / a.block_size);
  for (int b = threadIdx.x; b < nblk; b += blockDim.x) {
    const int id = a.bt[(int64_t)s * a.bt_row + b];
    if (id < 0 || id >= a.num_blocks) err |= kErrBlock;
  }
  if (err) atomicOr(a.error_word, err);
}

}  // namespace

hipError_t launch_gather(const GatherArgs& a, hipStream_t st) {
  const int64_t keys = (int64_t)a.mb * a.block_size;
  if (a.num_seqs <= 0 || keys <= 0) return hipSuccess;
  dim3 grid((unsigned)((keys + 3) / 4), a.num_seqs, a.num_kv_heads), block(256);
  gather_kernel<<<grid, block, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateArgs& a, hipStream_t st) {
  if (a.num_seqs <= 0) return hipSuccess;
  validate_kernel<<<dim3(a.num_seqs), dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace pa

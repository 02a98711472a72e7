// Device-side metadata validation.
//
// validate_kernel checks the preconditions of a well-formed paged batch
// (Sec. 4.2 terminology, Sec. 4.3 block table) and ORs an error code into a
// device word.
#include "common.hpp"
#include "kernels.h"

namespace pa {

namespace {

// Error bits written by validate_kernel.
enum : uint32_t {
  kErrQsl0 = 1u,          // query_start_loc[0] != 0
  kErrQslOrder = 2u,      // query_start_loc decreasing
  kErrQLen = 4u,          // query length > seq_len or seq_len < 0
  kErrCapacity = 8u,      // seq_len > table width * block_size
  kErrBlock = 16u,        // block id outside [0, num_blocks)
  kErrTokens = 32u,       // query_start_loc[S] > num_tokens
  kErrHint = 64u,         // the batch hint does not hold
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
    if ((a.hint_no_decode && q1 - q0 == 1) || (a.hint_max_q >= 0 && q1 - q0 > a.hint_max_q)) err |= kErrHint;
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

hipError_t launch_validate(const ValidateArgs& a, hipStream_t st) {
  if (a.num_seqs <= 0) return hipSuccess;
  validate_kernel<<<dim3(a.num_seqs), dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace pa

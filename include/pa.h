/*
 * pa.h -- C ABI of libpa.so, paged attention for AMD MI355X (gfx950).
 *
 * What is computed (arxiv 2511.11581, Sec. 4.1 Eq. 1 and Eq. 2; Sec. 4.2
 * terminology; Sec. 4.3 paged KV cache and block table): for a batch of
 * sequences described by query_start_loc (the accumulated query lengths,
 * App. A) and seq_lens (sequence length = context length + query length),
 * every query token j of sequence i (absolute position c_i + j, where
 * c_i = seq_lens[i] - q_i) and every query head h attends causally to keys
 * 0 .. c_i + j of its sequence, using kv head h / (Hq / Hkv) (grouped-query
 * attention, Sec. 4.1):
 *     out[t, h, :] = softmax_p(scale * <q[t, h, :], K[p]>) . V[p]
 * Key position p of sequence i is stored in physical block
 * block_table[i][p / block_size], slot p % block_size.  Q, K and V are
 * already computed and K/V of the query tokens are already in the cache
 * (Sec. 4.3).
 *
 * Conventions shared by every entry point:
 *  - Pointers inside pa_tensor are device pointers; the caller owns all
 *    device memory and keeps it alive until the stream work completes.
 *  - Host-visible problems (dtype, ndim, shapes, strides, alignment, head
 *    configuration, workspace size) are reported by the return value BEFORE
 *    anything is enqueued; a thread-local message is then available from
 *    pa_last_error().
 *  - Device-resident metadata (query_start_loc, seq_lens, block ids) is not
 *    read by the host.  Malformed metadata gives unspecified output values
 *    but never an out-of-bounds access: kernels clamp block ids into
 *    [0, num_blocks), sequence lengths to the table capacity and token
 *    ranges to [0, num_tokens).  With PA_FLAG_VALIDATE the metadata is
 *    checked on the device first and pa_forward synchronises to report it.
 *  - Nothing here allocates device memory or synchronises the stream
 *    (except the PA_FLAG_VALIDATE check), so pa_forward can be captured in
 *    a HIP graph.
 */
#ifndef PA_H_
#define PA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A hipStream_t, declared opaquely so that this header needs no HIP
 * headers.  NULL means the default stream. */
typedef struct ihipStream_t *pa_stream;

typedef enum pa_status {
  PA_OK = 0,
  PA_ERR_INVALID_ARG = 1,  /* malformed argument (shape, dtype, stride, null) */
  PA_ERR_UNSUPPORTED = 2,  /* well-formed but not supported by this library */
  PA_ERR_WORKSPACE = 3,    /* workspace missing or too small */
  PA_ERR_DEVICE = 4,       /* HIP error, or PA_FLAG_VALIDATE found bad metadata */
} pa_status;

typedef enum pa_dtype {
  PA_DTYPE_BF16 = 0,       /* bfloat16 */
  PA_DTYPE_FP8_E4M3 = 1,   /* OCP 8-bit e4m3fn, stored as bytes */
  PA_DTYPE_I32 = 2,
  PA_DTYPE_F32 = 3,
} pa_dtype;

#define PA_MAX_DIMS 4

/* A strided device array.  shape/stride are in elements; the innermost
 * dimension must have stride 1. */
typedef struct pa_tensor {
  void *data;
  int32_t dtype;              /* pa_dtype */
  int32_t ndim;
  int64_t shape[PA_MAX_DIMS];
  int64_t stride[PA_MAX_DIMS];
} pa_tensor;

/* Check query_start_loc / seq_lens / block ids on the device before the
 * attention kernels run; pa_forward then synchronises its stream and
 * returns PA_ERR_DEVICE on a violation.  Debug only. */
#define PA_FLAG_VALIDATE 1u

/* Time every kernel launch of pa_forward so that pa_profile_read can report
 * per-kernel durations: each kernel is launched through hipExtLaunchKernel
 * with a pair of the handle's HIP events, which the runtime stamps at the
 * kernel's own dispatch start and end (the timestamps a rocprofv3 kernel
 * trace reports).  Off by default; not meant for calls under HIP-graph
 * capture. */
#define PA_FLAG_PROFILE 2u

/* Ablation only (the middle rung of the optimisation ladder of Sec. 7):
 * rows with one query token go through the Q-block kernel too, as Q-blocks
 * of one token whose G heads are the rows (Sec. 4.4), with no split of
 * their keys and no merge, instead of through the split-KV decode kernel
 * (Sec. 4.5).  Same results within the tolerances; slower on small batches
 * of long rows. */
#define PA_FLAG_NO_SPLIT_KV 4u

typedef struct pa_config {
  int32_t num_q_heads;     /* Hq */
  int32_t num_kv_heads;    /* Hkv; Hq % Hkv == 0; G = Hq / Hkv must divide 128 and be <= 16 */
  int32_t head_dim;        /* d: 64 or 128 */
  int32_t block_size;      /* tokens per KV-cache block: any multiple of 16 in [16, 2^20]
                              (powers of two, and the large non-power-of-two sizes
                              of hybrid attention / state-space models, Sec. 4.6) */
  int32_t kv_dtype;        /* PA_DTYPE_BF16 or PA_DTYPE_FP8_E4M3 */
  float k_scale;           /* fp8 dequantisation: K = decode(k_cache) * k_scale (1 for bf16) */
  float v_scale;           /* V = decode(v_cache) * v_scale (1 for bf16) */
  uint32_t flags;          /* PA_FLAG_* */
  void *workspace;         /* device scratch owned by the caller, 256-byte aligned */
  uint64_t workspace_bytes;
} pa_config;

typedef struct pa_handle pa_handle;

/* Kernel kinds reported by pa_profile_read. */
enum {
  PA_KERNEL_DECODE = 0,   /* persistent split-KV decode workers */
  PA_KERNEL_MERGE = 1,    /* log-sum-exp merge of decode pieces */
  PA_KERNEL_PREFILL = 2,  /* Q-block kernel (rows with >= 2 query tokens) */
  PA_KERNEL_PLAN = 3,     /* per-batch work lists built on the device */
  PA_KERNEL_KINDS = 4
};

typedef struct pa_profile {
  int64_t launches[PA_KERNEL_KINDS];  /* timed launches since the last reset */
  double total_ms[PA_KERNEL_KINDS];   /* summed event-to-event durations */
} pa_profile;

/* The launch decisions for one batch shape (host-visible sizes only).
 *
 * Decode work (rows with one query token) is split as the parallel tiled
 * softmax of Sec. 4.5, with the segment boundaries chosen for a static
 * launch grid (Sec. 4.7).  The kv heads are grouped in units of
 * decode_unit_heads (HU) adjacent heads, so that a unit's cache rows of one
 * token form a run of at least 256 bytes; the (sequence, unit) pairs of the
 * batch, each ceil(L / decode_step) steps long, are laid end to end and the
 * resulting step range is cut into equal contiguous shares, one per worker
 * group of HU waves, wave i of a group taking kv head HU u + i of every unit
 * u in its share.  The part of one (sequence, kv head) pair inside one
 * share is a segment ("piece").  The device activates
 * min(decode_workers / HU, ceil(total steps / decode_min_steps)) groups, so
 * a single pair of 32 steps with decode_min_steps = 8 is cut into 4
 * segments of 8 steps (the example of Fig. 4).  The default minimum share is
 * 1 step (environment PA_DECODE_MIN_STEPS, read when a handle is created):
 * for batches too small to fill the grid, the serial steps of one worker
 * cost more than the merge of more segments.  Where no sequence can be
 * longer than PA_DECODE_WHOLE_STEPS steps (default 8; from the table width,
 * max_blocks_per_seq x block_size keys), the shares are whole pairs
 * instead (decode_whole_units): every segment covers its pair and the
 * merge launch is skipped. */
typedef struct pa_plan_info {
  int32_t decode_launch;     /* 1 if the decode kernel is launched (single-token rows on it) */
  int32_t decode_step;       /* keys per decode step (32, 64 or 128) */
  int32_t decode_waves;      /* waves per decode workgroup */
  int32_t decode_workers;    /* waves in the static decode grid */
  int32_t decode_min_steps;  /* fewest steps per active worker group, batch permitting */
  int32_t decode_unit_heads; /* kv heads per decode unit (HU, see above) */
  int32_t decode_whole_units; /* 1: no sequence can exceed PA_DECODE_WHOLE_STEPS decode steps
                                 (default 8; max_blocks_per_seq x block_size keys), so each
                                 worker takes whole (sequence, unit) pairs and no merge runs */
  int32_t merge_launch;      /* 1 if the log-sum-exp merge kernel is launched */
  int32_t prefill_qmin;      /* fewest query tokens of a Q-block row: 2 (single-token rows
                                take the decode kernel), or 1 (every row as Q-blocks, no
                                decode launch: PA_FLAG_NO_SPLIT_KV, or a hinted mixed batch
                                whose Q-blocks, its single-token rows included, fill at most
                                one round of workgroups and whose table width bounds every
                                sequence to PA_UNIFY_MAX_KEYS keys, default 8192) */
  int32_t prefill_launch;    /* 1 if the Q-block (q_len >= 2) kernel is launched */
  int32_t block_m;           /* rows per Q-block (BLOCK_M, Sec. 4.4) */
  int32_t block_q;           /* query tokens per Q-block (BLOCK_Q = BLOCK_M / G) */
  int32_t prefill_tile;      /* keys per prefill tile */
  int64_t decode_grid[3];
  int64_t merge_grid[3];
  int64_t prefill_grid[3];
  int64_t prefill_units;     /* Q-block slots x kv heads: the prefill work units */
  uint64_t workspace_bytes;  /* workspace this batch shape needs */
} pa_plan_info;

/* One segment of the decode partition (see pa_plan_info). */
typedef struct pa_decode_piece {
  int32_t seq;        /* sequence index */
  int32_t kv_head;
  int32_t worker;     /* worker (wave) that computes it */
  int32_t first_key;  /* keys [first_key, end_key) of the sequence */
  int32_t end_key;
  int32_t slot;       /* -1: the whole row, written to out directly;
                         0 / 1: partial slot of the worker, merged afterwards */
} pa_decode_piece;

/* Workspace bytes that suffice for every batch with at most max_seqs
 * sequences, max_tokens query rows and max_blocks_per_seq table entries per
 * sequence, under cfg's head configuration.  cfg->workspace is ignored. */
pa_status pa_workspace_bytes(const pa_config *cfg, int64_t max_tokens, int64_t max_seqs,
                             int64_t max_blocks_per_seq, uint64_t *bytes);

/* Validate cfg and create a handle bound to the current HIP device.  The
 * handle holds host state only (device properties, the workspace pointer);
 * it is immutable after creation.  Concurrent pa_forward calls on different
 * streams need handles with distinct workspaces. */
pa_status pa_create(const pa_config *cfg, pa_handle **out);

/* Enqueue attention for one batch on `stream`.
 *   q               bf16 [T, Hq, d]
 *   k_cache/v_cache kv_dtype [num_blocks, block_size, Hkv, d]
 *   block_table     int32 [S, MB]; entries past a sequence's last block are ignored
 *   seq_lens        int32 [S]
 *   query_start_loc int32 [S + 1]; query_start_loc[0] = 0, non-decreasing,
 *                   query_start_loc[S] <= T
 *   scale           softmax scale (1/sqrt(d) for Eq. 1)
 *   out             bf16 [T, Hq, d]; rows [0, query_start_loc[S]) are written
 *                   exactly once, other rows are untouched.
 * All base pointers and all non-unit strides must be 16-byte aligned in
 * bytes.  Sequences with query length 1 run on the persistent split-KV
 * decode kernel (+ merge), the others on the Q-block kernel; a one-workgroup
 * plan kernel builds both work lists on the device first (batches of at most
 * 16 sequences with no decode launch, whose Q-blocks fit two rounds of
 * workgroups, skip it: each Q-block workgroup finds its own work item). */
pa_status pa_forward(pa_handle *h, const pa_tensor *q, const pa_tensor *k_cache,
                     const pa_tensor *v_cache, const pa_tensor *block_table,
                     const pa_tensor *seq_lens, const pa_tensor *query_start_loc, float scale,
                     const pa_tensor *out, pa_stream stream);

/* Facts about a batch that the host already has (the metadata step of
 * Sec. 6.1 computes them from host-side lengths), so that pa_forward_hinted
 * skips launches that would find no work.  -1 means unknown. */
typedef struct pa_batch_hint {
  int32_t num_decode_seqs;  /* sequences with exactly one query token */
  int32_t max_query_len;    /* the longest query length in the batch */
} pa_batch_hint;

/* pa_forward with a hint: num_decode_seqs == 0 skips the split-KV decode
 * and merge launches; 0 <= max_query_len <= 1 skips the Q-block launch and
 * its work list.  hint == NULL, or -1 in both fields, is pa_forward.  The
 * hint must hold: rows of a kind the hint rules out are left unwritten
 * (with PA_FLAG_VALIDATE a violated hint is reported as PA_ERR_DEVICE). */
pa_status pa_forward_hinted(pa_handle *h, const pa_tensor *q, const pa_tensor *k_cache,
                            const pa_tensor *v_cache, const pa_tensor *block_table,
                            const pa_tensor *seq_lens, const pa_tensor *query_start_loc,
                            float scale, const pa_tensor *out, const pa_batch_hint *hint,
                            pa_stream stream);

/* For callers that cannot allocate device memory (code under HIP-graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * attention, kernels and arguments as pa_forward, but the call's scratch
 * (decode list, decode partials, Q-block work list) lives in a static
 * device array of the library (48 MiB, held on every GPU the library runs
 * on until the process ends) instead of the handle's workspace, which may
 * be NULL.  The handle must have been created on the device of `stream`.
 * Returns PA_ERR_WORKSPACE, before enqueuing anything, when the batch's
 * plan needs more scratch than the array holds (pa_plan reports the
 * bytes).  Allocates nothing.  Every call on one GPU shares that GPU's
 * array: calls that overlap in time on one GPU (other streams, other
 * threads, other handles) race and must be serialised by the caller. */
pa_status pa_forward_noalloc(pa_handle *h, const pa_tensor *q, const pa_tensor *k_cache,
                             const pa_tensor *v_cache, const pa_tensor *block_table,
                             const pa_tensor *seq_lens, const pa_tensor *query_start_loc,
                             float scale, const pa_tensor *out, pa_stream stream);

/* Ablation only: the same attention as pa_forward, computed with the
 * paper's baseline decomposition (Sec. 4 / App. A, the first rung of the
 * optimisation ladder of Sec. 7): one wave per (query token, query head),
 * the sequence found by binary search over query_start_loc, one page per
 * key tile, no GQA packing, no split, no matrix cores.  Same arguments,
 * checks and output as pa_forward; much slower; not for production use. */
pa_status pa_forward_baseline(pa_handle *h, const pa_tensor *q, const pa_tensor *k_cache,
                              const pa_tensor *v_cache, const pa_tensor *block_table,
                              const pa_tensor *seq_lens, const pa_tensor *query_start_loc,
                              float scale, const pa_tensor *out, pa_stream stream);

/* Debug: the block-table walk of the attention kernels, checked bit for
 * bit (Sec. 4.3).  Runs the same work lists and the same K/V loaders as
 * pa_forward for a batch with this metadata, but stores the bytes each
 * loader reads instead of computing with them: every key p < seq_lens[i] of
 * a sequence with query length 1 through the decode kernel's loads, of a
 * sequence with query length >= 2 through the Q-block kernel's loads (its
 * last Q-block, which reads all of the sequence's keys).  The bytes go to
 * k_dense / v_dense, both of the cache dtype and shape
 * [S, MB * block_size, Hkv, d], at [i, p, g, :]; positions >= seq_lens[i]
 * and sequences with query length 0 (which attention reads nothing of) are
 * untouched.  num_tokens is the q row count pa_forward would get (T); the
 * handle's workspace must fit the batch as for pa_forward.  Asynchronous on
 * `stream`. */
pa_status pa_debug_gather(pa_handle *h, const pa_tensor *k_cache, const pa_tensor *v_cache,
                          const pa_tensor *block_table, const pa_tensor *seq_lens,
                          const pa_tensor *query_start_loc, int64_t num_tokens,
                          const pa_tensor *k_dense, const pa_tensor *v_dense, pa_stream stream);

/* Write the keys and values of new tokens into the paged caches (the step
 * before attention; arxiv 2511.11581 Sec. 4.2 / 4.3 take it as done).
 *   key, value      bf16 [T, Hkv, d], last dimension contiguous, rows 16-byte
 *                   aligned (views into a larger projection output are fine)
 *   slot_mapping    int32 [T]: slot = block * block_size + offset of token t;
 *                   slots < 0 (padding) or >= num_blocks * block_size are
 *                   skipped
 *   k_cache/v_cache kv_dtype [num_blocks, block_size, Hkv, d] as for pa_forward
 * bf16 caches receive the bits unchanged; fp8 caches receive the e4m3fn code
 * of value / k_scale (resp. v_scale) computed in fp32, limited to +-448,
 * rounded to nearest with ties to even (so that pa_forward's
 * decode(cache) * scale returns the value).  Every new token owns its slot
 * (Sec. 4.3): slot_mapping must not name one slot twice among its non-skipped
 * entries; if it does, that slot ends up holding an unspecified mix of the
 * tokens' 16-byte chunks (the tokens are written concurrently) and the call
 * still returns PA_OK.  Asynchronous on `stream`; allocates nothing;
 * capturable. */
pa_status pa_cache_write(pa_handle *h, const pa_tensor *key, const pa_tensor *value,
                         const pa_tensor *slot_mapping, const pa_tensor *k_cache,
                         const pa_tensor *v_cache, pa_stream stream);

/* The launch plan pa_forward (hint NULL) or pa_forward_hinted (hint given)
 * would use for a batch with these host-visible sizes on a device with
 * num_cus compute units (num_cus <= 0: the handle's device, or 256 without
 * a handle).  Host only; no HIP call.  h may be NULL, then cfg is used. */
pa_status pa_plan(const pa_handle *h, const pa_config *cfg, int32_t num_cus, int64_t num_tokens,
                  int64_t num_seqs, int64_t max_blocks_per_seq, const pa_batch_hint *hint,
                  pa_plan_info *out);

/* The decode partition pa_forward computes on the device, reproduced on
 * the host for metadata given in HOST memory (seq_lens [num_seqs],
 * query_start_loc [num_seqs + 1]) and a device with num_cus compute units
 * (<= 0: the handle's device, or 256).  Writes the first `cap` pieces in
 * order of workers and sets *count to the total.  For inspection and tests;
 * no HIP call.  h may be NULL, then cfg is used. */
pa_status pa_decode_pieces(const pa_handle *h, const pa_config *cfg, int32_t num_cus,
                           const int32_t *seq_lens, const int32_t *query_start_loc,
                           int64_t num_seqs, int64_t num_tokens, int64_t max_blocks_per_seq,
                           pa_decode_piece *pieces, int64_t cap, int64_t *count);

/* Per-kernel durations recorded under PA_FLAG_PROFILE (zeros otherwise).
 * Waits for the recorded events to complete; with reset != 0 the counters
 * restart from zero afterwards. */
pa_status pa_profile_read(pa_handle *h, pa_profile *out, int reset);

/* Release the handle (and its profiling events). */
void pa_destroy(pa_handle *h);

/* Message of the last failing call on this thread ("" if none). */
const char *pa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PA_H_ */

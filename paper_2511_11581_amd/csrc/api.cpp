// Host side of libpa.so: argument validation, the launch planner and the
// kernel launches behind the C ABI declared in include/pa.h.
//
// The planner sees host-visible sizes only (T, S, the block-table width MB,
// the head configuration and the CU count); it never reads device metadata,
// so pa_forward neither synchronises nor copies anything to the host.  Per
// call it launches, in stream order:
//   1. the plan kernel (one workgroup): decode list and Q-block work list,
//      built from the device metadata (Sec. 6.1);
//   2. the decode kernel: a static grid of persistent waves (Sec. 4.7) that
//      split the key tiles of all single-token rows evenly (Sec. 4.5);
//   3. the log-sum-exp merge of pairs that span several workers;
//   4. the Q-block kernel for rows with two or more query tokens (Sec. 4.4),
//      BLOCK_M = 256 or 128 rows (bf16 caches, chosen from the batch shape),
//      256 (fp8 caches), i.e. BLOCK_Q = BLOCK_M / G tokens.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pa.h"
#include "kernels.h"

// Ring of event pairs of one kernel kind (PA_FLAG_PROFILE).
struct pa_event_ring {
  std::vector<hipEvent_t> start, stop;
  int used = 0;
};

// Launch-planner knobs, read from the environment when a handle is created
// (defaults: the offline tuning's rules below).
struct pa_tunables {
  int decode_min_steps;    // fewest decode steps per active worker group (PA_DECODE_MIN_STEPS, 1..4096)
  int decode_whole_steps;  // whole pairs per worker up to this many steps (PA_DECODE_WHOLE_STEPS; 0: off)
  int64_t unify_max_keys;  // hinted mixed batches as Q-blocks only up to this many keys (PA_UNIFY_MAX_KEYS)
  int qblock_rows;         // 0: chosen from the batch shape; else 128 or 256 (PA_QBLOCK_ROWS, bf16 caches)
};

struct pa_handle {
  pa_config cfg;
  int device;
  int cus;
  uint8_t* scratch;   // this device's copy of the library's static scratch (pa_forward_noalloc)
  pa_tunables tun;
  bool profile;
  pa_event_ring ring[PA_KERNEL_KINDS];
  int64_t launches[PA_KERNEL_KINDS];
  double total_ms[PA_KERNEL_KINDS];
};

namespace {

// Scratch for pa_forward_noalloc: the same contents as a caller's workspace
// (decode list, decode partials, Q-block work list), in a file-scope device
// array that every GPU the library runs on holds until the process ends.
// Host code never passes `scratch` itself to a kernel: its name is a
// host-side stand-in, not a device address; pa_create takes each device's
// address with hipGetSymbolAddress once and keeps it in g_scratch[device].
constexpr uint64_t kScratchBytes = 48ull << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
uint8_t* g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

thread_local std::string g_err;

pa_status fail(pa_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

constexpr int kMaxCus = 256;
// Minimum decode share (steps per active worker group), from an offline
// sweep over 15 decode shapes (1..128 sequences, 1K..32K keys; Sec. 5's
// tuning exported as a rule): 1 was best or within noise in all but one.
constexpr int kMinStepsDefault = 1;
// Whole (sequence, unit) pairs per decode worker, with no merge launch, when
// no sequence can exceed this many steps (table width x block size): below
// it the merge launch costs more than splitting the keys saves.
constexpr int kWholeStepsDefault = 8;
// A hinted batch mixing single-token rows with longer queries runs every row
// as Q-blocks (one launch: no decode kernel, no merge) when all its Q-block
// units, the single-token rows' included, fit in one round of workgroups
// and no sequence can be longer than this many keys (table width x block
// size): then the single-token rows run beside the prefill Q-blocks instead
// of before them.  This is the paper's choice for mixed batches (Sec. 4.5:
// the split kernel is for decode batches of long sequences); the key bound
// keeps a long decode row from becoming the batch's longest Q-block.
constexpr int64_t kUnifyMaxKeysDefault = 8192;
constexpr int kPrefillTile = 64;
constexpr uint64_t kHeader = 256;  // validation word + alignment
constexpr uint64_t kMeta = 256;    // decode-list counters written by the plan kernel

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

int elem_bytes(int dt) {
  switch (dt) {
    case PA_DTYPE_BF16: return 2;
    case PA_DTYPE_FP8_E4M3: return 1;
    case PA_DTYPE_I32: return 4;
    case PA_DTYPE_F32: return 4;
    default: return 0;
  }
}

pa_status check_config(const pa_config* c) {
  if (!c) return fail(PA_ERR_INVALID_ARG, "config is NULL");
  if (c->num_q_heads <= 0 || c->num_kv_heads <= 0)
    return fail(PA_ERR_INVALID_ARG, "head counts must be positive (Hq=%d, Hkv=%d)", c->num_q_heads,
                c->num_kv_heads);
  if (c->num_q_heads % c->num_kv_heads != 0)
    return fail(PA_ERR_INVALID_ARG, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)",
                c->num_q_heads, c->num_kv_heads);
  const int G = c->num_q_heads / c->num_kv_heads;
  if (G > 16 || (128 % G) != 0)
    return fail(PA_ERR_UNSUPPORTED, "query heads per kv head must be 1, 2, 4, 8 or 16 (got %d)", G);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(PA_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", c->head_dim);
  if (c->block_size < 16 || c->block_size % 16 != 0 || c->block_size > (1 << 20))
    return fail(PA_ERR_UNSUPPORTED, "block_size must be a multiple of 16 in [16, 2^20] (got %d)",
                c->block_size);
  if (c->kv_dtype != PA_DTYPE_BF16 && c->kv_dtype != PA_DTYPE_FP8_E4M3)
    return fail(PA_ERR_UNSUPPORTED, "kv_dtype must be bf16 or fp8 e4m3 (got %d)", c->kv_dtype);
  if (!(c->k_scale > 0.f) || !(c->v_scale > 0.f))
    return fail(PA_ERR_INVALID_ARG, "k_scale and v_scale must be positive");
  if (c->flags & ~(PA_FLAG_VALIDATE | PA_FLAG_PROFILE | PA_FLAG_NO_SPLIT_KV))
    return fail(PA_ERR_INVALID_ARG, "unknown flags 0x%x", c->flags);
  if (c->workspace && (reinterpret_cast<uintptr_t>(c->workspace) & 255))
    return fail(PA_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  return PA_OK;
}

// Q-block slots of the prefill grid: sum_i ceil(q_i / BQ) <= ceil(T / BQ) +
// (#sequences with q_i >= qmin), qmin = 2 (1 when single-token rows also
// take Q-blocks).
int64_t prefill_items(int64_t T, int64_t S, int64_t bq, int qmin = 2) {
  return cdiv(T, bq) + std::min<int64_t>(S, T / qmin);
}

int decode_unit_heads(const pa_config& c);
int decode_step_keys(const pa_config& c) {
  const int eb = c.kv_dtype == PA_DTYPE_FP8_E4M3 ? 1 : 2;
  return pa::decode_step_keys(decode_unit_heads(c) * c.head_dim * eb, eb);
}

// Rows per Q-block.  fp8 caches: 256 (the bf16 kernel's 8-wave shape,
// widening its copies to bf16 in LDS).  bf16 caches: 256
// (8 waves, one workgroup per CU) or 128 (4 waves, two workgroups per CU),
// chosen from host-visible sizes by a decision tree fitted offline to the
// faster of the two on 47 prefill-heavy shapes (1-64 sequences, 16-4096 new
// tokens, 0 or 4096 cached, G 4 and 8; Sec. 5 / Lst. 2 / Fig. 8), which
// brings the geometric-mean loss against the best choice from 7.4% (always
// 256) to 0.3%, the worst from 41% to 4.5%.  Smaller Q-blocks pay off while
// sequences are short or the 256-row grid would not fill the CUs twice.
// PA_QBLOCK_ROWS (128 or 256, read when a handle is created) forces one.
constexpr int kBlockMMin = 128;
constexpr int kBlockMMax = 256;   // one workgroup per CU; 128 rows: two
int block_m(const pa_config& c, const pa_tunables& tun, int cus, int64_t T, int64_t S, int64_t MB) {
  if (c.kv_dtype == PA_DTYPE_FP8_E4M3) return 256;   // the fp8 staging runs 8 waves
  if (tun.qblock_rows) return tun.qblock_rows;
  if (T < 2 || S < 1) return 256;
  const int G = c.num_q_heads / c.num_kv_heads;
  const double waves256 =
      (double)(prefill_items(T, S, 256 / G, 2) * c.num_kv_heads) / (double)std::max(cus, 1);
  const double tokens_per_seq = (double)T / (double)S;
  const int64_t max_keys = MB * c.block_size;
  if (tokens_per_seq <= 1536.0) return (max_keys <= 4736 || waves256 <= 1.33) ? 128 : 256;
  return (tokens_per_seq <= 3072.0 && waves256 > 9.14) ? 128 : 256;
}

int decode_workers(int cus) { return std::min(std::max(cus, 1), kMaxCus) * pa::kDecodeWaves; }

// kv heads one decode worker computes together: the most adjacent heads (a
// power of two dividing Hkv) whose rows of one token stay within 256 bytes,
// so that the worker's reads per token form one run of 256 bytes when rows
// are shorter.
int decode_unit_heads(const pa_config& c) {
  const int row = c.head_dim * (c.kv_dtype == PA_DTYPE_FP8_E4M3 ? 1 : 2);
  int hu = 1;
  while (hu * 2 * row <= 256 && c.num_kv_heads % (hu * 2) == 0) hu *= 2;
  return hu;
}

// Workspace layout: validation header, decode-list counters, decode list
// [S + 1] int4, piece partials [workers, 2, HU, G, d] and
// [workers, 2, HU, G, 2] fp32, then the Q-block work list (seq_start
// [S + 1], list_seq, list_qb, the per-item records, count).
struct WsLayout {
  uint64_t meta, dec, part_o, part_ml, seq_start, list_seq, list_qb, rec, count, total;
};

WsLayout ws_layout(const pa_config& c, int workers, int64_t S, int64_t items) {
  const int G = c.num_q_heads / c.num_kv_heads * decode_unit_heads(c);   // partial rows per slot
  WsLayout l;
  uint64_t off = kHeader;
  l.meta = off;
  off += kMeta;
  l.dec = off;
  off += align256((uint64_t)(S + 1) * 16);
  l.part_o = off;
  off += align256((uint64_t)workers * 2 * G * c.head_dim * 4);
  l.part_ml = off;
  off += align256((uint64_t)workers * 2 * G * 2 * 4);
  l.seq_start = off;
  off += items > 0 ? align256((uint64_t)(S + 1) * 4) : 0;
  l.list_seq = off;
  off += align256((uint64_t)items * 4);
  l.list_qb = off;
  off += align256((uint64_t)items * 4);
  l.rec = off;
  off += align256((uint64_t)items * 16);
  l.count = off;
  off += items > 0 ? 256 : 0;
  l.total = off;
  return l;
}

pa_tunables tunables_from_env() {
  pa_tunables t{kMinStepsDefault, kWholeStepsDefault, kUnifyMaxKeysDefault, 0};
  if (const char* e = std::getenv("PA_DECODE_MIN_STEPS")) {
    const int v = std::atoi(e);
    if (v >= 1) t.decode_min_steps = std::min(v, 4096);
  }
  if (const char* e = std::getenv("PA_DECODE_WHOLE_STEPS")) {
    const int v = std::atoi(e);
    if (v >= 0) t.decode_whole_steps = std::min(v, 4096);
  }
  if (const char* e = std::getenv("PA_UNIFY_MAX_KEYS")) {
    const long long v = std::atoll(e);
    if (v >= 0) t.unify_max_keys = v;
  }
  if (const char* e = std::getenv("PA_QBLOCK_ROWS")) {
    const int v = std::atoi(e);
    if (v == 128 || v == 256) t.qblock_rows = v;
  }
  return t;
}

void make_plan(const pa_config& c, const pa_tunables& tun, int cus, int64_t T, int64_t S,
               int64_t MB, pa_plan_info* p, const pa_batch_hint* hint = nullptr) {
  std::memset(p, 0, sizeof *p);
  const int G = c.num_q_heads / c.num_kv_heads;
  const int64_t max_len = MB * c.block_size;
  p->decode_step = decode_step_keys(c);
  p->decode_waves = pa::kDecodeWaves;
  p->decode_workers = decode_workers(cus);
  p->decode_min_steps = tun.decode_min_steps;
  p->decode_unit_heads = decode_unit_heads(c);
  p->block_m = block_m(c, tun, cus, T, S, MB);
  p->block_q = p->block_m / G;
  p->prefill_tile = kPrefillTile;
  int64_t items = 0;
  if (S >= 1 && T >= 1 && max_len >= 1) {
    int qmin = (c.flags & PA_FLAG_NO_SPLIT_KV) ? 1 : 2;
    if (qmin == 2 && hint && hint->num_decode_seqs > 0 && hint->max_query_len >= 2 &&
        max_len <= tun.unify_max_keys &&
        prefill_items(T, S, p->block_q, 1) * c.num_kv_heads <=
            (int64_t)cus * (kBlockMMax / p->block_m))
      qmin = 1;   // a small mixed batch: every row as Q-blocks
    p->prefill_qmin = qmin;
    if (qmin == 2) {
      p->decode_launch = 1;
      p->decode_grid[0] = p->decode_workers / p->decode_waves;
      p->decode_grid[1] = 1;
      p->decode_grid[2] = 1;
      p->decode_whole_units = cdiv(max_len, p->decode_step) <= tun.decode_whole_steps ? 1 : 0;
      if (!p->decode_whole_units) {
        p->merge_launch = 1;
        p->merge_grid[0] = S;
        p->merge_grid[1] = (G + 3) / 4;
        p->merge_grid[2] = c.num_kv_heads;
      }
    }
    if (T >= qmin && max_len >= qmin) {
      p->prefill_launch = 1;
      items = prefill_items(T, S, p->block_q, qmin);
      p->prefill_units = items * c.num_kv_heads;
      p->prefill_grid[0] = p->prefill_units;   // one workgroup per unit
      p->prefill_grid[1] = 1;
      p->prefill_grid[2] = 1;
    }
    p->workspace_bytes = ws_layout(c, p->decode_workers, S, items).total;
  } else {
    p->workspace_bytes = kHeader;
  }
}

// ---- tensor checks -------------------------------------------------------

pa_status check_tensor(const pa_tensor* t, const char* name, int dtype, int ndim) {
  if (!t) return fail(PA_ERR_INVALID_ARG, "%s is NULL", name);
  if (t->dtype != dtype) return fail(PA_ERR_INVALID_ARG, "%s has dtype %d, expected %d", name, t->dtype, dtype);
  if (t->ndim != ndim) return fail(PA_ERR_INVALID_ARG, "%s has %d dims, expected %d", name, t->ndim, ndim);
  for (int i = 0; i < ndim; ++i) {
    if (t->shape[i] < 0 || t->shape[i] > INT32_MAX)
      return fail(PA_ERR_INVALID_ARG, "%s dim %d has size %lld", name, i, (long long)t->shape[i]);
    if (t->stride[i] < 0) return fail(PA_ERR_INVALID_ARG, "%s has a negative stride", name);
  }
  if (t->stride[ndim - 1] != 1 && t->shape[ndim - 1] > 1)
    return fail(PA_ERR_INVALID_ARG, "%s must be contiguous in its last dimension", name);
  int64_t numel = 1;
  for (int i = 0; i < ndim; ++i) numel *= t->shape[i];
  if (numel > 0 && !t->data) return fail(PA_ERR_INVALID_ARG, "%s has a NULL data pointer", name);
  return PA_OK;
}

// 16-byte alignment of the base and of every outer stride, in bytes.
pa_status check_aligned16(const pa_tensor* t, const char* name) {
  const int eb = elem_bytes(t->dtype);
  if (reinterpret_cast<uintptr_t>(t->data) & 15)
    return fail(PA_ERR_INVALID_ARG, "%s base pointer must be 16-byte aligned", name);
  for (int i = 0; i + 1 < t->ndim; ++i)
    if ((t->stride[i] * eb) & 15)
      return fail(PA_ERR_INVALID_ARG, "%s stride %d (%lld elements) must be a multiple of 16 bytes",
                  name, i, (long long)t->stride[i]);
  return PA_OK;
}

#define TRY(x)                   \
  do {                           \
    pa_status st_ = (x);         \
    if (st_ != PA_OK) return st_; \
  } while (0)

struct Shapes {
  int64_t T, S, MB, NB;
};

pa_status check_batch(const pa_config& c, const pa_tensor* q, const pa_tensor* k, const pa_tensor* v,
                      const pa_tensor* bt, const pa_tensor* sl, const pa_tensor* qsl,
                      const pa_tensor* out, Shapes* sh) {
  TRY(check_tensor(q, "q", PA_DTYPE_BF16, 3));
  TRY(check_tensor(k, "k_cache", c.kv_dtype, 4));
  TRY(check_tensor(v, "v_cache", c.kv_dtype, 4));
  TRY(check_tensor(bt, "block_table", PA_DTYPE_I32, 2));
  TRY(check_tensor(sl, "seq_lens", PA_DTYPE_I32, 1));
  TRY(check_tensor(qsl, "query_start_loc", PA_DTYPE_I32, 1));
  if (out) TRY(check_tensor(out, "out", PA_DTYPE_BF16, 3));
  const int64_t T = q->shape[0], S = sl->shape[0], NB = k->shape[0], MB = bt->shape[1];
  if (q->shape[1] != c.num_q_heads || q->shape[2] != c.head_dim)
    return fail(PA_ERR_INVALID_ARG, "q must be [T, %d, %d]", c.num_q_heads, c.head_dim);
  for (const pa_tensor* kv : {k, v}) {
    if (kv->shape[1] != c.block_size || kv->shape[2] != c.num_kv_heads || kv->shape[3] != c.head_dim)
      return fail(PA_ERR_INVALID_ARG, "caches must be [num_blocks, %d, %d, %d]", c.block_size,
                  c.num_kv_heads, c.head_dim);
  }
  if (v->shape[0] != NB) return fail(PA_ERR_INVALID_ARG, "k_cache and v_cache block counts differ");
  if (bt->shape[0] != S) return fail(PA_ERR_INVALID_ARG, "block_table has %lld rows, seq_lens %lld",
                                     (long long)bt->shape[0], (long long)S);
  if (qsl->shape[0] != S + 1)
    return fail(PA_ERR_INVALID_ARG, "query_start_loc must have num_seqs + 1 = %lld entries", (long long)(S + 1));
  if (out && (out->shape[0] != T || out->shape[1] != c.num_q_heads || out->shape[2] != c.head_dim))
    return fail(PA_ERR_INVALID_ARG, "out must have the shape of q");
  if (S > 0 && NB < 1) return fail(PA_ERR_INVALID_ARG, "the cache holds no blocks");
  if (S > 65535) return fail(PA_ERR_UNSUPPORTED, "at most 65535 sequences per call (got %lld)", (long long)S);
  if (MB * c.block_size > INT32_MAX - 65536) return fail(PA_ERR_UNSUPPORTED, "block table too wide");
  for (const pa_tensor* kv : {k, v})
    if ((int64_t)c.block_size * kv->stride[1] * elem_bytes(kv->dtype) >= INT32_MAX ||
        kv->stride[2] * elem_bytes(kv->dtype) >= INT32_MAX)
      return fail(PA_ERR_UNSUPPORTED, "cache slot/head strides too large for 32-bit in-block offsets");
  for (const pa_tensor* kv : {k, v})
    if (kv->stride[0] * elem_bytes(kv->dtype) >= ((int64_t)1 << 32))
      return fail(PA_ERR_UNSUPPORTED, "cache block stride must be below 4 GiB");
  TRY(check_aligned16(q, "q"));
  TRY(check_aligned16(k, "k_cache"));
  TRY(check_aligned16(v, "v_cache"));
  if (out) TRY(check_aligned16(out, "out"));
  if (reinterpret_cast<uintptr_t>(bt->data) & 3 || reinterpret_cast<uintptr_t>(sl->data) & 3 ||
      reinterpret_cast<uintptr_t>(qsl->data) & 3)
    return fail(PA_ERR_INVALID_ARG, "int32 metadata must be 4-byte aligned");
  sh->T = T;
  sh->S = S;
  sh->MB = MB;
  sh->NB = NB;
  return PA_OK;
}

// The decode and Q-block work-list descriptors of plan p inside workspace ws.
void device_plans(const pa_config& c, const pa_plan_info& p, uint8_t* ws, int64_t S,
                  pa::DecodePlan* dp, pa::PrefillPlan* pp) {
  const int64_t items = p.prefill_launch ? p.prefill_units / c.num_kv_heads : 0;
  const WsLayout wl = ws_layout(c, p.decode_workers, S, items);
  dp->workers = p.decode_workers;
  dp->step_keys = p.decode_step;
  dp->min_steps = p.decode_min_steps;
  dp->whole_units = p.decode_whole_units;
  dp->unit_heads = p.decode_unit_heads;
  dp->meta = reinterpret_cast<int32_t*>(ws + wl.meta);
  dp->fused = 0;
  dp->dec = reinterpret_cast<int4*>(ws + wl.dec);
  dp->part_o = reinterpret_cast<float*>(ws + wl.part_o);
  dp->part_ml = reinterpret_cast<float*>(ws + wl.part_ml);
  pp->block_m = p.block_m;
  pp->block_q = p.block_q;
  pp->qmin = p.prefill_qmin;
  pp->work_items = (int32_t)items;
  pp->seq_start = reinterpret_cast<int32_t*>(ws + wl.seq_start);
  pp->list_seq = reinterpret_cast<int32_t*>(ws + wl.list_seq);
  pp->list_qb = reinterpret_cast<int32_t*>(ws + wl.list_qb);
  pp->count = reinterpret_cast<int32_t*>(ws + wl.count);
  pp->rec = reinterpret_cast<int4*>(ws + wl.rec);
  pp->fused = 0;
}

// floor(p / bs) by multiply-high and shift (see pa::BlockDiv).
pa::BlockDiv block_div(int bs) {
  int l = 0;
  while ((1 << l) < bs) ++l;   // ceil(log2 bs), bs >= 16
  pa::BlockDiv d;
  d.mul = (uint32_t)((((uint64_t)1 << (31 + l)) + (uint64_t)bs - 1) / (uint64_t)bs);
  d.shr = l - 1;
  d.bs = bs;
  return d;
}

pa::KvGeom geom(const pa_tensor* t) {
  const int eb = elem_bytes(t->dtype);
  return pa::KvGeom{t->stride[0] * eb, t->stride[1] * eb, t->stride[2] * eb};
}

pa_status hip_fail(hipError_t e, const char* what) {
  return fail(PA_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kRingCap = 512;

// Wait for the recorded events of one kind and add their durations.
hipError_t flush_ring(pa_handle* h, int kind) {
  pa_event_ring& r = h->ring[kind];
  for (int i = 0; i < r.used; ++i) {
    hipError_t e = hipEventSynchronize(r.stop[i]);
    if (e != hipSuccess) return e;
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.start[i], r.stop[i]);
    if (e != hipSuccess) return e;
    h->total_ms[kind] += ms;
    h->launches[kind] += 1;
  }
  r.used = 0;
  return hipSuccess;
}

// Launch through `fn(tm)`.  When profiling, tm carries the next event pair
// of the kernel kind's ring: the launcher has the runtime stamp the
// kernel's own start and end into it; a launcher that finds nothing to
// launch leaves it unused, and the pair is then recorded back to back (a
// zero duration).
template <class F>
hipError_t timed_launch(pa_handle* h, int kind, hipStream_t st, F&& fn) {
  if (!h->profile) return fn(nullptr);
  pa_event_ring& r = h->ring[kind];
  if (r.used == kRingCap) {
    hipError_t e = flush_ring(h, kind);
    if (e != hipSuccess) return e;
  }
  pa::KernelTiming tm{r.start[r.used], r.stop[r.used], false};
  hipError_t e = fn(&tm);
  if (e != hipSuccess) return e;
  if (!tm.used) {
    e = hipEventRecord(tm.start, st);
    if (e != hipSuccess) return e;
    e = hipEventRecord(tm.stop, st);
    if (e != hipSuccess) return e;
  }
  r.used += 1;
  return hipSuccess;
}

void destroy_events(pa_handle* h) {
  for (auto& r : h->ring) {
    for (hipEvent_t ev : r.start) (void)hipEventDestroy(ev);
    for (hipEvent_t ev : r.stop) (void)hipEventDestroy(ev);
    r.start.clear();
    r.stop.clear();
  }
}

}  // namespace

extern "C" {

const char* pa_last_error(void) { return g_err.c_str(); }

pa_status pa_workspace_bytes(const pa_config* cfg, int64_t max_tokens, int64_t max_seqs,
                             int64_t max_blocks_per_seq, uint64_t* bytes) {
  TRY(check_config(cfg));
  if (!bytes) return fail(PA_ERR_INVALID_ARG, "bytes is NULL");
  if (max_tokens < 0 || max_seqs < 0 || max_blocks_per_seq < 0)
    return fail(PA_ERR_INVALID_ARG, "negative maximum");
  // The layout grows with S and T and with the worker count, which is
  // largest on the largest device, so that batch and device bound all.
  uint64_t best = kHeader;
  if (max_seqs >= 1 && max_tokens >= 1 && max_blocks_per_seq * cfg->block_size >= 1) {
    // most Q-blocks: the smallest BLOCK_M, single-token rows included (the
    // no-split flag, or a hinted small mixed batch)
    const int64_t bq = kBlockMMin / (cfg->num_q_heads / cfg->num_kv_heads);
    const int64_t items = prefill_items(max_tokens, max_seqs, bq, 1);
    best = ws_layout(*cfg, decode_workers(kMaxCus), max_seqs, items).total;
  }
  *bytes = best;
  return PA_OK;
}

pa_status pa_plan(const pa_handle* h, const pa_config* cfg, int32_t num_cus, int64_t num_tokens,
                  int64_t num_seqs, int64_t max_blocks_per_seq, const pa_batch_hint* hint,
                  pa_plan_info* out) {
  const pa_config* c = h ? &h->cfg : cfg;
  TRY(check_config(c));
  if (!out) return fail(PA_ERR_INVALID_ARG, "out is NULL");
  if (num_tokens < 0 || num_seqs < 0 || max_blocks_per_seq < 0)
    return fail(PA_ERR_INVALID_ARG, "negative size");
  int cus = num_cus > 0 ? num_cus : (h ? h->cus : kMaxCus);
  make_plan(*c, h ? h->tun : tunables_from_env(), cus, num_tokens, num_seqs, max_blocks_per_seq, out,
            hint);
  return PA_OK;
}

pa_status pa_decode_pieces(const pa_handle* h, const pa_config* cfg, int32_t num_cus,
                           const int32_t* seq_lens, const int32_t* query_start_loc, int64_t num_seqs,
                           int64_t num_tokens, int64_t max_blocks_per_seq, pa_decode_piece* pieces,
                           int64_t cap, int64_t* count) {
  const pa_config* c = h ? &h->cfg : cfg;
  TRY(check_config(c));
  if (!count) return fail(PA_ERR_INVALID_ARG, "count is NULL");
  if (num_seqs < 0 || num_tokens < 0 || max_blocks_per_seq < 0 || cap < 0)
    return fail(PA_ERR_INVALID_ARG, "negative size");
  if (num_seqs > 0 && (!seq_lens || !query_start_loc))
    return fail(PA_ERR_INVALID_ARG, "metadata pointer is NULL");
  if (cap > 0 && !pieces) return fail(PA_ERR_INVALID_ARG, "pieces is NULL");
  const int cus = num_cus > 0 ? num_cus : (h ? h->cus : kMaxCus);
  const pa_tunables tun = h ? h->tun : tunables_from_env();
  const int KS = decode_step_keys(*c), HU = decode_unit_heads(*c), Hu = c->num_kv_heads / HU;
  const int64_t cap_keys = max_blocks_per_seq * c->block_size;
  // The decode list, as the plan kernel builds it.
  struct Dec { int32_t s, L; int64_t P; };
  std::vector<Dec> dec;
  int64_t P = 0;
  for (int64_t i = 0; i < num_seqs; ++i) {
    const int64_t t0 = query_start_loc[i], L = std::min<int64_t>(seq_lens[i], cap_keys);
    if (query_start_loc[i + 1] - t0 == 1 && t0 >= 0 && t0 < num_tokens && L >= 1) {
      dec.push_back(Dec{(int32_t)i, (int32_t)L, P});
      P += cdiv(L, KS);
    }
  }
  const int64_t total = (int64_t)Hu * P;
  int64_t n = 0;
  auto put = [&](int64_t jj, int64_t gu, int w, int64_t k0, int64_t k1, int slot) {
    for (int hu = 0; hu < HU; ++hu, ++n) {
      if (n >= cap) continue;
      pa_decode_piece& pc = pieces[n];
      pc.seq = dec[jj].s;
      pc.kv_head = (int32_t)(gu * HU + hu);
      pc.worker = w;
      pc.first_key = (int32_t)(k0 * KS);
      pc.end_key = (int32_t)std::min<int64_t>(k1 * KS, dec[jj].L);
      pc.slot = slot;
    }
  };
  if (cdiv(cap_keys, KS) <= tun.decode_whole_steps) {
    // Whole pairs per workgroup, their steps split over its waves (the
    // pieces merged inside the workgroup).
    const int64_t U = (int64_t)Hu * (int64_t)dec.size();
    const int64_t B = std::min<int64_t>(U, decode_workers(cus) / pa::kDecodeWaves);
    for (int64_t b = 0; b < B; ++b)
      for (int64_t u = U * b / B; u < U * (b + 1) / B; ++u) {
        const int64_t jj = u / Hu, gu = u % Hu, nt = cdiv(dec[jj].L, KS);
        const int64_t np = std::min<int64_t>(pa::kDecodeWaves, nt);
        for (int64_t i = 0; i < np; ++i)
          put(jj, gu, (int)(b * pa::kDecodeWaves + i), i * nt / np, (i + 1) * nt / np,
              np == 1 ? -1 : (i == 0 ? 1 : 0));
      }
    *count = n;
    return PA_OK;
  }
  const int W = pa::active_workers(total, tun.decode_min_steps, decode_workers(cus));
  // Walk every worker's range of the unit step space, unit by unit; a unit
  // piece is one piece per head of the unit.
  size_t j = 0;
  for (int w = 0; w < W; ++w) {
    int64_t t = pa::worker_begin(w, total, W);
    const int64_t te = pa::worker_begin(w + 1, total, W);
    while (t < te) {
      while (j + 1 < dec.size() && (int64_t)Hu * dec[j + 1].P <= t) ++j;
      const int64_t nt = cdiv(dec[j].L, KS);
      const int64_t off = t - (int64_t)Hu * dec[j].P;
      const int64_t gu = off / nt, k0 = off % nt, k1 = std::min(nt, k0 + (te - t));
      const bool head = k0 > 0, tail = k1 < nt;
      put(j, gu, w, k0, k1, (!head && !tail) ? -1 : (head ? 0 : 1));
      t += k1 - k0;
    }
  }
  *count = n;
  return PA_OK;
}

pa_status pa_create(const pa_config* cfg, pa_handle** out) {
  TRY(check_config(cfg));
  if (!out) return fail(PA_ERR_INVALID_ARG, "out is NULL");
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  uint8_t* scr = nullptr;
  if (dev >= 0 && dev < kMaxDevices) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[dev]) {
      void* ptr = nullptr;
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
      g_scratch[dev] = static_cast<uint8_t*>(ptr);
    }
    scr = g_scratch[dev];
  }
  pa_handle* h = new (std::nothrow) pa_handle;
  if (!h) return fail(PA_ERR_INVALID_ARG, "out of host memory");
  h->cfg = *cfg;
  h->device = dev;
  h->scratch = scr;
  h->cus = cus > 0 ? cus : kMaxCus;
  h->tun = tunables_from_env();
  h->profile = (cfg->flags & PA_FLAG_PROFILE) != 0;
  for (int k = 0; k < PA_KERNEL_KINDS; ++k) {
    h->launches[k] = 0;
    h->total_ms[k] = 0.0;
  }
  if (h->profile) {
    for (auto& r : h->ring) {
      r.start.resize(kRingCap);
      r.stop.resize(kRingCap);
      for (int i = 0; i < kRingCap; ++i) {
        hipError_t e1 = hipEventCreate(&r.start[i]);
        hipError_t e2 = hipEventCreate(&r.stop[i]);
        if (e1 != hipSuccess || e2 != hipSuccess) {
          r.start.resize(e1 == hipSuccess ? i + 1 : i);
          r.stop.resize(e2 == hipSuccess ? i + 1 : i);
          destroy_events(h);
          delete h;
          return hip_fail(e1 != hipSuccess ? e1 : e2, "hipEventCreate");
        }
      }
    }
  }
  *out = h;
  return PA_OK;
}

void pa_destroy(pa_handle* h) {
  if (!h) return;
  destroy_events(h);
  delete h;
}

pa_status pa_profile_read(pa_handle* h, pa_profile* out, int reset) {
  if (!h || !out) return fail(PA_ERR_INVALID_ARG, "handle or out is NULL");
  for (int k = 0; k < PA_KERNEL_KINDS; ++k) {
    hipError_t e = flush_ring(h, k);
    if (e != hipSuccess) return hip_fail(e, "profile events");
    out->launches[k] = h->launches[k];
    out->total_ms[k] = h->total_ms[k];
    if (reset) {
      h->launches[k] = 0;
      h->total_ms[k] = 0.0;
    }
  }
  return PA_OK;
}

// ws / ws_bytes: the device scratch the call uses (the caller's workspace,
// or this device's static scratch for pa_forward_noalloc).
static pa_status forward_impl(pa_handle* h, const pa_tensor* q, const pa_tensor* k_cache,
                              const pa_tensor* v_cache, const pa_tensor* block_table,
                              const pa_tensor* seq_lens, const pa_tensor* query_start_loc,
                              float scale, const pa_tensor* out, pa_stream stream, bool baseline,
                              uint8_t* ws, uint64_t ws_bytes, bool static_scratch,
                              const pa_batch_hint* hint = nullptr) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  const pa_config& c = h->cfg;
  if (!out) return fail(PA_ERR_INVALID_ARG, "out is NULL");
  if (hint && (hint->num_decode_seqs < -1 || hint->max_query_len < -1))
    return fail(PA_ERR_INVALID_ARG, "hint fields must be >= -1");
  Shapes sh;
  TRY(check_batch(c, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out, &sh));
  if (!(scale > 0.f) || !(scale < 1e30f)) return fail(PA_ERR_INVALID_ARG, "scale must be positive and finite");
  pa_plan_info p;
  make_plan(c, h->tun, h->cus, sh.T, sh.S, sh.MB, &p, hint);
  if (sh.S * cdiv(sh.MB * c.block_size, p.decode_step) * c.num_kv_heads > INT32_MAX)
    return fail(PA_ERR_UNSUPPORTED, "batch too large for 32-bit decode step indices");
  if (static_scratch && (!ws || p.workspace_bytes > ws_bytes))
    return fail(PA_ERR_WORKSPACE, "batch needs %llu bytes of scratch; the static scratch holds %llu",
                (unsigned long long)p.workspace_bytes, (unsigned long long)ws_bytes);
  if (!ws || ws_bytes < p.workspace_bytes)
    return fail(PA_ERR_WORKSPACE, "workspace of %llu bytes needed, %llu given",
                (unsigned long long)p.workspace_bytes, (unsigned long long)ws_bytes);
  if (sh.S == 0 || sh.T == 0) return PA_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);

  if (c.flags & PA_FLAG_VALIDATE) {
    uint32_t* word = reinterpret_cast<uint32_t*>(ws);
    hipError_t e = hipMemsetAsync(word, 0, 4, st);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    pa::ValidateArgs va{static_cast<const int32_t*>(block_table->data), block_table->stride[0],
                        (int32_t)sh.MB, static_cast<const int32_t*>(seq_lens->data),
                        static_cast<const int32_t*>(query_start_loc->data), (int32_t)sh.S,
                        (int32_t)sh.T, (int32_t)sh.NB, c.block_size,
                        hint && hint->num_decode_seqs == 0 ? 1 : 0, hint ? hint->max_query_len : -1,
                        word};
    e = pa::launch_validate(va, st);
    if (e != hipSuccess) return hip_fail(e, "validate launch");
    uint32_t host_word = 0;
    e = hipMemcpyAsync(&host_word, word, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "validate readback");
    if (host_word)
      return fail(PA_ERR_DEVICE, "metadata check failed (code 0x%x: 1 qsl[0]!=0, 2 qsl decreasing, "
                  "4 q_len>seq_len, 8 seq_len>table capacity, 16 block id out of range, "
                  "32 qsl[S]>num_tokens, 64 batch hint violated)", host_word);
  }

  const bool fp8 = c.kv_dtype == PA_DTYPE_FP8_E4M3;
  pa::BatchArgs a;
  a.q = static_cast<const uint8_t*>(q->data);
  a.q_tok = q->stride[0] * 2;
  a.q_head = q->stride[1] * 2;
  a.k = static_cast<const uint8_t*>(k_cache->data);
  a.v = static_cast<const uint8_t*>(v_cache->data);
  a.kg = geom(k_cache);
  a.vg = geom(v_cache);
  a.bt = static_cast<const int32_t*>(block_table->data);
  a.bt_row = block_table->stride[0];
  a.mb = (int32_t)sh.MB;
  a.seq_lens = static_cast<const int32_t*>(seq_lens->data);
  a.qsl = static_cast<const int32_t*>(query_start_loc->data);
  a.out = static_cast<uint8_t*>(out->data);
  a.o_tok = out->stride[0] * 2;
  a.o_head = out->stride[1] * 2;
  a.num_seqs = (int32_t)sh.S;
  a.num_tokens = (int32_t)sh.T;
  a.num_blocks = (int32_t)std::min<int64_t>(sh.NB, INT32_MAX);
  a.block_size = c.block_size;
  a.bdiv = block_div(c.block_size);
  a.num_q_heads = c.num_q_heads;
  a.num_kv_heads = c.num_kv_heads;
  a.group = c.num_q_heads / c.num_kv_heads;
  a.sl2 = scale * c.k_scale * 1.4426950408889634f;
  a.v_scale = c.v_scale;
  a.kd = a.vd = nullptr;
  a.d_seq = a.d_tok = a.d_head = 0;

  if (baseline) {
    hipError_t e = pa::launch_baseline(a, c.head_dim, fp8, st);
    if (e != hipSuccess) return hip_fail(e, "baseline launch");
    return PA_OK;
  }
  if (!p.decode_launch && !p.prefill_launch) return PA_OK;
  pa::DecodePlan dp;
  pa::PrefillPlan pp;
  device_plans(c, p, ws, sh.S, &dp, &pp);
  // What the hint rules out.  Single-token rows take Q-blocks under
  // PA_FLAG_NO_SPLIT_KV and in a hinted small mixed batch (the plan's
  // prefill_qmin 1); then only the Q-block launch is needed.
  const bool no_split = p.prefill_qmin == 1;
  const bool run_decode = p.decode_launch && !(hint && hint->num_decode_seqs == 0);
  const bool run_qblock = p.prefill_launch &&
                          !(hint && hint->max_query_len >= 0 && hint->max_query_len < (no_split ? 1 : 2));

  // A batch the hint says is decode-only, with a decode list that fits in the
  // decode kernel's LDS: the decode kernel builds the list itself (no plan
  // launch), then the merge.
  const int eb = fp8 ? 1 : 2;
  const bool fused = run_decode && !run_qblock && hint && hint->max_query_len >= 0 &&
                     sh.S < pa::decode_list_cap(c.head_dim, eb, p.decode_unit_heads);
  hipError_t e;
  if (fused) {
    dp.fused = 1;
    e = timed_launch(h, PA_KERNEL_DECODE, st,
                     [&](pa::KernelTiming* tm) { return pa::launch_decode(a, dp, c.head_dim, fp8, st, false, tm); });
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    if (p.merge_launch) {
      e = timed_launch(h, PA_KERNEL_MERGE, st,
                       [&](pa::KernelTiming* tm) { return pa::launch_merge(a, dp, c.head_dim, st, tm); });
      if (e != hipSuccess) return hip_fail(e, "merge launch");
    }
    return PA_OK;
  }
  // Few sequences, no split-KV decode launch, and Q-blocks that fit two
  // rounds of workgroups: the Q-block workgroups derive their records
  // themselves (~1.4 us each, once per round), so no plan launch precedes
  // them.
  if (run_qblock && !run_decode && sh.S <= pa::kFusedPlanSeqs &&
      p.prefill_units <= 2 * (int64_t)h->cus * (256 / p.block_m)) {
    pp.fused = 1;
    e = timed_launch(h, PA_KERNEL_PREFILL, st, [&](pa::KernelTiming* tm) {
      return pa::launch_qblock(a, pp, c.head_dim, fp8, st, false, tm);
    });
    if (e != hipSuccess) return hip_fail(e, "prefill launch");
    return PA_OK;
  }
  e = timed_launch(h, PA_KERNEL_PLAN, st,
                   [&](pa::KernelTiming* tm) { return pa::launch_plan(a, dp, pp, run_qblock, st, tm); });
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  if (run_decode) {
    e = timed_launch(h, PA_KERNEL_DECODE, st,
                     [&](pa::KernelTiming* tm) { return pa::launch_decode(a, dp, c.head_dim, fp8, st, false, tm); });
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    if (p.merge_launch) {
      e = timed_launch(h, PA_KERNEL_MERGE, st,
                       [&](pa::KernelTiming* tm) { return pa::launch_merge(a, dp, c.head_dim, st, tm); });
      if (e != hipSuccess) return hip_fail(e, "merge launch");
    }
  }
  if (run_qblock) {
    e = timed_launch(h, PA_KERNEL_PREFILL, st,
                     [&](pa::KernelTiming* tm) { return pa::launch_qblock(a, pp, c.head_dim, fp8, st, false, tm); });
    if (e != hipSuccess) return hip_fail(e, "prefill launch");
  }
  return PA_OK;
}

pa_status pa_forward(pa_handle* h, const pa_tensor* q, const pa_tensor* k_cache,
                     const pa_tensor* v_cache, const pa_tensor* block_table,
                     const pa_tensor* seq_lens, const pa_tensor* query_start_loc, float scale,
                     const pa_tensor* out, pa_stream stream) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  return forward_impl(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
                      stream, false, static_cast<uint8_t*>(h->cfg.workspace), h->cfg.workspace_bytes,
                      false);
}

pa_status pa_forward_hinted(pa_handle* h, const pa_tensor* q, const pa_tensor* k_cache,
                            const pa_tensor* v_cache, const pa_tensor* block_table,
                            const pa_tensor* seq_lens, const pa_tensor* query_start_loc,
                            float scale, const pa_tensor* out, const pa_batch_hint* hint,
                            pa_stream stream) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  return forward_impl(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
                      stream, false, static_cast<uint8_t*>(h->cfg.workspace), h->cfg.workspace_bytes,
                      false, hint);
}

pa_status pa_forward_noalloc(pa_handle* h, const pa_tensor* q, const pa_tensor* k_cache,
                             const pa_tensor* v_cache, const pa_tensor* block_table,
                             const pa_tensor* seq_lens, const pa_tensor* query_start_loc,
                             float scale, const pa_tensor* out, pa_stream stream) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  if (!h->scratch)
    return fail(PA_ERR_UNSUPPORTED, "no static scratch on device %d (devices 0..%d only)", h->device,
                kMaxDevices - 1);
  return forward_impl(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
                      stream, false, h->scratch, kScratchBytes, true);
}

pa_status pa_forward_baseline(pa_handle* h, const pa_tensor* q, const pa_tensor* k_cache,
                              const pa_tensor* v_cache, const pa_tensor* block_table,
                              const pa_tensor* seq_lens, const pa_tensor* query_start_loc,
                              float scale, const pa_tensor* out, pa_stream stream) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  return forward_impl(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
                      stream, true, static_cast<uint8_t*>(h->cfg.workspace), h->cfg.workspace_bytes,
                      false);
}

pa_status pa_debug_gather(pa_handle* h, const pa_tensor* k_cache, const pa_tensor* v_cache,
                          const pa_tensor* block_table, const pa_tensor* seq_lens,
                          const pa_tensor* query_start_loc, int64_t num_tokens,
                          const pa_tensor* k_dense, const pa_tensor* v_dense, pa_stream stream) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  const pa_config& c = h->cfg;
  TRY(check_tensor(k_cache, "k_cache", c.kv_dtype, 4));
  TRY(check_tensor(v_cache, "v_cache", c.kv_dtype, 4));
  TRY(check_tensor(block_table, "block_table", PA_DTYPE_I32, 2));
  TRY(check_tensor(seq_lens, "seq_lens", PA_DTYPE_I32, 1));
  TRY(check_tensor(query_start_loc, "query_start_loc", PA_DTYPE_I32, 1));
  TRY(check_tensor(k_dense, "k_dense", c.kv_dtype, 4));
  TRY(check_tensor(v_dense, "v_dense", c.kv_dtype, 4));
  const int64_t S = seq_lens->shape[0], MB = block_table->shape[1], NB = k_cache->shape[0];
  for (const pa_tensor* kv : {k_cache, v_cache})
    if (kv->shape[0] != NB || kv->shape[1] != c.block_size || kv->shape[2] != c.num_kv_heads ||
        kv->shape[3] != c.head_dim)
      return fail(PA_ERR_INVALID_ARG, "caches must be [num_blocks, %d, %d, %d]", c.block_size,
                  c.num_kv_heads, c.head_dim);
  if (block_table->shape[0] != S) return fail(PA_ERR_INVALID_ARG, "block_table rows != num_seqs");
  if (query_start_loc->shape[0] != S + 1)
    return fail(PA_ERR_INVALID_ARG, "query_start_loc must have num_seqs + 1 entries");
  if (num_tokens < 0 || num_tokens > INT32_MAX) return fail(PA_ERR_INVALID_ARG, "num_tokens out of range");
  for (const pa_tensor* dn : {k_dense, v_dense})
    if (dn->shape[0] != S || dn->shape[1] != MB * c.block_size || dn->shape[2] != c.num_kv_heads ||
        dn->shape[3] != c.head_dim)
      return fail(PA_ERR_INVALID_ARG, "dense outputs must be [S, MB * block_size, Hkv, d]");
  if (k_dense->stride[0] != v_dense->stride[0] || k_dense->stride[1] != v_dense->stride[1] ||
      k_dense->stride[2] != v_dense->stride[2])
    return fail(PA_ERR_INVALID_ARG, "k_dense and v_dense must share strides");
  if (S > 65535) return fail(PA_ERR_UNSUPPORTED, "at most 65535 sequences");
  if (S > 0 && NB < 1) return fail(PA_ERR_INVALID_ARG, "the cache holds no blocks");
  if (MB * c.block_size > INT32_MAX - 65536) return fail(PA_ERR_UNSUPPORTED, "block table too wide");
  for (const pa_tensor* kv : {k_cache, v_cache})
    if ((int64_t)c.block_size * kv->stride[1] * elem_bytes(kv->dtype) >= INT32_MAX ||
        kv->stride[2] * elem_bytes(kv->dtype) >= INT32_MAX ||
        kv->stride[0] * elem_bytes(kv->dtype) >= ((int64_t)1 << 32))
      return fail(PA_ERR_UNSUPPORTED, "cache strides too large for the loaders' offsets");
  TRY(check_aligned16(k_cache, "k_cache"));
  TRY(check_aligned16(v_cache, "v_cache"));
  TRY(check_aligned16(k_dense, "k_dense"));
  TRY(check_aligned16(v_dense, "v_dense"));
  if (reinterpret_cast<uintptr_t>(block_table->data) & 3 || reinterpret_cast<uintptr_t>(seq_lens->data) & 3 ||
      reinterpret_cast<uintptr_t>(query_start_loc->data) & 3)
    return fail(PA_ERR_INVALID_ARG, "int32 metadata must be 4-byte aligned");
  pa_plan_info p;
  make_plan(c, h->tun, h->cus, num_tokens, S, MB, &p);
  if (S * cdiv(MB * c.block_size, p.decode_step) * c.num_kv_heads > INT32_MAX)
    return fail(PA_ERR_UNSUPPORTED, "batch too large for 32-bit decode step indices");
  if (!c.workspace || c.workspace_bytes < p.workspace_bytes)
    return fail(PA_ERR_WORKSPACE, "workspace of %llu bytes needed, %llu given",
                (unsigned long long)p.workspace_bytes, (unsigned long long)c.workspace_bytes);
  if (S == 0 || num_tokens == 0 || (!p.decode_launch && !p.prefill_launch)) return PA_OK;
  const int eb = elem_bytes(c.kv_dtype);
  pa::BatchArgs a;
  std::memset(&a, 0, sizeof a);
  a.k = static_cast<const uint8_t*>(k_cache->data);
  a.v = static_cast<const uint8_t*>(v_cache->data);
  a.kg = geom(k_cache);
  a.vg = geom(v_cache);
  a.bt = static_cast<const int32_t*>(block_table->data);
  a.bt_row = block_table->stride[0];
  a.mb = (int32_t)MB;
  a.seq_lens = static_cast<const int32_t*>(seq_lens->data);
  a.qsl = static_cast<const int32_t*>(query_start_loc->data);
  a.num_seqs = (int32_t)S;
  a.num_tokens = (int32_t)num_tokens;
  a.num_blocks = (int32_t)std::min<int64_t>(NB, INT32_MAX);
  a.block_size = c.block_size;
  a.bdiv = block_div(c.block_size);
  a.num_q_heads = c.num_q_heads;
  a.num_kv_heads = c.num_kv_heads;
  a.group = c.num_q_heads / c.num_kv_heads;
  a.sl2 = 1.f;
  a.v_scale = 1.f;
  a.kd = static_cast<uint8_t*>(k_dense->data);
  a.vd = static_cast<uint8_t*>(v_dense->data);
  a.d_seq = k_dense->stride[0] * eb;
  a.d_tok = k_dense->stride[1] * eb;
  a.d_head = k_dense->stride[2] * eb;
  pa::DecodePlan dp;
  pa::PrefillPlan pp;
  device_plans(c, p, static_cast<uint8_t*>(c.workspace), S, &dp, &pp);
  const bool fp8 = c.kv_dtype == PA_DTYPE_FP8_E4M3;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = pa::launch_plan(a, dp, pp, p.prefill_launch != 0, st);
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  if (p.decode_launch) {
    e = pa::launch_decode(a, dp, c.head_dim, fp8, st, true);
    if (e != hipSuccess) return hip_fail(e, "decode gather launch");
  }
  if (p.prefill_launch) {
    e = pa::launch_qblock(a, pp, c.head_dim, fp8, st, true);
    if (e != hipSuccess) return hip_fail(e, "Q-block gather launch");
  }
  return PA_OK;
}

pa_status pa_cache_write(pa_handle* h, const pa_tensor* key, const pa_tensor* value,
                         const pa_tensor* slot_mapping, const pa_tensor* k_cache,
                         const pa_tensor* v_cache, pa_stream stream) {
  if (!h) return fail(PA_ERR_INVALID_ARG, "handle is NULL");
  const pa_config& c = h->cfg;
  TRY(check_tensor(key, "key", PA_DTYPE_BF16, 3));
  TRY(check_tensor(value, "value", PA_DTYPE_BF16, 3));
  TRY(check_tensor(slot_mapping, "slot_mapping", PA_DTYPE_I32, 1));
  TRY(check_tensor(k_cache, "k_cache", c.kv_dtype, 4));
  TRY(check_tensor(v_cache, "v_cache", c.kv_dtype, 4));
  const int64_t T = key->shape[0], NB = k_cache->shape[0];
  for (const pa_tensor* x : {key, value})
    if (x->shape[0] != T || x->shape[1] != c.num_kv_heads || x->shape[2] != c.head_dim)
      return fail(PA_ERR_INVALID_ARG, "key and value must be [T, %d, %d]", c.num_kv_heads, c.head_dim);
  for (const pa_tensor* x : {key, value})
    if (x->stride[2] != 1 || x->stride[0] % 8 != 0 || x->stride[1] % 8 != 0)
      return fail(PA_ERR_INVALID_ARG, "key / value: last dim contiguous, token and head strides multiples of 8");
  if (slot_mapping->shape[0] != T || slot_mapping->stride[0] != 1)
    return fail(PA_ERR_INVALID_ARG, "slot_mapping must be a contiguous int32 [T]");
  for (const pa_tensor* kv : {k_cache, v_cache})
    if (kv->shape[0] != NB || kv->shape[1] != c.block_size || kv->shape[2] != c.num_kv_heads ||
        kv->shape[3] != c.head_dim || kv->stride[3] != 1)
      return fail(PA_ERR_INVALID_ARG, "caches must be [num_blocks, %d, %d, %d] with contiguous rows",
                  c.block_size, c.num_kv_heads, c.head_dim);
  if (T > INT32_MAX) return fail(PA_ERR_UNSUPPORTED, "at most 2^31 - 1 tokens");
  TRY(check_aligned16(key, "key"));
  TRY(check_aligned16(value, "value"));
  TRY(check_aligned16(k_cache, "k_cache"));
  TRY(check_aligned16(v_cache, "v_cache"));
  if (T == 0) return PA_OK;
  pa::CacheWriteArgs a;
  a.key = static_cast<const uint8_t*>(key->data);
  a.value = static_cast<const uint8_t*>(value->data);
  a.k_tok = key->stride[0] * 2;
  a.k_head = key->stride[1] * 2;
  a.v_tok = value->stride[0] * 2;
  a.v_head = value->stride[1] * 2;
  a.slots = static_cast<const int32_t*>(slot_mapping->data);
  a.kc = static_cast<uint8_t*>(k_cache->data);
  a.vc = static_cast<uint8_t*>(v_cache->data);
  a.kg = geom(k_cache);
  a.vg = geom(v_cache);
  a.num_slots = NB * c.block_size;
  a.num_tokens = (int32_t)T;
  a.num_kv_heads = c.num_kv_heads;
  a.head_dim = c.head_dim;
  a.block_size = c.block_size;
  a.bdiv = block_div(c.block_size);
  a.fp8 = c.kv_dtype == PA_DTYPE_FP8_E4M3 ? 1 : 0;
  a.k_scale = c.k_scale;
  a.v_scale = c.v_scale;
  hipError_t e = pa::launch_cache_write(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "cache write launch");
  return PA_OK;
}

}  // extern "C"

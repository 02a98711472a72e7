/*
 * pa_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct fp64 CPU reference for paged attention
 * over a block-table KV cache (arxiv 2511.11581, Sec. 4.1 Eq. 1 and Eq. 2,
 * Sec. 4.2 terminology, Sec. 4.3 block table).  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load this library.
 * It shares no code, header, table or helper with the GPU library.
 *
 * What it computes, for every sequence i of a batch:
 *   t0 = query_start_loc[i], q = query_start_loc[i+1] - t0,
 *   L  = seq_lens[i] (sequence length = context + query, Sec. 4.2),
 *   c  = L - q (context length).
 *   Logical key position p in [0, L) lives in physical block
 *   block_table[i][p / bs] at slot p % bs (Sec. 4.3: the block table maps
 *   logical to physical blocks, bs = BLOCK_SIZE tokens per block).
 *   Query token j in [0, q) sits at absolute position c + j and attends to
 *   keys 0 .. c + j inclusive (causal; the token's own K/V is already in
 *   the cache).  Query head h reads KV head h / (Hq / Hkv) (GQA, Sec. 4.1).
 *   Row result (Eq. 1 with the stable softmax of Eq. 2):
 *     s_p  = scale * sum_x q[t0+j,h,x] * K[p,g,x]
 *     m    = max_p s_p,   w_p = exp(s_p - m),   l = sum_p w_p
 *     out  = sum_p w_p * V[p,g,:] / l
 *
 * Inputs are the stored bits: bf16 as uint16, fp8 e4m3fn (OCP) as uint8.
 * They are decoded to fp64 exactly (every bf16 and every e4m3fn value is
 * exactly representable in fp64).  fp8 caches are dequantised as
 * decode(x) * k_scale (resp. v_scale).  Sums use Neumaier compensation.
 *
 * The split/merge functions restate the parallel tiled softmax of Sec. 4.5
 * (segments of contiguous tiles, each keeping a running max, a running sum
 * of exponentials and an unnormalised result, merged afterwards by
 * rescaling) in fp64, so that the merge rule itself can be checked against
 * the plain definition.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_ERR 1

static char g_err[512];

const char *pa_oracle_last_error(void) { return g_err; }

static int fail(const char *msg, long long a, long long b) {
    snprintf(g_err, sizeof g_err, "%s (%lld, %lld)", msg, a, b);
    return ORACLE_ERR;
}

/* ---- exact decoders ---------------------------------------------------- */

/* bf16: the upper 16 bits of an IEEE binary32. */
double pa_oracle_bf16_to_f64(uint16_t bits) {
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* OCP 8-bit E4M3 ("e4m3fn"): 1 sign bit, 4 exponent bits (bias 7), 3
 * mantissa bits, no infinities, S.1111.111 is NaN, exponent 0 encodes
 * subnormals m * 2^-9. */
double pa_oracle_fp8e4m3_to_f64(uint8_t bits) {
    int sign = (bits >> 7) & 1;
    int e = (bits >> 3) & 0xF;
    int m = bits & 7;
    double v;
    if (e == 0xF && m == 7) return NAN;
    if (e == 0)
        v = ldexp((double)m, -9);
    else
        v = ldexp(1.0 + m / 8.0, e - 7);
    return sign ? -v : v;
}

/* ---- problem description ----------------------------------------------- */

typedef struct {
    const uint16_t *q;      /* [T, Hq, d] bf16 bits */
    const void *k_cache;    /* [NB, bs, Hkv, d] bf16 bits or fp8 bytes */
    const void *v_cache;
    int kv_fp8;
    double k_scale, v_scale;
    const int32_t *block_table; /* [S, MB] */
    const int32_t *seq_lens;    /* [S] */
    const int32_t *qsl;         /* [S+1] */
    int64_t S, T, NB, MB, bs, Hq, Hkv, d;
    double scale;
} problem;

static double kv_at(const problem *P, const void *cache, double sc, int64_t blk,
                    int64_t slot, int64_t g, int64_t x) {
    int64_t idx = ((blk * P->bs + slot) * P->Hkv + g) * P->d + x;
    if (P->kv_fp8) return pa_oracle_fp8e4m3_to_f64(((const uint8_t *)cache)[idx]) * sc;
    return pa_oracle_bf16_to_f64(((const uint16_t *)cache)[idx]);
}

/* Check the batch description against the preconditions that define a
 * well-formed paged batch (Sec. 4.2, Sec. 4.3). */
static int validate(const problem *P) {
    if (P->Hkv <= 0 || P->Hq <= 0 || P->Hq % P->Hkv != 0)
        return fail("num_q_heads must be a positive multiple of num_kv_heads", P->Hq, P->Hkv);
    if (P->d <= 0 || P->bs <= 0) return fail("head_dim and block_size must be positive", P->d, P->bs);
    if (P->S < 0 || P->T < 0) return fail("negative batch size", P->S, P->T);
    if (P->S > 0 && P->qsl[0] != 0) return fail("query_start_loc[0] must be 0", P->qsl[0], 0);
    for (int64_t i = 0; i < P->S; ++i) {
        int64_t q = (int64_t)P->qsl[i + 1] - P->qsl[i];
        int64_t L = P->seq_lens[i];
        if (q < 0) return fail("query_start_loc must be non-decreasing", i, q);
        if (L < q) return fail("seq_len must be >= query length", i, L);
        if (L > P->MB * P->bs) return fail("seq_len exceeds block table capacity", i, L);
        for (int64_t b = 0; b < (L + P->bs - 1) / P->bs; ++b) {
            int32_t blk = P->block_table[i * P->MB + b];
            if (blk < 0 || blk >= P->NB) return fail("block id out of range", i, blk);
        }
    }
    if (P->S > 0 && P->qsl[P->S] > P->T) return fail("query_start_loc[S] exceeds num_tokens", P->qsl[P->S], P->T);
    return ORACLE_OK;
}

/* Neumaier-compensated accumulator. */
typedef struct { double s, c; } acc_t;
static inline void acc_add(acc_t *a, double x) {
    double t = a->s + x;
    if (fabs(a->s) >= fabs(x))
        a->c += (a->s - t) + x;
    else
        a->c += (x - t) + a->s;
    a->s = t;
}
static inline double acc_get(const acc_t *a) { return a->s + a->c; }

/* Scores of one (sequence, query token, query head) row over keys [0, nkeys). */
static void row_scores(const problem *P, int64_t i, int64_t t, int64_t h, int64_t nkeys,
                       double *s) {
    int64_t g = h / (P->Hq / P->Hkv);
    const uint16_t *qrow = P->q + (t * P->Hq + h) * P->d;
    for (int64_t p = 0; p < nkeys; ++p) {
        int64_t blk = P->block_table[i * P->MB + p / P->bs];
        int64_t slot = p % P->bs;
        acc_t a = {0, 0};
        for (int64_t x = 0; x < P->d; ++x)
            acc_add(&a, pa_oracle_bf16_to_f64(qrow[x]) * kv_at(P, P->k_cache, P->k_scale, blk, slot, g, x));
        s[p] = P->scale * acc_get(&a);
    }
}

/* One output row: out[d], optional lse (= m + ln l) and normalised weights. */
static void row_attend(const problem *P, int64_t i, int64_t t, int64_t h, int64_t nkeys,
                       double *s, double *out, double *lse, double *weights) {
    int64_t g = h / (P->Hq / P->Hkv);
    row_scores(P, i, t, h, nkeys, s);
    double m = -INFINITY;
    for (int64_t p = 0; p < nkeys; ++p)
        if (s[p] > m) m = s[p];
    acc_t l = {0, 0};
    for (int64_t p = 0; p < nkeys; ++p) {
        s[p] = exp(s[p] - m); /* s now holds w_p */
        acc_add(&l, s[p]);
    }
    double lsum = acc_get(&l);
    /* out[x] = sum_p w_p V[p, x] / l: one compensated sum per x, each taking
     * the keys in increasing order (keys in the outer loop, so that a key's
     * V row is read once). */
    acc_t *o = (acc_t *)calloc((size_t)P->d, sizeof(acc_t));
    for (int64_t p = 0; p < nkeys; ++p) {
        int64_t blk = P->block_table[i * P->MB + p / P->bs];
        for (int64_t x = 0; x < P->d; ++x)
            acc_add(&o[x], s[p] * kv_at(P, P->v_cache, P->v_scale, blk, p % P->bs, g, x));
    }
    for (int64_t x = 0; x < P->d; ++x) out[x] = acc_get(&o[x]) / lsum;
    free(o);
    if (lse) *lse = m + log(lsum);
    if (weights)
        for (int64_t p = 0; p < nkeys; ++p) weights[p] = s[p] / lsum;
}

/* ---- threaded full forward --------------------------------------------- */

/* Work unit: one query token row t and one kv head g (its G query heads),
 * handed out most keys first. */
typedef struct {
    int64_t keys, unit; /* unit = t * Hkv + g */
} unit_t;

typedef struct {
    const problem *P;
    double *out, *lse;
    unit_t *units;
    int64_t *seq; /* sequence owning each token row, -1 for rows past qsl[S] */
    int64_t nunits;
    int64_t next;
    pthread_mutex_t mu;
} job_t;

static void *worker(void *arg) {
    job_t *J = (job_t *)arg;
    const problem *P = J->P;
    int64_t maxL = 0;
    for (int64_t i = 0; i < P->S; ++i)
        if (P->seq_lens[i] > maxL) maxL = P->seq_lens[i];
    double *s = (double *)malloc(sizeof(double) * (size_t)(maxL > 0 ? maxL : 1));
    int64_t G = P->Hq / P->Hkv;
    for (;;) {
        pthread_mutex_lock(&J->mu);
        int64_t u = J->next < J->nunits ? J->units[J->next++].unit : -1;
        pthread_mutex_unlock(&J->mu);
        if (u < 0) break;
        int64_t t = u / P->Hkv, g = u % P->Hkv, i = J->seq[t];
        int64_t t0 = P->qsl[i], q = P->qsl[i + 1] - t0, L = P->seq_lens[i], c = L - q;
        int64_t j = t - t0;
        for (int64_t h = g * G; h < (g + 1) * G; ++h)
            row_attend(P, i, t, h, c + j + 1, s, J->out + (t * P->Hq + h) * P->d,
                       J->lse ? J->lse + t * P->Hq + h : NULL, NULL);
    }
    free(s);
    return NULL;
}

static int cmp_units(const void *a, const void *b) {
    const unit_t *x = (const unit_t *)a, *y = (const unit_t *)b;
    if (x->keys != y->keys) return x->keys > y->keys ? -1 : 1;
    return x->unit < y->unit ? -1 : (x->unit > y->unit);
}

#define PROBLEM_ARGS                                                                     \
    const uint16_t *q, const void *k_cache, const void *v_cache, int kv_fp8,             \
        double k_scale, double v_scale, const int32_t *block_table, int64_t max_blocks,   \
        const int32_t *seq_lens, const int32_t *query_start_loc, int64_t num_seqs,        \
        int64_t num_tokens, int64_t num_blocks, int64_t block_size, int64_t num_q_heads,  \
        int64_t num_kv_heads, int64_t head_dim, double scale

#define PROBLEM_INIT                                                                     \
    problem P = {q, k_cache, v_cache, kv_fp8, k_scale, v_scale, block_table, seq_lens,   \
                 query_start_loc, num_seqs, num_tokens, num_blocks, max_blocks,           \
                 block_size, num_q_heads, num_kv_heads, head_dim, scale}

/* Full forward.  Writes out[t, h, :] for every t < query_start_loc[S];
 * rows beyond are untouched.  lse may be NULL.  num_threads <= 0 means 1. */
int pa_oracle_forward(PROBLEM_ARGS, double *out, double *lse, int num_threads) {
    PROBLEM_INIT;
    if (validate(&P)) return ORACLE_ERR;
    job_t J;
    J.P = &P;
    J.out = out;
    J.lse = lse;
    int64_t rows = P.S > 0 ? P.qsl[P.S] : 0;
    J.seq = (int64_t *)malloc(sizeof(int64_t) * (size_t)(rows > 0 ? rows : 1));
    for (int64_t i = 0; i < P.S; ++i)
        for (int64_t t = P.qsl[i]; t < P.qsl[i + 1]; ++t) J.seq[t] = i;
    J.nunits = rows * P.Hkv;
    J.units = (unit_t *)malloc(sizeof(unit_t) * (size_t)(J.nunits > 0 ? J.nunits : 1));
    for (int64_t u = 0; u < J.nunits; ++u) {
        int64_t t = u / P.Hkv, i = J.seq[t];
        int64_t q = P.qsl[i + 1] - P.qsl[i];
        J.units[u].keys = (P.seq_lens[i] - q) + (t - P.qsl[i]) + 1;
        J.units[u].unit = u;
    }
    qsort(J.units, (size_t)J.nunits, sizeof(unit_t), cmp_units);
    J.next = 0;
    pthread_mutex_init(&J.mu, NULL);
    int nt = num_threads > 0 ? num_threads : 1;
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nt);
    for (int k = 0; k < nt; ++k) pthread_create(&th[k], NULL, worker, &J);
    for (int k = 0; k < nt; ++k) pthread_join(th[k], NULL);
    pthread_mutex_destroy(&J.mu);
    free(th);
    free(J.units);
    free(J.seq);
    return ORACLE_OK;
}

/* Locate the sequence owning token row t (plain linear scan). */
static int64_t seq_of_token(const problem *P, int64_t t) {
    for (int64_t i = 0; i < P->S; ++i)
        if (t >= P->qsl[i] && t < P->qsl[i + 1]) return i;
    return -1;
}

/* Selected rows: rows[k] = (token, head); out is [n, d]; lse [n] or NULL;
 * weights, if non-NULL, is [n, max_keys] and receives the normalised
 * softmax weights of each row (zero beyond the row's key count). */
int pa_oracle_rows(PROBLEM_ARGS, const int64_t *rows, int64_t n, double *out, double *lse,
                   double *weights, int64_t max_keys) {
    PROBLEM_INIT;
    if (validate(&P)) return ORACLE_ERR;
    int64_t maxL = 1;
    for (int64_t i = 0; i < P.S; ++i)
        if (P.seq_lens[i] > maxL) maxL = P.seq_lens[i];
    double *s = (double *)malloc(sizeof(double) * (size_t)maxL);
    for (int64_t k = 0; k < n; ++k) {
        int64_t t = rows[2 * k], h = rows[2 * k + 1];
        int64_t i = seq_of_token(&P, t);
        if (i < 0 || h < 0 || h >= P.Hq) {
            free(s);
            return fail("row outside the batch", t, h);
        }
        int64_t qlen = P.qsl[i + 1] - P.qsl[i], c = P.seq_lens[i] - qlen, j = t - P.qsl[i];
        int64_t nkeys = c + j + 1;
        double *w = NULL;
        if (weights) {
            if (nkeys > max_keys) {
                free(s);
                return fail("max_keys too small for row", nkeys, max_keys);
            }
            w = weights + k * max_keys;
            for (int64_t p = 0; p < max_keys; ++p) w[p] = 0.0;
        }
        row_attend(&P, i, t, h, nkeys, s, out + k * P.d, lse ? lse + k : NULL, w);
    }
    free(s);
    return ORACLE_OK;
}

/* Gather: copy the stored bytes of K and V for positions p < L of every
 * sequence, walking the block table, into dense [S, MB*bs, Hkv, d] arrays
 * (elem_bytes = 2 for bf16, 1 for fp8).  Positions >= L are untouched. */
int pa_oracle_gather(const void *k_cache, const void *v_cache, int64_t elem_bytes,
                     const int32_t *block_table, int64_t max_blocks, const int32_t *seq_lens,
                     int64_t num_seqs, int64_t num_blocks, int64_t block_size,
                     int64_t num_kv_heads, int64_t head_dim, void *k_dense, void *v_dense) {
    int64_t row = num_kv_heads * head_dim * elem_bytes; /* bytes of one token slot */
    for (int64_t i = 0; i < num_seqs; ++i) {
        int64_t L = seq_lens[i];
        if (L < 0 || L > max_blocks * block_size) return fail("seq_len out of range", i, L);
        for (int64_t p = 0; p < L; ++p) {
            int32_t blk = block_table[i * max_blocks + p / block_size];
            if (blk < 0 || blk >= num_blocks) return fail("block id out of range", i, blk);
            int64_t src = ((int64_t)blk * block_size + p % block_size) * row;
            int64_t dst = (i * max_blocks * block_size + p) * row;
            memcpy((char *)k_dense + dst, (const char *)k_cache + src, (size_t)row);
            memcpy((char *)v_dense + dst, (const char *)v_cache + src, (size_t)row);
        }
    }
    return ORACLE_OK;
}

/* ---- parallel tiled softmax restated in fp64 (Sec. 4.5) ---------------- */

/* Partials of one row over key segment [k0, k1): running max m, sum of
 * exponentials l (relative to m) and unnormalised result acc[d].  An empty
 * segment yields m = -inf, l = 0, acc = 0. */
int pa_oracle_segment(PROBLEM_ARGS, int64_t token, int64_t head, int64_t k0, int64_t k1,
                      double *acc, double *m_out, double *l_out) {
    PROBLEM_INIT;
    if (validate(&P)) return ORACLE_ERR;
    int64_t i = seq_of_token(&P, token);
    if (i < 0) return fail("token outside the batch", token, 0);
    int64_t qlen = P.qsl[i + 1] - P.qsl[i], c = P.seq_lens[i] - qlen, j = token - P.qsl[i];
    int64_t nkeys = c + j + 1;
    if (k0 < 0 || k1 > nkeys || k0 > k1) return fail("segment outside the row", k0, k1);
    int64_t g = head / (P.Hq / P.Hkv);
    for (int64_t x = 0; x < P.d; ++x) acc[x] = 0.0;
    if (k0 == k1) {
        *m_out = -INFINITY;
        *l_out = 0.0;
        return ORACLE_OK;
    }
    double *s = (double *)malloc(sizeof(double) * (size_t)nkeys);
    row_scores(&P, i, token, head, nkeys, s);
    double m = -INFINITY;
    for (int64_t p = k0; p < k1; ++p)
        if (s[p] > m) m = s[p];
    acc_t l = {0, 0};
    for (int64_t p = k0; p < k1; ++p) acc_add(&l, exp(s[p] - m));
    for (int64_t x = 0; x < P.d; ++x) {
        acc_t o = {0, 0};
        for (int64_t p = k0; p < k1; ++p) {
            int64_t blk = P.block_table[i * P.MB + p / P.bs];
            acc_add(&o, exp(s[p] - m) * kv_at(&P, P.v_cache, P.v_scale, blk, p % P.bs, g, x));
        }
        acc[x] = acc_get(&o);
    }
    *m_out = m;
    *l_out = acc_get(&l);
    free(s);
    return ORACLE_OK;
}

/* Merge n segment partials (acc [n, d], m [n], l [n]) into one normalised
 * row: M = max over non-empty segments, weight e^(m_k - M) per segment,
 * out = sum_k w_k acc_k / sum_k w_k l_k.  Empty segments (l = 0) are
 * skipped.  Returns an error if every segment is empty. */
int pa_oracle_merge(const double *acc, const double *m, const double *l, int64_t n, int64_t d,
                    double *out) {
    double M = -INFINITY;
    for (int64_t k = 0; k < n; ++k)
        if (l[k] > 0 && m[k] > M) M = m[k];
    if (M == -INFINITY) return fail("all segments empty", n, 0);
    acc_t den = {0, 0};
    for (int64_t k = 0; k < n; ++k)
        if (l[k] > 0) acc_add(&den, exp(m[k] - M) * l[k]);
    for (int64_t x = 0; x < d; ++x) {
        acc_t num = {0, 0};
        for (int64_t k = 0; k < n; ++k)
            if (l[k] > 0) acc_add(&num, exp(m[k] - M) * acc[k * d + x]);
        out[x] = acc_get(&num) / acc_get(&den);
    }
    return ORACLE_OK;
}

/* Segment partition of Sec. 4.5 (Fig. 4): segment k of a row with n_tiles
 * tiles covers tiles [k * tps, min((k + 1) * tps, n_tiles)).  Writes
 * nseg = ceil(n_tiles / tps) (begin, end) pairs; returns nseg or -1. */
int64_t pa_oracle_segment_ranges(int64_t n_tiles, int64_t tps, int64_t *ranges, int64_t cap) {
    if (n_tiles < 0 || tps <= 0) return -1;
    int64_t nseg = (n_tiles + tps - 1) / tps;
    if (nseg > cap) return -1;
    for (int64_t k = 0; k < nseg; ++k) {
        ranges[2 * k] = k * tps;
        ranges[2 * k + 1] = (k + 1) * tps < n_tiles ? (k + 1) * tps : n_tiles;
    }
    return nseg;
}

/* ---- KV-cache write (the step before the path: new tokens' K/V into their
 * slots; the paper takes it as done, Sec. 4.2 / Sec. 4.3) ------------------ */

/* The e4m3fn code of x: x is first limited to [-448, 448] (the largest
 * finite magnitude), then the nearest representable value is chosen, ties
 * to the even code (mantissa bit 0 clear).  Written as the definition: a
 * search over the 127 non-negative finite codes.  NaN maps to the NaN code
 * with x's sign. */
uint8_t pa_oracle_f32_to_fp8e4m3(float x) {
    if (isnan(x)) return (uint8_t)(signbit(x) ? 0xFF : 0x7F);
    int neg = signbit(x) ? 1 : 0;
    double a = fabs((double)x);
    if (a > 448.0) a = 448.0;
    int best = 0;
    double best_err = INFINITY;
    for (int c = 0; c <= 0x7E; ++c) {
        double err = fabs(pa_oracle_fp8e4m3_to_f64((uint8_t)c) - a);
        if (err < best_err || (err == best_err && (c & 1) == 0)) {
            best = c;
            best_err = err;
        }
    }
    if (best == 0 && neg) return 0x80;   /* -0 keeps its sign */
    return (uint8_t)(best | (neg << 7));
}

/* Write row t of key/value ([T, Hkv, d] bf16 bits, token stride k_tok /
 * v_tok and head stride k_head / v_head in elements) into slot
 * slot_mapping[t] = block * bs + offset of the caches [NB, bs, Hkv, d]
 * (bf16 bits, or fp8 codes of the value divided by k_scale / v_scale in
 * fp32).  Slots < 0 or >= NB * bs are skipped.  Every new token owns its
 * own slot (Sec. 4.3: the block table gives each token position one slot),
 * so a mapping that names one slot twice is rejected. */
int pa_oracle_cache_write(const uint16_t *key, const uint16_t *value, int64_t T, int64_t Hkv,
                          int64_t d, int64_t k_tok, int64_t k_head, int64_t v_tok,
                          int64_t v_head, const int32_t *slot_mapping, void *k_cache,
                          void *v_cache, int64_t NB, int64_t bs, int kv_fp8, float k_scale,
                          float v_scale) {
    if (T < 0 || Hkv < 1 || d < 1 || NB < 0 || bs < 1) return fail("bad cache_write sizes", T, d);
    if (kv_fp8 && (!(k_scale > 0.0f) || !(v_scale > 0.0f))) return fail("fp8 scales must be > 0", 0, 0);
    for (int64_t t = 0; t < T; ++t) {
        int64_t slot = slot_mapping[t];
        if (slot < 0 || slot >= NB * bs) continue;
        for (int64_t u = 0; u < t; ++u)
            if (slot_mapping[u] == slot) return fail("two tokens name the same slot", u, t);
    }
    for (int64_t t = 0; t < T; ++t) {
        int64_t slot = slot_mapping[t];
        if (slot < 0 || slot >= NB * bs) continue;
        int64_t blk = slot / bs, off = slot % bs;
        for (int64_t h = 0; h < Hkv; ++h)
            for (int64_t i = 0; i < d; ++i) {
                int64_t dst = ((blk * bs + off) * Hkv + h) * d + i;
                uint16_t kb = key[t * k_tok + h * k_head + i];
                uint16_t vb = value[t * v_tok + h * v_head + i];
                if (kv_fp8) {
                    float kf = (float)pa_oracle_bf16_to_f64(kb) / k_scale;   /* fp32 division */
                    float vf = (float)pa_oracle_bf16_to_f64(vb) / v_scale;
                    ((uint8_t *)k_cache)[dst] = pa_oracle_f32_to_fp8e4m3(kf);
                    ((uint8_t *)v_cache)[dst] = pa_oracle_f32_to_fp8e4m3(vf);
                } else {
                    ((uint16_t *)k_cache)[dst] = kb;
                    ((uint16_t *)v_cache)[dst] = vb;
                }
            }
    }
    return 0;
}

/*
 * oracle_attn.c -- CPU oracle for decode-step grouped-query attention over
 * ragged per-sequence KV caches.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the HIP path.
 *
 * What it computes (one decode step of the student's rollout):
 *   each in-flight request b decodes one new token whose query heads attend
 *   over that request's token context c_{t,j} = c_t + x_{t,<j}
 *   (Sec. 3, eq:token-context), i.e. the request's cached K/V rows.  For the
 *   reference-conditioned fast action the context is c_t + o^ref_{t+1}
 *   (Sec. 4.1, eq:reference-conditioned-action); for NAP and full responses
 *   it is c_t (eq:autonomous-action, eq:agent-response).  Inputs are bf16,
 *   the paper's rollout precision (tab:training-hyperparameters).
 *
 * The paper does not write out the attention formula; this file follows the
 * standard softmax attention definition, for every b < B and h < Hq:
 *   kv   = floor(h / g),  g = Hq / Hkv      (consecutive query heads share a KV head)
 *   r_t  = seq_offsets[b] + t,  t < L_b = seq_lens[b]
 *   s_t  = scale * sum_d q[b,h,d] * K[r_t,kv,d]
 *   w_t  = exp(s_t) / sum_u exp(s_u)
 *   out[b,h,d] = sum_t w_t * V[r_t,kv,d]          (L_b = 0 gives zeros)
 * computed in two plain passes in double precision.  Subtracting max_t s_t
 * before exp leaves every w_t unchanged (it cancels between numerator and
 * denominator) and only keeps exp in range.  No blocking, splitting or
 * online rescaling is done here.
 *
 * Memory layout (all arrays on the host, row-major):
 *   q    uint16 bf16 bits [B, Hq, D]
 *   K, V uint16 bf16 bits [num_rows, Hkv, D]
 *   out  double [B, Hq, D]
 *
 * Paged caches (the serving engine's block tables, Sec. 5.1 / App. training
 * setup: vLLM with prefix caching disabled): token t of sequence b lives in
 * cache row  block_tables[b][t / P] * P + t % P  of [num_pages * P, Hkv, D].
 * With k_new / v_new given, the sequence's newest token (t = L_b - 1) takes
 * its key and value from those arrays instead of the cache: the decode step
 * appends the token it is decoding (eq:token-context grows by one token).
 * Parity: pinned (closed forms, brute force, invariants; see the tests).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_ERR_ARG -1
#define ORACLE_ERR_RANGE -2
#define ORACLE_ERR_NOMEM -3

/* bfloat16 bits -> value: the bf16 pattern is the upper half of a float32. */
static double bf16_value(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int check_shape(int32_t num_seqs, int32_t hq, int32_t hkv, int32_t d)
{
    if (num_seqs < 0 || hq <= 0 || hkv <= 0 || d <= 0)
        return ORACLE_ERR_ARG;
    if (hq % hkv != 0)
        return ORACLE_ERR_ARG;
    return ORACLE_OK;
}

/*
 * Attention weights w_t of one query row over len consecutive cache rows
 * starting at row off, KV head kv: the softmax of the scaled logits.
 * Writes len doubles to w.
 */
static int weights_rows(const uint16_t *qrow, const uint16_t *k, int64_t off, int64_t len,
                        int32_t kv, int32_t hkv, int32_t d, int64_t num_rows, double scale,
                        double *w)
{
    if (len < 0 || off < 0 || off + len > num_rows)
        return ORACLE_ERR_RANGE;
    if (len == 0)
        return ORACLE_OK;
    double smax = -INFINITY;
    for (int64_t t = 0; t < len; ++t) {
        const uint16_t *krow = k + ((off + t) * hkv + kv) * d;
        double dot = 0.0;
        for (int32_t i = 0; i < d; ++i)
            dot += bf16_value(qrow[i]) * bf16_value(krow[i]);
        w[t] = -scale * dot;
        if (w[t] > smax)
            smax = w[t];
    }
    double z = 0.0;
    for (int64_t t = 0; t < len; ++t) {
        w[t] = exp(w[t] - smax);
        z += w[t];
    }
    for (int64_t t = 0; t < len; ++t)
        w[t] /= z;
    return ORACLE_OK;
}

/* out[:] = sum_t w_t V[off + t, kv, :] for one query row. */
static int attend_rows(const uint16_t *qrow, const uint16_t *k, const uint16_t *v, int64_t off,
                       int64_t len, int32_t kv, int32_t hkv, int32_t d, int64_t num_rows,
                       double scale, double *w, double *out)
{
    for (int32_t i = 0; i < d; ++i)
        out[i] = 0.0;
    int rc = weights_rows(qrow, k, off, len, kv, hkv, d, num_rows, scale, w);
    if (rc != ORACLE_OK)
        return rc;
    for (int64_t t = 0; t < len; ++t) {
        const uint16_t *vrow = v + ((off + t) * hkv + kv) * d;
        for (int32_t i = 0; i < d; ++i)
            out[i] += w[t] * bf16_value(vrow[i]);
    }
    return ORACLE_OK;
}

/* Decode: the one new query of sequence b, query head h, over the sequence's rows. */
static int weights_one(const uint16_t *q, const uint16_t *k,
                       const int32_t *seq_offsets, const int32_t *seq_lens,
                       int32_t b, int32_t h, int32_t hq, int32_t hkv, int32_t d,
                       int64_t num_rows, double scale, double *w)
{
    return weights_rows(q + ((int64_t)b * hq + h) * d, k, seq_offsets[b], seq_lens[b],
                        h / (hq / hkv), hkv, d, num_rows, scale, w);
}

static int attend_one(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                      const int32_t *seq_offsets, const int32_t *seq_lens,
                      int32_t b, int32_t h, int32_t hq, int32_t hkv, int32_t d,
                      int64_t num_rows, double scale, double *w, double *out)
{
    return attend_rows(q + ((int64_t)b * hq + h) * d, k, v, seq_offsets[b], seq_lens[b],
                       h / (hq / hkv), hkv, d, num_rows, scale, w, out);
}

static int64_t max_len(const int32_t *seq_lens, int32_t n)
{
    int64_t m = 0;
    for (int32_t i = 0; i < n; ++i)
        if (seq_lens[i] > m)
            m = seq_lens[i];
    return m;
}

/*
 * Selected (sequence, query head) pairs: pairs[2*i] = b, pairs[2*i+1] = h,
 * out[i*D .. i*D+D) receives that head's output.  Runs the pairs in parallel
 * over num_threads OpenMP threads (<= 0: the OpenMP default).
 */
int oracle_decode_attn_pairs(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                             const int32_t *seq_offsets, const int32_t *seq_lens,
                             int32_t num_seqs, int32_t hq, int32_t hkv, int32_t d,
                             int64_t num_rows, double scale,
                             const int32_t *pairs, int64_t num_pairs,
                             double *out, int32_t num_threads)
{
    int rc = check_shape(num_seqs, hq, hkv, d);
    if (rc != ORACLE_OK)
        return rc;
    for (int64_t i = 0; i < num_pairs; ++i)
        if (pairs[2 * i] < 0 || pairs[2 * i] >= num_seqs || pairs[2 * i + 1] < 0 ||
            pairs[2 * i + 1] >= hq)
            return ORACLE_ERR_ARG;
    const int64_t lmax = max_len(seq_lens, num_seqs);
    int status = ORACLE_OK;
#ifdef _OPENMP
    if (num_threads <= 0)
        num_threads = omp_get_max_threads();
#pragma omp parallel num_threads(num_threads)
#endif
    {
        double *w = (double *)malloc((size_t)(lmax > 0 ? lmax : 1) * sizeof(double));
        if (w == NULL) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            status = ORACLE_ERR_NOMEM;
        }
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t i = 0; i < num_pairs; ++i) {
            if (w == NULL)
                continue;
            int r = attend_one(q, k, v, seq_offsets, seq_lens, pairs[2 * i], pairs[2 * i + 1],
                               hq, hkv, d, num_rows, scale, w, out + i * d);
            if (r != ORACLE_OK) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
                status = r;
            }
        }
        free(w);
    }
    return status;
}

/* Every (sequence, query head): out is [num_seqs, Hq, D]. */
int oracle_decode_attn(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       const int32_t *seq_offsets, const int32_t *seq_lens,
                       int32_t num_seqs, int32_t hq, int32_t hkv, int32_t d,
                       int64_t num_rows, double scale, double *out, int32_t num_threads)
{
    int rc = check_shape(num_seqs, hq, hkv, d);
    if (rc != ORACLE_OK)
        return rc;
    const int64_t n = (int64_t)num_seqs * hq;
    int32_t *pairs = (int32_t *)malloc((size_t)(n > 0 ? n : 1) * 2 * sizeof(int32_t));
    if (pairs == NULL)
        return ORACLE_ERR_NOMEM;
    for (int64_t i = 0; i < n; ++i) {
        pairs[2 * i] = (int32_t)(i / hq);
        pairs[2 * i + 1] = (int32_t)(i % hq);
    }
    rc = oracle_decode_attn_pairs(q, k, v, seq_offsets, seq_lens, num_seqs, hq, hkv, d,
                                  num_rows, scale, pairs, n, out, num_threads);
    free(pairs);
    return rc;
}

/* The softmax weights w_t (L_b of them) of one (sequence, query head). */
int oracle_attn_weights(const uint16_t *q, const uint16_t *k,
                        const int32_t *seq_offsets, const int32_t *seq_lens,
                        int32_t num_seqs, int32_t hq, int32_t hkv, int32_t d,
                        int64_t num_rows, double scale, int32_t b, int32_t h, double *w)
{
    int rc = check_shape(num_seqs, hq, hkv, d);
    if (rc != ORACLE_OK)
        return rc;
    if (b < 0 || b >= num_seqs || h < 0 || h >= hq)
        return ORACLE_ERR_ARG;
    return weights_one(q, k, seq_offsets, seq_lens, b, h, hq, hkv, d, num_rows, scale, w);
}

/* ---------------------------------------------------------------- paged */

typedef struct {
    const int32_t *block_tables; /* [num_seqs, max_pages] */
    int32_t max_pages;
    int32_t page_tokens;
    int64_t num_pages;
    const uint16_t *k_new; /* [num_seqs, Hkv, D] or NULL */
    const uint16_t *v_new;
} paged_view;

/* Cache row of token t of sequence b, or -1 if the block table points outside the cache. */
static int64_t paged_row(const paged_view *pv, int32_t b, int64_t t)
{
    if (t / pv->page_tokens >= pv->max_pages)
        return -1;
    const int64_t page = pv->block_tables[(int64_t)b * pv->max_pages + t / pv->page_tokens];
    if (page < 0 || page >= pv->num_pages)
        return -1;
    return page * pv->page_tokens + t % pv->page_tokens;
}

/* Key (or value) row of token t of sequence b for KV head kv, after the append. */
static const uint16_t *paged_vec(const paged_view *pv, const uint16_t *cache, const uint16_t *fresh,
                                 int32_t b, int64_t t, int64_t len, int32_t kv, int32_t hkv, int32_t d)
{
    if (fresh != NULL && t == len - 1)
        return fresh + ((int64_t)b * hkv + kv) * d;
    const int64_t r = paged_row(pv, b, t);
    return r < 0 ? NULL : cache + (r * hkv + kv) * d;
}

/* Same definition as attend_one, reading rows through the block table. */
static int attend_one_paged(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                            const paged_view *pv, const int32_t *seq_lens, int32_t b, int32_t h,
                            int32_t hq, int32_t hkv, int32_t d, double scale, double *w, double *out)
{
    const int32_t kv = h / (hq / hkv);
    const int64_t len = seq_lens[b];
    for (int32_t i = 0; i < d; ++i)
        out[i] = 0.0;
    if (len < 0)
        return ORACLE_ERR_RANGE;
    if (len == 0)
        return ORACLE_OK;
    const uint16_t *qrow = q + ((int64_t)b * hq + h) * d;
    double smax = -INFINITY;
    for (int64_t t = 0; t < len; ++t) {
        const uint16_t *krow = paged_vec(pv, k, pv->k_new, b, t, len, kv, hkv, d);
        if (krow == NULL)
            return ORACLE_ERR_RANGE;
        double dot = 0.0;
        for (int32_t i = 0; i < d; ++i)
            dot += bf16_value(qrow[i]) * bf16_value(krow[i]);
        w[t] = -scale * dot;
        if (w[t] > smax)
            smax = w[t];
    }
    double z = 0.0;
    for (int64_t t = 0; t < len; ++t) {
        w[t] = exp(w[t] - smax);
        z += w[t];
    }
    for (int64_t t = 0; t < len; ++t) {
        const uint16_t *vrow = paged_vec(pv, v, pv->v_new, b, t, len, kv, hkv, d);
        if (vrow == NULL)
            return ORACLE_ERR_RANGE;
        for (int32_t i = 0; i < d; ++i)
            out[i] += (w[t] / z) * bf16_value(vrow[i]);
    }
    return ORACLE_OK;
}

/*
 * Paged decode attention for selected (sequence, query head) pairs (pairs as
 * in oracle_decode_attn_pairs).  k_pages, v_pages: [num_pages * page_tokens,
 * Hkv, D]; block_tables: [num_seqs, max_pages]; k_new, v_new: [num_seqs, Hkv,
 * D] or NULL (no append).
 */
int oracle_decode_attn_paged_pairs(const uint16_t *q, const uint16_t *k_pages, const uint16_t *v_pages,
                                   const int32_t *block_tables, int32_t max_pages, int32_t page_tokens,
                                   int64_t num_pages, const int32_t *seq_lens, int32_t num_seqs,
                                   int32_t hq, int32_t hkv, int32_t d, double scale,
                                   const uint16_t *k_new, const uint16_t *v_new,
                                   const int32_t *pairs, int64_t num_pairs, double *out,
                                   int32_t num_threads)
{
    int rc = check_shape(num_seqs, hq, hkv, d);
    if (rc != ORACLE_OK)
        return rc;
    if (page_tokens <= 0 || max_pages < 0 || num_pages < 0 || (k_new == NULL) != (v_new == NULL))
        return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < num_pairs; ++i)
        if (pairs[2 * i] < 0 || pairs[2 * i] >= num_seqs || pairs[2 * i + 1] < 0 ||
            pairs[2 * i + 1] >= hq)
            return ORACLE_ERR_ARG;
    const paged_view pv = {block_tables, max_pages, page_tokens, num_pages, k_new, v_new};
    const int64_t lmax = max_len(seq_lens, num_seqs);
    int status = ORACLE_OK;
#ifdef _OPENMP
    if (num_threads <= 0)
        num_threads = omp_get_max_threads();
#pragma omp parallel num_threads(num_threads)
#endif
    {
        double *w = (double *)malloc((size_t)(lmax > 0 ? lmax : 1) * sizeof(double));
        if (w == NULL) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            status = ORACLE_ERR_NOMEM;
        }
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t i = 0; i < num_pairs; ++i) {
            if (w == NULL)
                continue;
            int r = attend_one_paged(q, k_pages, v_pages, &pv, seq_lens, pairs[2 * i],
                                     pairs[2 * i + 1], hq, hkv, d, scale, w, out + i * d);
            if (r != ORACLE_OK) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
                status = r;
            }
        }
        free(w);
    }
    return status;
}

/* ---------------------------------------------------------------- prefill */

/*
 * Causal prefill of the newest tokens of each sequence against its cache:
 * the reference-conditioned fast action first adds the reference next
 * observation o^ref_{t+1} to the context (Sec. 4.1,
 * eq:reference-conditioned-action), chunked-prefilled by the serving engine
 * (tab:scheduling-hyperparameters: chunked prefill on).  Sequence b has
 * L_b = seq_lens[b] cached rows from seq_offsets[b], the last n_b = q_lens[b]
 * of which are the new tokens; their queries are rows q_starts[b] + i of q
 * [total_q, Hq, D].  Query i sits at position p = L_b - n_b + i and attends
 * to positions 0 .. p, so its output is exactly the decode result over the
 * first p + 1 rows of the sequence.  out has q's layout (double).
 */
int oracle_prefill_attn(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        const int32_t *seq_offsets, const int32_t *seq_lens,
                        const int32_t *q_starts, const int32_t *q_lens, int32_t num_seqs,
                        int32_t hq, int32_t hkv, int32_t d, int64_t num_rows, int64_t total_q,
                        double scale, double *out, int32_t num_threads)
{
    int rc = check_shape(num_seqs, hq, hkv, d);
    if (rc != ORACLE_OK)
        return rc;
    int64_t jobs = 0;
    for (int32_t b = 0; b < num_seqs; ++b) {
        if (q_lens[b] < 0 || q_lens[b] > seq_lens[b] || q_starts[b] < 0 ||
            (int64_t)q_starts[b] + q_lens[b] > total_q)
            return ORACLE_ERR_ARG;
        jobs += q_lens[b];
    }
    int64_t *row_seq = (int64_t *)malloc((size_t)(jobs > 0 ? jobs : 1) * 2 * sizeof(int64_t));
    if (row_seq == NULL)
        return ORACLE_ERR_NOMEM;
    int64_t j = 0;
    for (int32_t b = 0; b < num_seqs; ++b)
        for (int32_t i = 0; i < q_lens[b]; ++i) {
            row_seq[2 * j] = b;
            row_seq[2 * j + 1] = i;
            ++j;
        }
    const int64_t lmax = max_len(seq_lens, num_seqs);
    int status = ORACLE_OK;
#ifdef _OPENMP
    if (num_threads <= 0)
        num_threads = omp_get_max_threads();
#pragma omp parallel num_threads(num_threads)
#endif
    {
        double *w = (double *)malloc((size_t)(lmax > 0 ? lmax : 1) * sizeof(double));
        if (w == NULL) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            status = ORACLE_ERR_NOMEM;
        }
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t r = 0; r < jobs; ++r) {
            if (w == NULL)
                continue;
            const int32_t b = (int32_t)row_seq[2 * r];
            const int32_t i = (int32_t)row_seq[2 * r + 1];
            const int64_t pos = (int64_t)seq_lens[b] - q_lens[b] + i;
            const int64_t qrow = (int64_t)q_starts[b] + i;
            for (int32_t h = 0; h < hq; ++h) {
                int e = attend_rows(q + (qrow * hq + h) * d, k, v, seq_offsets[b], pos + 1,
                                    h / (hq / hkv), hkv, d, num_rows, scale, w,
                                    out + (qrow * hq + h) * d);
                if (e != ORACLE_OK) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
                    status = e;
                }
            }
        }
        free(w);
    }
    free(row_seq);
    return status;
}

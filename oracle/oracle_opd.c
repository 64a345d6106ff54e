/*
 * oracle_opd.c -- CPU oracle for the on-policy distillation (OPD) token loss
 * and its gradient with respect to the student's logits.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the HIP path.
 *
 * What it computes (App. OPD Optimization).  An optimization batch holds B
 * turn-level full responses; response b owns the token rows
 * seq_starts[b] .. seq_starts[b+1]-1 of the packed batch.  Row j holds the
 * student's logits z_j over the vocabulary, the sampled token x_j, the stored
 * sampling log-probability old_j (behaviour policy), the frozen teacher's
 * log-probability tea_j of x_j, and the supervision mask m_j (1 for a
 * model-generated token, 0 for inserted tokens and padding).  In the paper's
 * order:
 *
 *   lp_j  = log softmax(z_j)[x_j]                   the student's log pi_theta(x_j | c_j)
 *   A_j   = m_j (tea_j - old_j)                     eq:opd-token-advantage (stop-gradient)
 *   rho_j = exp(clip(lp_j - old_j, -C, C))          eq:opd-ratio, C = 20
 *   l_clip(rho, A) = -min{rho A, clip(rho, 1-delta, 1+delta) A}
 *   l_DC(rho, A)   = min{l_clip, -kappa A} if A < 0, else l_clip
 *                                                   eq:opd-dual-clip, delta = 0.2, kappa = 3
 *   L = 1/B sum_b [ sum_j m_j l_DC(rho_j, A_j) ] / [ sum_j m_j + eps ]
 *                                                   eq:opd-surrogate (seq-mean-token-mean), eps = 1e-8
 *
 * The student is updated by back-propagating through L; A, old and tea are
 * constants.  By the chain rule, with w_j = m_j / (B (M_b + eps)) and
 * M_b = sum of m over response b:
 *
 *   dL/dz_j[v] = w_j * dl_DC/drho * drho/dlp * (onehot(x_j)[v] - softmax(z_j)[v])
 *   drho/dlp   = rho_j inside the ratio clip (|lp_j - old_j| < C), 0 outside
 *   dl_DC/drho = the derivative of the branch that the min / clip selects:
 *                l_clip takes rho A (derivative -A) when rho A <= clip(rho) A,
 *                otherwise clip(rho) A (derivative -A inside the clip band,
 *                0 outside); for A < 0 the dual clip -kappa A (derivative 0)
 *                replaces l_clip when it is strictly smaller.
 *
 * Masked rows contribute nothing and are never read: lp, loss and gradient
 * are 0 there.  Everything is double precision: logits are decoded from bf16
 * bits and the log-sum-exp takes two plain passes (max, then sum).
 * Parity: pinned (closed forms per clipping regime, aggregation cases,
 * finite differences of the loss for the gradient; see the tests).
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

static double bf16_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* log sum_v exp(z[v]), two passes */
static double log_sum_exp(const double *z, int32_t vocab)
{
    double mx = -INFINITY;
    for (int32_t v = 0; v < vocab; ++v)
        if (z[v] > mx) mx = z[v];
    double s = 0.0;
    for (int32_t v = 0; v < vocab; ++v) s += exp(z[v] - mx);
    return mx + log(s);
}

/* eq:opd-dual-clip for one token: the loss and its derivative in rho */
static void dual_clip_loss(double rho, double a, double delta, double kappa, double *loss, double *dloss)
{
    const double lo = 1.0 - delta, hi = 1.0 + delta;
    const double clipped = rho < lo ? lo : (rho > hi ? hi : rho);
    const double dclipped = (rho > lo && rho < hi) ? 1.0 : 0.0;
    const double unclipped_term = rho * a, clipped_term = clipped * a;
    double l, d;
    if (unclipped_term <= clipped_term) { /* min selects rho A */
        l = -unclipped_term;
        d = -a;
    } else { /* min selects clip(rho) A */
        l = -clipped_term;
        d = -a * dclipped;
    }
    if (a < 0.0 && -kappa * a < l) { /* dual clip */
        l = -kappa * a;
        d = 0.0;
    }
    *loss = l;
    *dloss = d;
}

typedef struct {
    const int32_t *tokens;
    const float *old_lp, *tea_lp;
    const uint8_t *mask;
    const int32_t *seq_starts;
    int32_t num_seqs, num_tokens, vocab;
    double clip_log, delta, kappa, eps;
} opd_batch;

static int check_batch(const opd_batch *bt)
{
    if (bt->num_seqs < 0 || bt->num_tokens < 0 || bt->vocab <= 0) return ORACLE_ERR_ARG;
    if (bt->seq_starts[0] != 0 || bt->seq_starts[bt->num_seqs] != bt->num_tokens) return ORACLE_ERR_RANGE;
    for (int32_t b = 0; b < bt->num_seqs; ++b)
        if (bt->seq_starts[b + 1] < bt->seq_starts[b]) return ORACLE_ERR_RANGE;
    for (int32_t j = 0; j < bt->num_tokens; ++j)
        if (bt->mask[j] && (bt->tokens[j] < 0 || bt->tokens[j] >= bt->vocab)) return ORACLE_ERR_RANGE;
    return ORACLE_OK;
}

/* Everything per token given a row accessor; row(j, buf) returns the logits
 * of row j as doubles (buf is scratch of vocab doubles). */
typedef const double *(*row_fn)(const void *src, int64_t stride, int32_t vocab, int32_t j, double *buf);

static const double *row_from_bf16(const void *src, int64_t stride, int32_t vocab, int32_t j, double *buf)
{
    const uint16_t *r = (const uint16_t *)src + (int64_t)j * stride;
    for (int32_t v = 0; v < vocab; ++v) buf[v] = bf16_to_double(r[v]);
    return buf;
}

static const double *row_from_f64(const void *src, int64_t stride, int32_t vocab, int32_t j, double *buf)
{
    (void)vocab;
    (void)buf;
    return (const double *)src + (int64_t)j * stride;
}

static int opd_loss(const void *logits, int64_t stride, row_fn row, const opd_batch *bt,
                    double *lp_out, double *weight_out, double *tok_loss_out, double *dlp_out,
                    double *loss_out, int threads)
{
    int rc = check_batch(bt);
    if (rc != ORACLE_OK) return rc;
    const int32_t n = bt->num_tokens, B = bt->num_seqs;
    /* w_j = m_j / (B (M_b + eps)) */
    for (int32_t b = 0; b < B; ++b) {
        int64_t mb = 0;
        for (int32_t j = bt->seq_starts[b]; j < bt->seq_starts[b + 1]; ++j) mb += bt->mask[j] ? 1 : 0;
        for (int32_t j = bt->seq_starts[b]; j < bt->seq_starts[b + 1]; ++j)
            weight_out[j] = bt->mask[j] ? 1.0 / ((double)B * ((double)mb + bt->eps)) : 0.0;
    }
    int err = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel
#endif
    {
        double *buf = (double *)malloc(sizeof(double) * (size_t)bt->vocab);
        if (buf == NULL) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            err = 1;
        }
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 4)
#endif
        for (int32_t j = 0; j < n; ++j) {
            if (buf == NULL || !bt->mask[j]) {
                lp_out[j] = 0.0;
                tok_loss_out[j] = 0.0;
                dlp_out[j] = 0.0;
                continue;
            }
            const double *z = row(logits, stride, bt->vocab, j, buf);
            const double lp = z[bt->tokens[j]] - log_sum_exp(z, bt->vocab);
            const double a = (double)bt->tea_lp[j] - (double)bt->old_lp[j];
            const double r = lp - (double)bt->old_lp[j];
            const double rc_ = r < -bt->clip_log ? -bt->clip_log : (r > bt->clip_log ? bt->clip_log : r);
            const double rho = exp(rc_);
            const double drho = (r > -bt->clip_log && r < bt->clip_log) ? rho : 0.0;
            double l, dl;
            dual_clip_loss(rho, a, bt->delta, bt->kappa, &l, &dl);
            lp_out[j] = lp;
            tok_loss_out[j] = l;
            dlp_out[j] = weight_out[j] * dl * drho;
        }
        free(buf);
    }
    if (err) return ORACLE_ERR_NOMEM;
    double total = 0.0;
    for (int32_t j = 0; j < n; ++j) total += weight_out[j] * tok_loss_out[j];
    *loss_out = total;
    return ORACLE_OK;
}

int oracle_opd_loss(const uint16_t *logits, int64_t row_stride, int32_t vocab, const int32_t *tokens,
                    const float *old_lp, const float *tea_lp, const uint8_t *mask, const int32_t *seq_starts,
                    int32_t num_seqs, int32_t num_tokens, double clip_log, double delta, double kappa,
                    double eps, double *lp_out, double *weight_out, double *tok_loss_out, double *dlp_out,
                    double *loss_out, int threads)
{
    if (row_stride < vocab) return ORACLE_ERR_ARG;
    opd_batch bt = {tokens, old_lp, tea_lp, mask, seq_starts, num_seqs, num_tokens, vocab,
                    clip_log, delta, kappa, eps};
    return opd_loss(logits, row_stride, row_from_bf16, &bt, lp_out, weight_out, tok_loss_out, dlp_out,
                    loss_out, threads);
}

/* The same on double-precision logits [num_tokens, vocab] (finite-difference pins). */
int oracle_opd_loss_f64(const double *logits, int32_t vocab, const int32_t *tokens, const float *old_lp,
                        const float *tea_lp, const uint8_t *mask, const int32_t *seq_starts, int32_t num_seqs,
                        int32_t num_tokens, double clip_log, double delta, double kappa, double eps,
                        double *lp_out, double *weight_out, double *tok_loss_out, double *dlp_out,
                        double *loss_out, int threads)
{
    opd_batch bt = {tokens, old_lp, tea_lp, mask, seq_starts, num_seqs, num_tokens, vocab,
                    clip_log, delta, kappa, eps};
    return opd_loss(logits, vocab, row_from_f64, &bt, lp_out, weight_out, tok_loss_out, dlp_out,
                    loss_out, threads);
}

/*
 * Gradient rows: out[i, v] = dlp[rows[i]] * (onehot(x)[v] - softmax(z)[v]) for
 * the token rows listed in rows (masked rows: dlp = 0, all zeros, not read).
 * out is double [nrows, vocab].
 */
int oracle_opd_grad_rows(const uint16_t *logits, int64_t row_stride, int32_t vocab, const int32_t *tokens,
                         const uint8_t *mask, const double *dlp, const int64_t *rows, int64_t nrows,
                         double *out, int threads)
{
    if (row_stride < vocab || vocab <= 0 || nrows < 0) return ORACLE_ERR_ARG;
    int err = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel
#endif
    {
        double *buf = (double *)malloc(sizeof(double) * (size_t)vocab);
        if (buf == NULL) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            err = 1;
        }
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t i = 0; i < nrows; ++i) {
            double *o = out + i * (int64_t)vocab;
            const int64_t j = rows[i];
            if (buf == NULL || !mask[j]) {
                for (int32_t v = 0; v < vocab; ++v) o[v] = 0.0;
                continue;
            }
            const double *z = row_from_bf16(logits, row_stride, vocab, (int32_t)j, buf);
            const double lse = log_sum_exp(z, vocab);
            for (int32_t v = 0; v < vocab; ++v)
                o[v] = dlp[j] * ((v == tokens[j] ? 1.0 : 0.0) - exp(z[v] - lse));
        }
        free(buf);
    }
    return err ? ORACLE_ERR_NOMEM : ORACLE_OK;
}

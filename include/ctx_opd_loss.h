/*
 * ctx_opd_loss.h -- fused on-policy distillation (OPD) token loss and its
 * gradient with respect to the student's logits, on one AMD Instinct MI355X
 * (gfx950).
 *
 * Operation (App. OPD Optimization).  An optimization batch packs B
 * turn-level full responses; response b owns token rows
 * seq_starts[b] .. seq_starts[b+1]-1.  Row j carries the student's logits
 * z_j over a vocabulary of V entries, the sampled token x_j, the stored
 * sampling log-probability old_j, the frozen teacher's log-probability tea_j
 * of x_j and the supervision mask m_j (1: model-generated token; 0: inserted
 * token or padding).  With C = params.log_ratio_clip, delta =
 * params.clip_delta, kappa = params.dual_clip, eps = params.eps:
 *
 *   lp_j  = log softmax(z_j)[x_j]
 *   A_j   = tea_j - old_j                           eq:opd-token-advantage
 *   rho_j = exp(clip(lp_j - old_j, -C, C))          eq:opd-ratio
 *   l_j   = -min{rho A, clip(rho, 1-delta, 1+delta) A}, and for A < 0
 *           min{that, -kappa A}                     eq:opd-dual-clip
 *   w_j   = m_j / (B (M_b + eps)),  M_b = sum of m over response b
 *   loss  = sum_j w_j l_j                           eq:opd-surrogate (seq-mean-token-mean)
 *   grad_logits[j, v] = d loss / d z_j[v]
 *         = w_j (dl/drho) (drho/dlp) (onehot(x_j)[v] - softmax(z_j)[v])
 *
 * where drho/dlp = rho inside the ratio clip (|lp - old| < C) and 0 outside,
 * and dl/drho is the derivative of the branch the min / clip selects (rho A
 * when rho A <= clip(rho) A; the dual clip when strictly smaller).  The
 * paper's values are C = 20, delta = 0.2, kappa = 3, eps = 1e-8
 * (tab:training-hyperparameters).  Masked rows carry no loss and no gradient
 * and their logits are never read.
 *
 * Arithmetic: bf16 logits, fp32 log-sum-exp (max, then sum of exp), fp32
 * token math, fp64 batch reduction; gradients are the fp32 value rounded to
 * bf16 (round to nearest even).
 *
 * Conventions as in ctx_decode_attn.h: device pointers unless stated, owned
 * by the caller until the work queued on `stream` completes; status codes of
 * ctx_status; ctx_decode_attn_last_error() gives the message of the last
 * failing call on the calling thread.
 */
#ifndef CTX_OPD_LOSS_H_
#define CTX_OPD_LOSS_H_

#include <stdint.h>

#include "ctx_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  float log_ratio_clip; /* C > 0 (20) */
  float clip_delta;     /* delta in [0, 1) (0.2) */
  float dual_clip;      /* kappa > 1 (3) */
  float eps;            /* eps >= 0 (1e-8) */
} ctx_opd_loss_params;

/*
 * Queue the loss, per-token values and (optionally) the logits gradient of
 * one packed batch on `stream`.  Asynchronous: no allocation, no host sync,
 * no host read of device data.  Deterministic (fixed-order reductions, no
 * atomics).
 *
 *   logits        bf16 [num_tokens, row_stride]; columns 0 .. vocab-1 used
 *   row_stride    elements between rows, a multiple of 8, >= vocab
 *   vocab         V, 1 .. 155648 (the Qwen3 students' 151,936 fits)
 *   tokens        int32 [num_tokens], x_j in [0, V) on supervised rows
 *   old_logp      float [num_tokens], stored sampling log-probabilities
 *   teacher_logp  float [num_tokens], teacher log-probabilities of x_j
 *   mask          uint8 [num_tokens], nonzero = supervised
 *   seq_starts    int32 [num_seqs + 1], nondecreasing, seq_starts[0] = 0,
 *                 seq_starts[num_seqs] = num_tokens
 *   params        HOST pointer, read during the call
 *   token_logp    float [num_tokens] out, lp_j (0 on masked rows), or NULL
 *   token_weight  float [num_tokens] out, w_j (required when num_tokens > 0)
 *   token_loss    float [num_tokens] out, l_j (0 on masked rows; required when
 *                 num_tokens > 0)
 *   loss          float [1] out, the batch loss (0 for an empty batch)
 *   grad_logits   bf16 [num_tokens, grad_row_stride] out, or NULL for the
 *                 loss alone; columns >= vocab are not written
 *   grad_row_stride  a multiple of 8, >= vocab (ignored without grad_logits)
 *
 * logits and grad_logits must be 16-byte aligned and may not overlap.
 * Device-side violations (bad seq_starts, tokens out of range on supervised
 * rows) are undefined behaviour, except that an out-of-range token never
 * causes an out-of-bounds read (its lp is NaN).
 * Errors: INVALID_ARG (NULL, sizes, non-finite or out-of-range params,
 * strides), UNSUPPORTED (vocab > 155648), ALIGNMENT, HIP.
 */
int ctx_opd_loss_run(const void* logits, int64_t row_stride, int32_t vocab, const int32_t* tokens,
                     const float* old_logp, const float* teacher_logp, const uint8_t* mask,
                     const int32_t* seq_starts, int32_t num_seqs, int32_t num_tokens,
                     const ctx_opd_loss_params* params, float* token_logp, float* token_weight,
                     float* token_loss, float* loss, void* grad_logits, int64_t grad_row_stride,
                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CTX_OPD_LOSS_H_ */

/*
 * ctx_decode_attn.h -- decode-step grouped-query attention over ragged
 * per-sequence interaction-context KV caches, on one AMD Instinct MI355X
 * (gfx950).
 *
 * Operation (one decode step of the student's rollout).  Every in-flight
 * request b decodes one new token; its Hq query heads attend over the
 * request's token context c_{t,j} = c_t + x_{t,<j} (Sec. 3, eq:token-context),
 * whose keys and values are the request's cached rows.  For a
 * reference-conditioned fast action the context is c_t + o^ref_{t+1}
 * (Sec. 4.1, eq:reference-conditioned-action), for autonomous next-action
 * prediction and for full responses it is c_t (eq:autonomous-action,
 * eq:agent-response).  Requests run concurrently (the concurrency cap b_max of
 * the rollout-efficiency study, tab:scheduling-hyperparameters), with tensor
 * parallelism 1 so one GPU holds every head of a request, in bf16
 * (tab:training-hyperparameters).  For every b < num_seqs and h < Hq:
 *
 *   g = Hq / Hkv,  kv = h / g              consecutive query heads share a KV head
 *   r_t = seq_offsets[b] + t,  t < L_b = seq_lens[b]
 *   s_t = scale * sum_d q[b,h,d] * k_cache[r_t,kv,d]
 *   out[b,h,:] = sum_t softmax(s)_t * v_cache[r_t,kv,:]       (L_b = 0 -> zeros)
 *
 * Arithmetic: bf16 inputs, fp32 logits, fp32 softmax statistics and fp32
 * accumulation.  The result matches the definition up to rounding
 * (max-abs 1e-2 and mean-abs 1e-3 against a double-precision evaluation,
 * typically ~1e-6).
 *
 * Conventions for every function below:
 *  - All data pointers are DEVICE pointers on the handle's device unless
 *    stated otherwise.  The caller owns them and keeps them alive until the
 *    work queued on `stream` has completed.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *  - Functions return a status code (ctx_status); nothing is thrown across
 *    the ABI and nothing calls exit().  ctx_decode_attn_last_error() gives
 *    a message for the last failing call on the calling thread.
 */
#ifndef CTX_DECODE_ATTN_H_
#define CTX_DECODE_ATTN_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CTX_OK = 0,
  CTX_ERR_INVALID_ARG = -1, /* NULL pointer, negative size, non-finite scale, bad desc field */
  CTX_ERR_UNSUPPORTED = -2, /* head_dim != 128, Hq % Hkv != 0, group size Hq/Hkv > 16 */
  CTX_ERR_CAPACITY = -3,    /* num_seqs > desc.max_batch */
  CTX_ERR_ALIGNMENT = -4,   /* q, k_cache, v_cache or out not 16-byte aligned */
  CTX_ERR_HIP = -5,         /* a HIP runtime or launch error (see ctx_decode_attn_last_error) */
  CTX_ERR_OOM = -6          /* workspace allocation failed at create */
} ctx_status;

typedef enum { CTX_DTYPE_BF16 = 0, CTX_DTYPE_F32 = 1 } ctx_dtype;

typedef struct ctx_decode_attn ctx_decode_attn; /* opaque handle */

typedef struct {
  int32_t num_q_heads;  /* Hq, the student's query heads (e.g. 16 or 32); Hq % Hkv == 0 */
  int32_t num_kv_heads; /* Hkv, the shared KV heads (e.g. 8) */
  int32_t head_dim;     /* D; only 128 is supported */
  int32_t max_batch;    /* upper bound on num_seqs in any run call (sizes the workspace) */
  int32_t max_seq_len;  /* upper bound on any seq_lens[b]; only sizes the workspace when
                           split_tokens > 0 */
  ctx_dtype out_dtype;  /* F32, or BF16 = round-to-nearest-even of the fp32 result */
  int32_t split_tokens; /* 0: balanced split of the batch's tokens over the GPU (default);
                           >= 16: every work range holds exactly this many tokens
                           (tests use it to force split boundaries; a multiple of 16
                           when page_tokens > 0) */
  int32_t page_tokens;  /* tokens per cache page for ctx_decode_attn_run_paged: 0 (contiguous
                           caches only) or a positive multiple of 16 */
} ctx_decode_attn_desc;

/*
 * Create a handle on the current HIP device.  Validates desc, queries the
 * device and allocates the fp32 split workspace (owned by the handle).
 *   desc       host pointer, read only during the call
 *   out_handle host pointer; receives the handle (NULL on failure)
 * Errors: INVALID_ARG (NULL, non-positive sizes, split_tokens in 1..15, bad
 * dtype), UNSUPPORTED (head_dim, head ratio), OOM, HIP.
 */
int ctx_decode_attn_create(const ctx_decode_attn_desc* desc, ctx_decode_attn** out_handle);

/*
 * Queue one decode-attention step on `stream`.  Asynchronous: no host
 * synchronisation, no allocation and no host read of device data, so the
 * call can be captured in a HIP graph.
 *
 *   q           bf16 [num_seqs, Hq, D], contiguous: the new token's queries
 *   k_cache     bf16 [R, Hkv, D], contiguous rows: keys of every sequence
 *   v_cache     bf16 [R, Hkv, D], same layout: values
 *   seq_offsets int32 [num_seqs]: first cache row of sequence b
 *   seq_lens    int32 [num_seqs]: rows attended by sequence b, the current
 *               token included (its K/V row must already be in the cache)
 *   num_seqs    number of sequences, 0 <= num_seqs <= desc.max_batch
 *   scale       logit scale, e.g. 1/sqrt(128); applied in fp32 to q.k
 *   out         [num_seqs, Hq, D] of desc.out_dtype, contiguous
 *
 * Sequence b reads rows [seq_offsets[b], seq_offsets[b] + seq_lens[b]); the
 * regions may come in any order, may leave gaps between them (capacity
 * reserved for growth), and must lie inside the cache.  seq_lens[b] = 0
 * gives zeros.  Keys must be finite; a non-finite value V[r, kv, d] makes only
 * output dimension d of the heads reading it non-finite.  Device-side violations
 * (regions outside the cache, seq_lens[b] < 0, seq_lens[b] > max_seq_len
 * with split_tokens > 0) are undefined behaviour.
 *
 * The result is bitwise reproducible for fixed inputs on a fixed handle (no
 * floating-point atomics).  One handle serves any number of sequential run
 * calls on one stream (e.g. every layer); calls on different streams that
 * may overlap need separate handles, because they share the workspace.
 * Errors: INVALID_ARG, CAPACITY, ALIGNMENT, HIP.
 */
int ctx_decode_attn_run(ctx_decode_attn* handle, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* seq_offsets, const int32_t* seq_lens,
                        int32_t num_seqs, float scale, void* out, void* stream);

/*
 * Allocation-free variant of ctx_decode_attn_run, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  It takes no handle and allocates nothing
 * (no hipMalloc, hipFree or allocating library call): the split workspace is a
 * static device array of CTX_STATIC_SCRATCH_BYTES, one per device, held until
 * the process ends and looked up on the first call on each device.
 *
 *   desc        host pointer, read during the call: heads, head_dim, max_batch
 *               (num_seqs <= max_batch), out_dtype; split_tokens and page_tokens
 *               must be 0 (balanced split, contiguous caches).  max_seq_len is
 *               only checked to be positive.
 *   q, k_cache, v_cache, seq_offsets, seq_lens, num_seqs, scale, out, stream:
 *               as in ctx_decode_attn_run, with the same result bit for bit as
 *               a handle created from the same desc.
 *
 * The workspace a call needs is (R + num_seqs) x Hq x 520 bytes (R = 256 ranges
 * on an MI355X with Hkv = 8; 8.1 MiB for 256 sequences of 32 query heads);
 * larger calls fail with CTX_ERR_CAPACITY before launching anything.  Nothing in
 * the workspace needs to start at zero.  Every call on a device shares that
 * device's array: calls whose work may overlap on one device (different
 * streams, or different threads without ordering) race and must be serialised
 * by the caller.
 * Errors: INVALID_ARG, UNSUPPORTED (also for split_tokens or page_tokens != 0),
 * CAPACITY, ALIGNMENT, HIP.
 */
#define CTX_STATIC_SCRATCH_BYTES (16u << 20)
int ctx_decode_attn_run_static(const ctx_decode_attn_desc* desc, const void* q, const void* k_cache,
                               const void* v_cache, const int32_t* seq_offsets, const int32_t* seq_lens,
                               int32_t num_seqs, float scale, void* out, void* stream);

/*
 * Paged variant of ctx_decode_attn_run: the caches are split into pages of
 * P = desc.page_tokens tokens, as in the block tables of the paged-attention
 * serving engine the paper rolls out with (Sec. 5.1, vLLM; prefix caching is
 * off, tab:training-hyperparameters), and the step can append the token it
 * decodes (the token context grows by one token per step, eq:token-context).
 *
 *   q            bf16 [num_seqs, Hq, D]
 *   k_pages      bf16 [num_pages, P, Hkv, D]: token t of sequence b is slot t % P of
 *   v_pages      page block_tables[b][t / P] (same layout for V)
 *   block_tables int32 [num_seqs, max_pages_per_seq], row-major; entries
 *                0 .. ceil(seq_lens[b] / P) - 1 of row b must name valid pages
 *   seq_lens     int32 [num_seqs]: tokens attended, the new one included
 *   k_new, v_new bf16 [num_seqs, Hkv, D] or both NULL.  If given, the key and value
 *                of token seq_lens[b] - 1 are taken from them and also written
 *                into that token's cache slot (what the slot held before is never
 *                used); sequences with seq_lens[b] = 0 append nothing
 *   out          [num_seqs, Hq, D] of desc.out_dtype
 *
 * A page holding tokens of a sequence that appends must not be shared with
 * another sequence in the same call.  Same asynchrony, determinism and
 * ownership rules as ctx_decode_attn_run.
 * Errors: INVALID_ARG, CAPACITY, ALIGNMENT, HIP; UNSUPPORTED if the handle was
 * created with page_tokens = 0.
 */
int ctx_decode_attn_run_paged(ctx_decode_attn* handle, const void* q, void* k_pages, void* v_pages,
                              const int32_t* block_tables, int32_t max_pages_per_seq,
                              const int32_t* seq_lens, int32_t num_seqs, const void* k_new,
                              const void* v_new, float scale, void* out, void* stream);

/*
 * Causal prefill of each sequence's newest tokens against its cache.  The
 * reference-conditioned fast action adds the reference next observation
 * o^ref_{t+1} to the context before decoding (Sec. 4.1,
 * eq:reference-conditioned-action); the serving engine prefills such tokens
 * in chunks (tab:scheduling-hyperparameters).  Query i of sequence b sits at
 * position p = seq_lens[b] - q_lens[b] + i and attends to positions 0 .. p:
 *
 *   out[q_starts[b] + i, h, :] = sum_{t <= p} softmax_t(scale q.K[r_t, kv]) V[r_t, kv, :]
 *
 * with r_t = seq_offsets[b] + t and kv = h / (Hq / Hkv).
 *   q            bf16 [total_q, Hq, D]: sequence b's queries are rows q_starts[b] ..
 *                q_starts[b] + q_lens[b] - 1 (any order, no overlap)
 *   k_cache, v_cache  bf16 [R, Hkv, D] as in ctx_decode_attn_run; they already hold
 *                the new tokens' rows (the last q_lens[b] of the sequence)
 *   seq_offsets, seq_lens  int32 [num_seqs] as in ctx_decode_attn_run
 *   q_starts, q_lens  int32 [num_seqs]; 0 <= q_lens[b] <= seq_lens[b] and
 *                q_lens[b] <= max_q_len (device contract: undefined otherwise)
 *   max_q_len    host bound on q_lens (sizes the grid)
 *   flags        0 or CTX_PREFILL_SPLIT_P.  With 0 the softmax weights enter the
 *                P.V product rounded to bf16 (nearest even), and each row is
 *                normalised by the sum of the rounded weights, so it stays a convex
 *                combination of V rows (weights within 2^-8 relative of exact; a few
 *                1e-3 absolute on N(0,1) data).  CTX_PREFILL_SPLIT_P carries the
 *                weights as two bf16 terms (16 significant bits; about 1e-6
 *                absolute) at half again the matrix-core work.
 *   out          [total_q, Hq, D] of desc.out_dtype; rows of no sequence are untouched
 * Any group size the handle accepts (Hq / Hkv <= 16).  No workspace, no
 * allocation, no host sync; deterministic.
 * Errors: INVALID_ARG (also for unknown flag bits), CAPACITY, ALIGNMENT, HIP.
 */
#define CTX_PREFILL_SPLIT_P 1u
int ctx_prefill_attn_run(ctx_decode_attn* handle, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* seq_offsets, const int32_t* seq_lens, const int32_t* q_starts,
                         const int32_t* q_lens, int32_t num_seqs, int32_t max_q_len, float scale,
                         uint32_t flags, void* out, void* stream);

/* Wait for the handle's device, free the workspace and the handle.  NULL is a no-op. */
int ctx_decode_attn_destroy(ctx_decode_attn* handle);

/* Static description of a status code (never NULL). */
const char* ctx_decode_attn_status_string(int status);

/* Message for the last failing call on the calling thread ("" if none). */
const char* ctx_decode_attn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CTX_DECODE_ATTN_H_ */

/*
 * ctx_rollout_sim.h -- act-first rollout scheduling simulator (host code).
 *
 * Models the rollout batch of ActFirst-OPD against think-then-act rollout
 * (Sec. 4.3, Prop. 1, App. finite concurrency and rollout efficiency).  N
 * tasks each run T turns; turn t's interaction context becomes available when
 * the request gating it completes (environment steps take no time).  All
 * generation requests share max_concurrency slots (b_max): a request waits in
 * one FIFO queue ordered by submission time, then task, then turn, then kind
 * (fast action first), and holds a slot from admission to completion.
 *   VANILLA:  turn t submits a full response; its completion releases turn t+1.
 *   ACTFIRST: turn t submits a fast action and a full response together; the
 *             fast action's completion releases turn t+1 (the full response is
 *             asynchronous); the last turn submits both.
 * The completion time is when the last request finishes.
 *
 * Request k of task i, turn t is index (i * T + t) * 2 + k, k = 0 for the
 * fast action and 1 for the full response.  All pointers are HOST pointers
 * owned by the caller; outputs may be NULL when not wanted; unsubmitted
 * requests (VANILLA fast actions) report start = end = -1.  No function
 * allocates device memory or touches the GPU.
 * Errors (ctx_status): INVALID_ARG for NULL inputs, sizes out of range or
 * non-finite / negative costs, OOM if host memory runs out.
 */
#ifndef CTX_ROLLOUT_SIM_H_
#define CTX_ROLLOUT_SIM_H_

#include <stdint.h>

#include "ctx_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { CTX_ROLLOUT_VANILLA = 0, CTX_ROLLOUT_ACTFIRST = 1 } ctx_rollout_policy;

typedef struct {
  int32_t policy;          /* ctx_rollout_policy */
  int32_t num_tasks;       /* N >= 0 */
  int32_t turns;           /* T >= 1 */
  int32_t max_concurrency; /* b_max >= 1 */
} ctx_rollout_config;

/*
 * Latency model (the paper's analysis): a request holds its slot for a given
 * time, prefill and decoding included.
 *   fast_latency, full_latency  double [N * T] (task-major), > 0 and finite
 *   completion                  double [1] out
 *   req_start, req_end          double [N * T * 2] out, or NULL
 *   peak                        int32 [1] out: most requests admitted at once, or NULL
 */
int ctx_rollout_simulate(const ctx_rollout_config* cfg, const double* fast_latency, const double* full_latency,
                         double* completion, double* req_start, double* req_end, int32_t* peak);

typedef struct {
  double step_base;          /* seconds per decode step, whatever the batch (weight streaming) */
  double step_per_kv_token;  /* seconds per cached token of each admitted request, per step */
  double prefill_per_token;  /* seconds per context token of a request admitted at the step */
  int32_t fast_tokens;       /* output tokens of a fast action (>= 1) */
  int32_t full_tokens;       /* output tokens of a full response (>= 1) */
} ctx_rollout_engine;

/*
 * Engine model: decode steps.  At each step boundary the engine admits queued
 * requests up to b_max (each prefills its context), then every admitted
 * request generates one token.  A step lasts
 *   step_base + step_per_kv_token * (sum over admitted requests of context +
 *   tokens generated so far) + prefill_per_token * (context tokens admitted now).
 * A request completes at the end of the step producing its last token; what it
 * releases is submitted then and admitted at the next boundary.
 *   context_tokens  int32 [N * T] (task-major), >= 0: tokens of each turn's context
 *   steps           int64 [1] out: decode steps run, or NULL
 */
int ctx_rollout_simulate_engine(const ctx_rollout_config* cfg, const ctx_rollout_engine* engine,
                                const int32_t* context_tokens, double* completion, double* req_start,
                                double* req_end, int32_t* peak, int64_t* steps);

#ifdef __cplusplus
}
#endif

#endif /* CTX_ROLLOUT_SIM_H_ */

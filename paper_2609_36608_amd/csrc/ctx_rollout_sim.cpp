// ctx_rollout_sim.cpp -- act-first rollout scheduling simulator behind the C
// ABI declared in include/ctx_rollout_sim.h (host code).
//
// Two strategies share one FIFO admission queue and a cap of b_max admitted
// requests (Sec. 4.3; App. finite concurrency): think-then-act rollout
// releases a task's next turn when its full response completes, ActFirst-OPD
// when its fast action completes, with the full response running
// asynchronously.  The latency model advances from completion to completion
// (a heap of admitted requests by end time); the engine model advances one
// decode step at a time with a step cost that grows with the KV cache of the
// admitted requests, which is where the measured attention latency enters.

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <new>
#include <queue>
#include <set>
#include <tuple>
#include <vector>

#include "ctx_rollout_sim.h"

// the library's per-thread last-error message (defined with the attention entry points)
__attribute__((visibility("hidden"))) int ctx_report_error(int code, const char* msg);
__attribute__((visibility("hidden"))) void ctx_clear_error();

namespace {

constexpr int kFast = 0;
constexpr int kFull = 1;

// queue key: submission time, task, turn, kind (fast first)
using Pending = std::tuple<double, int, int, int>;

struct Sim {
  int policy, n, turns, cap;
  std::set<Pending> queue;
  double* start;
  double* end;

  void release(double when, int task, int turn) {
    if (policy == CTX_ROLLOUT_ACTFIRST) queue.emplace(when, task, turn, kFast);
    queue.emplace(when, task, turn, kFull);
  }
  bool gates(int kind) const {
    return (policy == CTX_ROLLOUT_VANILLA && kind == kFull) || (policy == CTX_ROLLOUT_ACTFIRST && kind == kFast);
  }
  void record(double* arr, int task, int turn, int kind, double v) {
    if (arr != nullptr) arr[((size_t)task * turns + turn) * 2 + kind] = v;
  }
};

int check_config(const ctx_rollout_config* cfg) {
  if (cfg == nullptr) return ctx_report_error(CTX_ERR_INVALID_ARG, "cfg is NULL");
  if (cfg->policy != CTX_ROLLOUT_VANILLA && cfg->policy != CTX_ROLLOUT_ACTFIRST)
    return ctx_report_error(CTX_ERR_INVALID_ARG, "unknown policy");
  if (cfg->num_tasks < 0 || cfg->turns < 1 || cfg->max_concurrency < 1)
    return ctx_report_error(CTX_ERR_INVALID_ARG, "need num_tasks >= 0, turns >= 1, max_concurrency >= 1");
  return CTX_OK;
}

void init_outputs(const ctx_rollout_config* cfg, double* start, double* end) {
  const size_t m = (size_t)cfg->num_tasks * cfg->turns * 2;
  for (size_t i = 0; i < m; ++i) {
    if (start != nullptr) start[i] = -1.0;
    if (end != nullptr) end[i] = -1.0;
  }
}

}  // namespace

extern "C" int ctx_rollout_simulate(const ctx_rollout_config* cfg, const double* fast_latency,
                                    const double* full_latency, double* completion, double* req_start,
                                    double* req_end, int32_t* peak) {
  ctx_clear_error();
  int rc = check_config(cfg);
  if (rc != CTX_OK) return rc;
  if (completion == nullptr || full_latency == nullptr ||
      (cfg->policy == CTX_ROLLOUT_ACTFIRST && fast_latency == nullptr))
    return ctx_report_error(CTX_ERR_INVALID_ARG, "NULL latency or completion pointer");
  const size_t m = (size_t)cfg->num_tasks * cfg->turns;
  for (size_t i = 0; i < m; ++i) {
    if (!(std::isfinite(full_latency[i]) && full_latency[i] > 0.0) ||
        (cfg->policy == CTX_ROLLOUT_ACTFIRST && !(std::isfinite(fast_latency[i]) && fast_latency[i] > 0.0)))
      return ctx_report_error(CTX_ERR_INVALID_ARG, "latencies must be finite and > 0");
  }
  try {
    init_outputs(cfg, req_start, req_end);
    Sim s{cfg->policy, cfg->num_tasks, cfg->turns, cfg->max_concurrency, {}, req_start, req_end};
    // admitted requests by (end time, task, turn, kind)
    std::priority_queue<Pending, std::vector<Pending>, std::greater<Pending>> running;
    for (int i = 0; i < s.n; ++i) s.release(0.0, i, 0);
    double now = 0.0, last = 0.0;
    int top = 0;
    while (!s.queue.empty() || !running.empty()) {
      while (!s.queue.empty() && (int)running.size() < s.cap && std::get<0>(*s.queue.begin()) <= now) {
        const auto [sub, i, t, k] = *s.queue.begin();
        s.queue.erase(s.queue.begin());
        const double lat = (k == kFast ? fast_latency : full_latency)[(size_t)i * s.turns + t];
        s.record(req_start, i, t, k, now);
        running.emplace(now + lat, i, t, k);
      }
      if ((int)running.size() > top) top = (int)running.size();
      if (running.empty()) {  // nothing admitted: jump to the next submission
        now = std::get<0>(*s.queue.begin());
        continue;
      }
      now = std::get<0>(running.top());
      while (!running.empty() && std::get<0>(running.top()) == now) {
        const auto [e, i, t, k] = running.top();
        running.pop();
        s.record(req_end, i, t, k, e);
        if (e > last) last = e;
        if (s.gates(k) && t + 1 < s.turns) s.release(e, i, t + 1);
      }
    }
    *completion = last;
    if (peak != nullptr) *peak = top;
  } catch (const std::bad_alloc&) {
    return ctx_report_error(CTX_ERR_OOM, "host memory");
  }
  return CTX_OK;
}

extern "C" int ctx_rollout_simulate_engine(const ctx_rollout_config* cfg, const ctx_rollout_engine* engine,
                                           const int32_t* context_tokens, double* completion, double* req_start,
                                           double* req_end, int32_t* peak, int64_t* steps) {
  ctx_clear_error();
  int rc = check_config(cfg);
  if (rc != CTX_OK) return rc;
  if (engine == nullptr || context_tokens == nullptr || completion == nullptr)
    return ctx_report_error(CTX_ERR_INVALID_ARG, "NULL engine, context_tokens or completion");
  const ctx_rollout_engine eng = *engine;
  if (!(std::isfinite(eng.step_base) && eng.step_base >= 0.0 && std::isfinite(eng.step_per_kv_token) &&
        eng.step_per_kv_token >= 0.0 && std::isfinite(eng.prefill_per_token) && eng.prefill_per_token >= 0.0))
    return ctx_report_error(CTX_ERR_INVALID_ARG, "step costs must be finite and >= 0");
  if (eng.fast_tokens < 1 || eng.full_tokens < 1)
    return ctx_report_error(CTX_ERR_INVALID_ARG, "fast_tokens and full_tokens must be >= 1");
  const size_t m = (size_t)cfg->num_tasks * cfg->turns;
  for (size_t i = 0; i < m; ++i)
    if (context_tokens[i] < 0) return ctx_report_error(CTX_ERR_INVALID_ARG, "negative context_tokens");
  try {
    init_outputs(cfg, req_start, req_end);
    Sim s{cfg->policy, cfg->num_tasks, cfg->turns, cfg->max_concurrency, {}, req_start, req_end};
    struct Active {
      int task, turn, kind, generated;
    };
    std::vector<Active> running, still;
    std::vector<Active> finished;
    for (int i = 0; i < s.n; ++i) s.release(0.0, i, 0);
    double now = 0.0, last = 0.0;
    int top = 0;
    int64_t nsteps = 0;
    while (!s.queue.empty() || !running.empty()) {
      int64_t admitted_ctx = 0;
      while (!s.queue.empty() && (int)running.size() < s.cap && std::get<0>(*s.queue.begin()) <= now) {
        const auto [sub, i, t, k] = *s.queue.begin();
        s.queue.erase(s.queue.begin());
        s.record(req_start, i, t, k, now);
        running.push_back({i, t, k, 0});
        admitted_ctx += context_tokens[(size_t)i * s.turns + t];
      }
      if ((int)running.size() > top) top = (int)running.size();
      if (running.empty()) {
        now = std::get<0>(*s.queue.begin());
        continue;
      }
      int64_t kv = 0;
      for (const Active& r : running) kv += (int64_t)context_tokens[(size_t)r.task * s.turns + r.turn] + r.generated;
      const double duration = eng.step_base + eng.step_per_kv_token * (double)kv +
                              eng.prefill_per_token * (double)admitted_ctx;
      now = now + duration;
      ++nsteps;
      still.clear();
      finished.clear();
      for (Active r : running) {
        r.generated += 1;
        const int target = r.kind == kFast ? eng.fast_tokens : eng.full_tokens;
        (r.generated >= target ? finished : still).push_back(r);
      }
      running.swap(still);
      for (const Active& r : finished) {
        s.record(req_end, r.task, r.turn, r.kind, now);
        if (now > last) last = now;
        if (s.gates(r.kind) && r.turn + 1 < s.turns) s.release(now, r.task, r.turn + 1);
      }
    }
    *completion = last;
    if (peak != nullptr) *peak = top;
    if (steps != nullptr) *steps = nsteps;
  } catch (const std::bad_alloc&) {
    return ctx_report_error(CTX_ERR_OOM, "host memory");
  }
  return CTX_OK;
}

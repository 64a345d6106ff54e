"""CPU oracle for the act-first rollout scheduler (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module.  It is a plain, slow simulation written from the paper's
description of the two rollout strategies (Sec. 4.3 and App. finite
concurrency / rollout efficiency), plus the paper's closed forms.

Rollout model.  N tasks each run T turns.  Turn t of task i has an interaction
context that becomes available at time s[i][t] (s[i][0] = 0; environment
steps take no time).  Generation requests share b_max concurrency slots: a
request waits in one FIFO queue (ordered by submission time, then task, then
turn, then kind with the fast action first) and, once admitted, holds a slot
until it completes.
  * Vanilla OPD: turn t submits one full response; its completion makes turn
    t+1's context available.
  * ActFirst-OPD: turn t submits a fast action and a full response together;
    the fast action's completion makes turn t+1's context available (the full
    response is asynchronous).  The last turn still submits both.
The batch completion time C is the time the last request finishes.

Two service models:
  * "latency" (the paper's analysis): a request holds its slot for a given
    latency l_fast[i][t] or l_full[i][t] (prefill and decoding included).
  * "engine": a serving engine runs decode steps; at each step boundary it
    admits queued requests up to b_max (each newly admitted request first
    prefills its context), then every admitted request generates one token.
    A step lasts  base + per_kv * (tokens held in the KV cache of the
    admitted requests: context + tokens generated so far) + prefill * (context
    tokens of the requests admitted at that boundary).  A request completes at
    the end of the step that produces its last output token; what it releases
    is submitted at that time and admitted at the next boundary.

Parity: pinned (Prop. 1 closed form, the calibrated estimate of
eq:calibrated-rollout-speedup, the bounds of eq:finite-capacity-time-bound,
a schedule worked by hand, and the exact agreement of the two models when the
step cost is constant; see the tests).
"""
from __future__ import annotations

VANILLA = 0
ACTFIRST = 1
FAST = 0
FULL = 1


def _requests_released(policy, task, turn, turns):
    """Requests submitted when turn `turn` of `task` becomes available, in queue order."""
    if policy == VANILLA:
        return [(task, turn, FULL)]
    return [(task, turn, FAST), (task, turn, FULL)]


def _gates_next_turn(policy, kind):
    return (policy == VANILLA and kind == FULL) or (policy == ACTFIRST and kind == FAST)


def simulate_latency(policy, l_fast, l_full, b_max):
    """Service model "latency".  l_fast, l_full: [N][T] seconds.  Returns a dict
    with completion, start and end times per request key (task, turn, kind)
    and the peak number of admitted requests."""
    n = len(l_full)
    turns = len(l_full[0]) if n else 0
    lat = {FAST: l_fast, FULL: l_full}
    queue = []          # (submit_time, task, turn, kind)
    running = []        # (end_time, task, turn, kind)
    start, end = {}, {}
    for i in range(n):
        for r in _requests_released(policy, i, 0, turns):
            queue.append((0.0,) + r)
    now = 0.0
    peak = 0
    while queue or running:
        # admit in FIFO order while slots are free
        queue.sort()
        while queue and len(running) < b_max and queue[0][0] <= now:
            sub, i, t, k = queue.pop(0)
            start[(i, t, k)] = now
            running.append((now + lat[k][i][t], i, t, k))
        peak = max(peak, len(running))
        if not running:  # nothing admitted yet: jump to the next submission
            now = min(q[0] for q in queue)
            continue
        # advance to the earliest completion; everything ending then finishes
        t_next = min(r[0] for r in running)
        now = t_next
        done = sorted(r for r in running if r[0] == t_next)
        running = [r for r in running if r[0] != t_next]
        for e, i, t, k in done:
            end[(i, t, k)] = e
            if _gates_next_turn(policy, k) and t + 1 < turns:
                for r in _requests_released(policy, i, t + 1, turns):
                    queue.append((e,) + r)
    completion = max(end.values()) if end else 0.0
    return {"completion": completion, "start": start, "end": end, "peak": peak}


def simulate_engine(policy, context_tokens, fast_tokens, full_tokens, b_max, base, per_kv, prefill):
    """Service model "engine".  context_tokens: [N][T] tokens of each turn's
    context.  Returns the same dict as simulate_latency plus the step count."""
    n = len(context_tokens)
    turns = len(context_tokens[0]) if n else 0
    out_tokens = {FAST: fast_tokens, FULL: full_tokens}
    queue = []      # (submit_time, task, turn, kind)
    running = []    # [task, turn, kind, generated]
    start, end = {}, {}
    for i in range(n):
        for r in _requests_released(policy, i, 0, turns):
            queue.append((0.0,) + r)
    now = 0.0
    peak = 0
    steps = 0
    while queue or running:
        queue.sort()
        admitted_ctx = 0
        while queue and len(running) < b_max and queue[0][0] <= now:
            _, i, t, k = queue.pop(0)
            start[(i, t, k)] = now
            running.append([i, t, k, 0])
            admitted_ctx += context_tokens[i][t]
        peak = max(peak, len(running))
        if not running:
            now = min(q[0] for q in queue)
            continue
        kv = 0
        for i, t, k, g in running:
            kv += context_tokens[i][t] + g
        duration = base + per_kv * kv + prefill * admitted_ctx
        now = now + duration
        steps += 1
        still = []
        finished = []
        for req in running:
            req[3] += 1
            if req[3] >= out_tokens[req[2]]:
                finished.append(req)
            else:
                still.append(req)
        running = still
        for i, t, k, _ in sorted(finished):
            end[(i, t, k)] = now
            if _gates_next_turn(policy, k) and t + 1 < turns:
                for r in _requests_released(policy, i, t + 1, turns):
                    queue.append((now,) + r)
    completion = max(end.values()) if end else 0.0
    return {"completion": completion, "start": start, "end": end, "peak": peak, "steps": steps}


# ------------------------------------------------------------ closed forms

def ideal_speedup(turns, l_fast, l_full):
    """Prop. 1, eq:ideal-rollout-speedup: T l_full / ((T - 1) l_fast + l_full)."""
    return turns * l_full / ((turns - 1) * l_fast + l_full)


def calibrated_completion(policy, l_fast, l_full, turns):
    """eq:calibrated-rollout-speedup for one batch with per-task constant
    latencies l_fast[i], l_full[i] and unrestricted overlap."""
    if policy == VANILLA:
        return max(turns * lf for lf in l_full)
    return max((turns - 1) * a + max(a, f) for a, f in zip(l_fast, l_full))


def completion_lower_bound(num_tasks, turns, l_fast, l_full, b_max):
    """eq:finite-capacity-time-bound (constant latencies): the larger of the
    dependency chain and the slot-time bound."""
    return max((turns - 1) * l_fast + l_full, num_tasks * turns * (l_fast + l_full) / b_max)

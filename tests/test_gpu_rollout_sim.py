"""The rollout scheduling simulator driven by costs measured on this GPU.

The engine model's parameters (the step model of App. finite concurrency,
priced as in the calibrated estimate eq:calibrated-rollout-speedup) are
measured in this process from the library's own kernels: the decode
attention's per-call and per-KV-token cost, the read ceiling (ctx_hbm_read)
that prices the weight streaming, and the causal prefill kernel's matrix-core
rate.  With those parameters the native simulator and the oracle must produce
the same schedule, request by request and bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import oracle_sched as sch
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import rollout_calibration as rc

from _gpu_util import dev

pytestmark = pytest.mark.gpu


def oracle_arrays(res, n, turns):
    st = np.full((n, turns, 2), -1.0)
    en = np.full((n, turns, 2), -1.0)
    for (i, t, k), v in res["start"].items():
        st[i, t, k] = v
    for (i, t, k), v in res["end"].items():
        en[i, t, k] = v
    return st, en


@pytest.fixture(scope="module")
def calibration():
    cal = rc.calibrate_engine(torch, dev(), reduced=True)
    for k, v in cal["sources"].items():
        print(f"{k} = {cal['engine'][k]:.6g}: {v}", flush=True)
    return cal


def test_measured_costs_are_physical(calibration):
    read, pf, att = calibration["read_ceiling"], calibration["prefill"], calibration["attention"]
    assert 2000.0 < read["gbs"] <= 8000.0, read          # below the 8 TB/s HBM peak
    assert 50.0 < pf["tflops"] <= 2500.0, pf             # below the 2.5 PFLOP/s bf16 MFMA peak
    assert att["per_kv_token_s"] > 0.0 and att["achieved_gbs"] <= 8000.0, att
    # the line fits every measured point: the cost is linear in the KV tokens
    # (within 15%, or 3 us, about one launch's jitter, at the smallest point)
    for p in att["points"]:
        fit = att["per_call_s"] + att["per_kv_token_s"] * p["kv_tokens"]
        assert abs(fit - p["seconds"]) <= max(0.15 * p["seconds"], 3e-6), (p, fit)
    eng = calibration["engine"]
    assert all(np.isfinite(v) and v > 0 for v in eng.values()), eng


@pytest.mark.parametrize("b_max", [8, 64, 256])
def test_native_schedule_equals_oracle_with_measured_engine(calibration, b_max):
    """The rollout-efficiency study's shape, reduced (16 tasks, T = 8 turns,
    16-token fast actions, 128-token full responses), fixed contexts
    U{1500..3000}: completion, every request's start and end, the peak and
    the step count agree exactly."""
    eng = calibration["engine"]
    n, turns = 16, 8
    rng = np.random.default_rng(30)
    ctx = np.repeat(rng.integers(1500, 3001, size=n)[:, None], turns, axis=1).astype(np.int32)
    comp = {}
    for policy in (sch.VANILLA, sch.ACTFIRST):
        ref = sch.simulate_engine(policy, ctx.tolist(), 16, 128, b_max, eng["step_base"], eng["step_per_kv_token"],
                                  eng["prefill_per_token"])
        got = bd.rollout_simulate_engine(policy, ctx, 16, 128, b_max, **eng)
        st, en = oracle_arrays(ref, n, turns)
        assert got["completion"] == ref["completion"]
        np.testing.assert_array_equal(got["start"], st)
        np.testing.assert_array_equal(got["end"], en)
        assert got["peak"] == ref["peak"] and got["steps"] == ref["steps"]
        comp[policy] = got["completion"]
    speedup = comp[sch.VANILLA] / comp[sch.ACTFIRST]
    print(f"b_max {b_max}: simulated speedup {speedup:.4f}", flush=True)
    # eq:finite-capacity-time-bound: no schedule beats T-fold (here also r = 128/16 = 8)
    assert 0.0 < speedup <= turns

"""The native rollout scheduling simulator (ctx_rollout_simulate*, host code
in the library) against the Python oracle, request by request."""
import numpy as np
import pytest

from oracle import oracle_sched as sch
from paper_2609_36608_amd import binding as bd


def oracle_arrays(res, n, turns):
    st = np.full((n, turns, 2), -1.0)
    en = np.full((n, turns, 2), -1.0)
    for (i, t, k), v in res["start"].items():
        st[i, t, k] = v
    for (i, t, k), v in res["end"].items():
        en[i, t, k] = v
    return st, en


def assert_same(native, ref, n, turns):
    st, en = oracle_arrays(ref, n, turns)
    assert native["completion"] == ref["completion"]
    np.testing.assert_array_equal(native["start"], st)
    np.testing.assert_array_equal(native["end"], en)
    assert native["peak"] == ref["peak"]


@pytest.mark.parametrize("seed", range(12))
def test_latency_model_parity(seed):
    rng = np.random.default_rng(seed)
    n, turns = int(rng.integers(1, 7)), int(rng.integers(1, 9))
    b = int(rng.integers(1, 3 * n + 2))
    fast = rng.uniform(0.05, 2.0, (n, turns))
    full = rng.uniform(0.1, 6.0, (n, turns))
    if seed % 3 == 0:  # integer latencies: many simultaneous events and queue ties
        fast, full = np.ceil(fast), np.ceil(full)
    for policy in (sch.VANILLA, sch.ACTFIRST):
        ref = sch.simulate_latency(policy, fast.tolist(), full.tolist(), b)
        got = bd.rollout_simulate(policy, fast, full, b)
        assert_same(got, ref, n, turns)


@pytest.mark.parametrize("seed", range(8))
def test_engine_model_parity(seed):
    rng = np.random.default_rng(100 + seed)
    n, turns = int(rng.integers(1, 6)), int(rng.integers(1, 6))
    b = int(rng.integers(1, 3 * n + 2))
    ctx = rng.integers(0, 400, (n, turns))
    fast_tokens, full_tokens = int(rng.integers(1, 6)), int(rng.integers(1, 20))
    base, per_kv, prefill = 1e-3 * rng.uniform(0.5, 2), 1e-7 * rng.uniform(0, 3), 1e-6 * rng.uniform(0, 2)
    for policy in (sch.VANILLA, sch.ACTFIRST):
        ref = sch.simulate_engine(policy, ctx.tolist(), fast_tokens, full_tokens, b, base, per_kv, prefill)
        got = bd.rollout_simulate_engine(policy, ctx, fast_tokens, full_tokens, b, base, per_kv, prefill)
        assert_same(got, ref, n, turns)
        assert got["steps"] == ref["steps"]


def test_paper_concurrency_scan_parity():
    """The rollout-efficiency scan of tab:scheduling-hyperparameters (16 tasks,
    T = 30, b_max 16..256) with per-task latencies: native equals oracle."""
    rng = np.random.default_rng(7)
    n, turns = 16, 30
    lf = rng.uniform(0.3, 0.6, n)[:, None].repeat(turns, 1)
    lu = rng.uniform(3.0, 9.0, n)[:, None].repeat(turns, 1)
    for b in (16, 32, 64, 128, 256):
        for policy in (sch.VANILLA, sch.ACTFIRST):
            ref = sch.simulate_latency(policy, lf.tolist(), lu.tolist(), b)
            got = bd.rollout_simulate(policy, lf, lu, b)
            assert_same(got, ref, n, turns)
    # with a slot for every request the calibrated estimate is exact
    big = 2 * n * turns
    for policy in (sch.VANILLA, sch.ACTFIRST):
        got = bd.rollout_simulate(policy, lf, lu, big)
        assert got["completion"] == pytest.approx(sch.calibrated_completion(policy, lf[:, 0], lu[:, 0], turns))


def test_engine_scan_parity_128_tokens():
    rng = np.random.default_rng(3)
    n, turns = 16, 6
    ctx = (2000 + 150 * np.arange(turns))[None, :].repeat(n, 0) + rng.integers(0, 300, (n, 1))
    for b in (16, 64, 256):
        for policy in (sch.VANILLA, sch.ACTFIRST):
            ref = sch.simulate_engine(policy, ctx.tolist(), 16, 128, b, 5e-4, 2e-8, 1e-7)
            got = bd.rollout_simulate_engine(policy, ctx, 16, 128, b, 5e-4, 2e-8, 1e-7)
            assert_same(got, ref, n, turns)


def test_edges_and_errors():
    z = np.zeros((0, 3))
    assert bd.rollout_simulate(sch.ACTFIRST, z, z, 4)["completion"] == 0.0
    one = np.ones((2, 3))
    with pytest.raises(bd.CtxError):
        bd.rollout_simulate(sch.ACTFIRST, one, one, 0)
    with pytest.raises(bd.CtxError):
        bd.rollout_simulate(sch.ACTFIRST, one, -one, 2)
    with pytest.raises(bd.CtxError):
        bd.rollout_simulate(5, one, one, 2)
    with pytest.raises(bd.CtxError):
        bd.rollout_simulate_engine(sch.VANILLA, np.ones((2, 3), np.int32), 0, 4, 2, 1.0, 0.0, 0.0)
    with pytest.raises(bd.CtxError):
        bd.rollout_simulate_engine(sch.VANILLA, np.ones((2, 3), np.int32), 1, 4, 2, float("nan"), 0.0, 0.0)
    # Vanilla never submits fast actions
    r = bd.rollout_simulate(sch.VANILLA, one, one, 2)
    assert (r["start"][:, :, 0] == -1).all() and (r["end"][:, :, 0] == -1).all()

"""The seeded input generator: determinism, bf16 rounding, length distributions."""
import hashlib
import math

import numpy as np
import pytest
import torch

from paper_2609_36608_amd import workloads as wl


def test_bf16_rounding_matches_torch_bit_for_bit():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(500_000).astype(np.float32),
        (rng.standard_normal(200_000) * 1e-39).astype(np.float32),   # subnormals
        rng.uniform(-1e30, 1e30, 100_000).astype(np.float32),
        # exact ties: low 16 bits = 0x8000, both parities of the kept bit, every
        # finite positive exponent (NaN payloads are not compared)
        (np.arange(1, 0x7F80, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38], np.float32),
    ])
    ours = wl.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = wl.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())
    assert wl.f32_to_bf16_bits(np.array([np.nan], np.float32))[0] == wl.BF16_NAN


def _digest(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_generator_is_deterministic_and_keyed():
    w = wl.WORKLOADS["tiny"]
    a = wl.draw_lengths(w), wl.query_bits(w, 0), *wl.sequence_kv_bits(w, 0, 2, 100)
    b = wl.draw_lengths(w), wl.query_bits(w, 0), *wl.sequence_kv_bits(w, 0, 2, 100)
    assert _digest(*a) == _digest(*b)
    c = wl.sequence_kv_bits(w, 0, 3, 100)
    assert _digest(*c) != _digest(*a[2:])
    # a sequence's rows do not depend on how many rows are drawn after them
    k_short, _ = wl.sequence_kv_bits(w, 0, 2, 50)
    np.testing.assert_array_equal(k_short, a[2][:50])


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_lengths_within_bounds(name):
    w = wl.WORKLOADS[name]
    lens = wl.draw_lengths(w)
    assert lens.shape == (w.batch,)
    assert lens.min() >= w.length_lo + w.extra_lo
    assert lens.max() <= w.length_hi + w.extra_hi
    lay = wl.workload_layout(w)
    assert lay.max_seq_len <= w.length_hi + w.extra_hi + w.steps - 1
    assert lay.num_rows == int((lens.astype(np.int64) + w.steps - 1).sum())
    # regions are disjoint and inside the cache
    order = np.argsort(lay.offsets)
    ends = lay.offsets[order] + lay.capacity[order]
    assert (lay.offsets[order][1:] >= ends[:-1]).all() and ends[-1] <= lay.num_rows


def test_loguniform_lengths_distribution():
    """log L is uniform on [ln 512, ln 32768]: check the mean of log L over a
    large draw, and the expected mean length (32768-512)/ln 64 ~ 7,756."""
    w = wl.Workload("lu", 77, 1, 200_000, 32, 8, 1, "loguniform", 512, 32768)
    lens = wl.draw_lengths(w)
    lo, hi = math.log(512), math.log(32768)
    assert abs(np.log(lens + 0.5).mean() - (lo + hi) / 2) < 0.02
    assert abs(lens.mean() / ((32768 - 512) / math.log(64)) - 1) < 0.02


def test_peaky_keys_rate_and_exact_gain():
    w = wl.WORKLOADS["act_first_burst"]
    rows = 40_000
    k, _ = wl.sequence_kv_bits(w, 0, 0, rows)
    mask = wl.peaky_mask(w, 0, 0, rows)
    assert abs(mask.mean() - 0.05) < 0.004
    # the same rows, drawn without the gain, are exactly a quarter
    plain = wl.normal_bf16(wl.rng_for(wl.DEFAULT_SEED, w.index, 0, 1, 0), (rows, w.num_kv_heads, 128))
    kf, pf = wl.bf16_bits_to_f32(k), wl.bf16_bits_to_f32(plain)
    np.testing.assert_array_equal(kf[mask], pf[mask] * 4)
    np.testing.assert_array_equal(kf[~mask], pf[~mask])


def test_layout_shuffle_and_gaps():
    rng = np.random.default_rng(3)
    lens = np.array([5, 0, 9, 1])
    lay = wl.make_layout(lens, steps=2, gap_max=3, shuffle=True, rng=rng)
    assert list(lay.capacity) == [6, 1, 10, 2]
    spans = sorted((o, o + c) for o, c in zip(lay.offsets, lay.capacity))
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert list(lay.lens_at(1)) == [6, 1, 10, 2]
    with pytest.raises(ValueError):
        lay.lens_at(2)

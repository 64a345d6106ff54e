"""Pins of the CPU oracle against facts fixed by mathematics, not by the oracle.

Each test names the mistake it is there to catch.  The oracle computes one
decode step of softmax attention of each request's new token over its token
context (Sec. 3, eq:token-context), with grouped KV heads.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2609_36608_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
bf = wl.f32_to_bf16_bits
unbf = wl.bf16_bits_to_f32


def rand_bits(rng, shape, scale=1.0):
    return bf(rng.standard_normal(shape).astype(np.float32) * np.float32(scale))


def single(q, k, v, scale):
    """One sequence at offset 0 using all rows."""
    n = k.shape[0]
    return oracle.decode_attn(q, k, v, np.array([0]), np.array([n]), scale)


# ------------------------------------------------------------- closed forms

def test_golden_three_keys():
    """Hand-derived closed form (weights 1/7, 2/7, 4/7). Catches a sign flip in
    the softmax, a missing normalisation and wrong q/K pairing."""
    g = json.load(open(os.path.join(GOLDEN, "three_keys.json")))
    q = bf(np.array(g["q"], np.float32)).reshape(1, 1, -1)
    k = bf(np.array(g["k"], np.float32)).reshape(3, 1, -1)
    v = bf(np.array(g["v"], np.float32)).reshape(3, 1, -1)
    out = single(q, k, v, g["scale"])[0, 0]
    np.testing.assert_allclose(out, g["out"], rtol=0, atol=1e-13)
    w = oracle.attn_weights(q, k, [0], [3], g["scale"], 0, 0)
    np.testing.assert_allclose(w, g["weights"], rtol=1e-14, atol=0)


def test_single_key_returns_its_value_row_exactly():
    """P1: L = 1 -> weight exp(0)/exp(0) = 1, output is the V row bit for bit.
    Catches off-by-one lengths (0 rows read) and row/head indexing slips."""
    rng = np.random.default_rng(1)
    hq, hkv, d = 8, 2, 128
    k = rand_bits(rng, (5, hkv, d))
    v = rand_bits(rng, (5, hkv, d))
    q = rand_bits(rng, (3, hq, d))
    offs, lens = np.array([4, 0, 2]), np.array([1, 1, 1])
    out = oracle.decode_attn(q, k, v, offs, lens, 0.0884)
    for b in range(3):
        for h in range(hq):
            assert np.array_equal(out[b, h], unbf(v[offs[b], h // (hq // hkv)]).astype(np.float64))


def test_identical_keys_give_mean_of_values():
    """P2: equal logits -> uniform weights -> mean of the sequence's V rows."""
    rng = np.random.default_rng(2)
    L, d = 37, 128
    krow = rand_bits(rng, (1, 1, d))
    k = np.repeat(krow, L, axis=0)
    v = rand_bits(rng, (L, 1, d))
    q = rand_bits(rng, (1, 1, d))
    out = single(q, k, v, 0.3)[0, 0]
    np.testing.assert_allclose(out, unbf(v[:, 0]).astype(np.float64).mean(axis=0), rtol=0, atol=1e-14)


def test_constant_values_are_returned():
    """P3: V = c everywhere -> out = c, whatever the keys.  Catches weights not
    summing to one (a dropped or doubled normaliser)."""
    rng = np.random.default_rng(3)
    L, d = 300, 128
    k = rand_bits(rng, (L, 2, d), scale=3.0)
    v = np.full((L, 2, d), bf(np.array([-1.375], np.float32))[0], dtype=np.uint16)
    q = rand_bits(rng, (1, 4, d))
    out = single(q, k, v, 1 / math.sqrt(d))
    np.testing.assert_allclose(out, -1.375, rtol=1e-14, atol=0)


def test_zero_query_averages_exactly_the_sequence_rows():
    """P4: q = 0 -> uniform weights over rows [off, off + L).  The cache holds
    other sequences and NaN gaps around it, so reading one row too many, too
    few or from the wrong offset shows up."""
    rng = np.random.default_rng(4)
    d, hkv, hq = 128, 2, 4
    rows = 64
    k = rand_bits(rng, (rows, hkv, d))
    v = rand_bits(rng, (rows, hkv, d))
    k[:10] = wl.BF16_NAN
    v[:10] = wl.BF16_NAN
    k[30:] = wl.BF16_NAN
    v[30:] = wl.BF16_NAN
    q = np.zeros((1, hq, d), np.uint16)
    out = oracle.decode_attn(q, k, v, [10], [20], 0.5)
    for h in range(hq):
        expect = unbf(v[10:30, h // 2]).astype(np.float64).mean(axis=0)
        np.testing.assert_allclose(out[0, h], expect, rtol=0, atol=1e-14)


def test_scale_zero_is_uniform_average():
    """scale = 0 -> all logits 0 -> mean over the rows, whatever q and K."""
    rng = np.random.default_rng(14)
    L, d = 50, 128
    k = rand_bits(rng, (L, 1, d), 4.0)
    v = rand_bits(rng, (L, 1, d))
    q = rand_bits(rng, (1, 1, d), 4.0)
    out = single(q, k, v, 0.0)[0, 0]
    np.testing.assert_allclose(out, unbf(v[:, 0]).astype(np.float64).mean(axis=0), rtol=0, atol=1e-14)


def test_two_keys_designed_logits():
    """P8: q = 1 in every dim, K row t = x_t in every dim, so
    s_t = scale * D * x_t without evaluating a dot product here, and
    out = sigmoid(s0 - s1) v0 + sigmoid(s1 - s0) v1.
    Catches a dropped dimension (D-1 terms), a missing or squared scale and a
    sign error in the softmax."""
    d = 128
    scale = 1 / math.sqrt(d)
    rng = np.random.default_rng(8)
    for x0, x1 in [(0.25, -0.5), (0.0, 0.015625), (-0.75, -0.75), (0.5, 0.125)]:
        q = np.full((1, 1, d), bf(np.array([1.0], np.float32))[0], np.uint16)
        k = np.stack([np.full((1, d), bf(np.array([x0], np.float32))[0]),
                      np.full((1, d), bf(np.array([x1], np.float32))[0])]).astype(np.uint16)
        v = rand_bits(rng, (2, 1, d))
        s0, s1 = scale * d * x0, scale * d * x1
        w0 = 1.0 / (1.0 + math.exp(s1 - s0))
        w1 = 1.0 / (1.0 + math.exp(s0 - s1))
        expect = w0 * unbf(v[0, 0]).astype(np.float64) + w1 * unbf(v[1, 0]).astype(np.float64)
        np.testing.assert_allclose(single(q, k, v, scale)[0, 0], expect, rtol=1e-13, atol=1e-14)


def test_query_dim_pairs_with_key_dim():
    """q = e_j (one-hot), so s_t = scale * K[t, kv, j].  With two keys the
    output is a sigmoid of K[0,kv,j] - K[1,kv,j]; pairing q's dim j with any
    other key dim, or reading another KV head's key, changes it."""
    d, hkv, hq = 128, 2, 4
    rng = np.random.default_rng(9)
    k = rand_bits(rng, (2, hkv, d))
    v = rand_bits(rng, (2, hkv, d))
    kf = unbf(k).astype(np.float64)
    vf = unbf(v).astype(np.float64)
    for j in [0, 1, 63, 64, 127]:
        q = np.zeros((1, hq, d), np.uint16)
        q[0, :, j] = bf(np.array([1.0], np.float32))[0]
        out = oracle.decode_attn(q, k, v, [0], [2], 2.0)
        for h in range(hq):
            kv = h // (hq // hkv)
            s0, s1 = 2.0 * kf[0, kv, j], 2.0 * kf[1, kv, j]
            w0 = 1.0 / (1.0 + math.exp(s1 - s0))
            expect = w0 * vf[0, kv] + (1 - w0) * vf[1, kv]
            np.testing.assert_allclose(out[0, h], expect, rtol=1e-13, atol=1e-14)


# ------------------------------------------------------------- invariants

def test_key_value_permutation_invariance():
    """P5: attention is a set function of the (K, V) rows of a sequence."""
    rng = np.random.default_rng(5)
    L, d = 129, 128
    k = rand_bits(rng, (L, 2, d))
    v = rand_bits(rng, (L, 2, d))
    q = rand_bits(rng, (1, 8, d))
    perm = rng.permutation(L)
    a = single(q, k, v, 0.1)
    b = single(q, k[perm], v[perm], 0.1)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-14)


def test_weights_are_a_distribution():
    """P6: weights are non-negative and sum to one."""
    rng = np.random.default_rng(6)
    L, d = 1000, 128
    k = rand_bits(rng, (L, 1, d), 2.0)
    q = rand_bits(rng, (1, 2, d), 2.0)
    for h in range(2):
        w = oracle.attn_weights(q, k, [0], [L], 1 / math.sqrt(d), 0, h)
        assert w.shape == (L,)
        assert (w >= 0).all()
        assert abs(w.sum() - 1.0) <= 1e-12


def test_values_enter_linearly():
    """out(2 V) = 2 out(V) exactly (doubling a bf16 is exact)."""
    rng = np.random.default_rng(15)
    L, d = 77, 128
    k = rand_bits(rng, (L, 1, d))
    v = rand_bits(rng, (L, 1, d))
    v2 = bf(unbf(v) * np.float32(2.0))
    q = rand_bits(rng, (1, 2, d))
    np.testing.assert_array_equal(single(q, k, v2, 0.2), 2.0 * single(q, k, v, 0.2))


def test_spike_retrieval_with_huge_logits():
    """P9: one key per (sequence, KV head) gets a logit about 1000 above the rest,
    so its V row is returned.  Logits this large also overflow exp() unless the
    maximum is subtracted first (a missing stabilisation gives NaN)."""
    rng = np.random.default_rng(10)
    d, hkv, hq, nseq = 128, 2, 4, 3
    lens = np.array([40, 17, 64])
    offs = np.array([100, 0, 20])
    rows = 140
    k = rand_bits(rng, (rows, hkv, d), 0.01)
    # V rows hold codes of (row, kv, dim), exact in bf16
    code = (np.arange(rows)[:, None, None] * 4 + np.arange(hkv)[None, :, None]) % 251
    v = bf((code + np.arange(d)[None, None, :] % 3).astype(np.float32))
    q = np.full((nseq, hq, d), bf(np.array([1.0], np.float32))[0], np.uint16)
    star = {}
    for b in range(nseq):
        for kv in range(hkv):
            t = int(rng.integers(0, lens[b]))
            star[(b, kv)] = offs[b] + t
            k[offs[b] + t, kv] = bf(np.array([96.0], np.float32))[0]
    out = oracle.decode_attn(q, k, v, offs, lens, 0.0884)
    assert np.isfinite(out).all()
    for b in range(nseq):
        for h in range(hq):
            kv = h // 2
            np.testing.assert_allclose(out[b, h], unbf(v[star[(b, kv)], kv]), rtol=0, atol=1e-9)


def test_gqa_head_mapping():
    """P12: V = kv index on each KV head -> out[b, h, :] = floor(h / g).
    Catches h % Hkv (interleaved) instead of h // g (consecutive) sharing."""
    rng = np.random.default_rng(12)
    d, hkv, hq = 128, 4, 16
    L = 33
    k = rand_bits(rng, (L, hkv, d))
    v = np.zeros((L, hkv, d), np.uint16)
    for kv in range(hkv):
        v[:, kv] = bf(np.array([float(kv)], np.float32))[0]
    q = rand_bits(rng, (2, hq, d))
    out = oracle.decode_attn(q, k, v, [0, 5], [L, L - 5], 0.09)
    for h in range(hq):
        np.testing.assert_allclose(out[:, h], float(h // (hq // hkv)), rtol=1e-14, atol=1e-14)


def test_placement_independence_and_poison():
    """P10/P11: a sequence's output depends only on its own rows: shuffled
    regions with NaN-filled gaps and NaN rows past each length give the same
    result as each sequence alone at offset 0."""
    rng = np.random.default_rng(11)
    w = wl.Workload("t", 90, 1, 5, 8, 2, 3, "uniform", 1, 50)
    lens = np.array([1, 15, 16, 17, 49], np.int32)
    lay = wl.make_layout(lens, steps=3, gap_max=7, shuffle=True, rng=rng)
    k, v = wl.layer_kv_bits(w, lay, 0, fill=wl.BF16_NAN)
    for b in range(5):  # rows past L_b inside the capacity: poison too
        k[lay.offsets[b] + lens[b]: lay.offsets[b] + lay.capacity[b]] = wl.BF16_NAN
        v[lay.offsets[b] + lens[b]: lay.offsets[b] + lay.capacity[b]] = wl.BF16_NAN
    q = wl.query_bits(w, 0)
    out = oracle.decode_attn(q, k, v, lay.offsets, lens, w.scale)
    assert np.isfinite(out).all()
    for b in range(5):
        o, L = lay.offsets[b], lens[b]
        alone = oracle.decode_attn(q[b:b + 1], k[o:o + L], v[o:o + L], [0], [L], w.scale)
        np.testing.assert_array_equal(out[b], alone[0])


def test_empty_sequence_gives_zeros():
    rng = np.random.default_rng(13)
    k = rand_bits(rng, (4, 1, 128))
    v = rand_bits(rng, (4, 1, 128))
    q = rand_bits(rng, (2, 2, 128))
    out = oracle.decode_attn(q, k, v, [0, 3], [0, 1], 0.1)
    assert (out[0] == 0).all()
    np.testing.assert_array_equal(out[1, 0], unbf(v[3, 0]))


def test_rejects_out_of_range_rows():
    rng = np.random.default_rng(16)
    k = rand_bits(rng, (4, 1, 128))
    q = rand_bits(rng, (1, 1, 128))
    with pytest.raises(ValueError):
        oracle.decode_attn(q, k, k, [2], [3], 0.1)


# ------------------------------------------------------------- brute force

def brute_force(q, k, v, offs, lens, scale):
    """Pure-Python float64: weights exp(s_t) / sum_u exp(s_u) without the max
    shift, sums with math.fsum (exactly rounded).  Logits are kept small so
    the unshifted form cannot overflow."""
    qf, kf, vf = (unbf(x).astype(np.float64).tolist() for x in (q, k, v))
    B, hq, d = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    out = np.zeros((B, hq, d))
    for b in range(B):
        for h in range(hq):
            kv = h // g
            rows = range(offs[b], offs[b] + lens[b])
            e = [math.exp(scale * math.fsum(qf[b][h][i] * kf[r][kv][i] for i in range(d))) for r in rows]
            z = math.fsum(e)
            for i in range(d):
                out[b, h, i] = math.fsum(e[j] * vf[r][kv][i] for j, r in enumerate(rows)) / z if e else 0.0
    return out


@pytest.mark.parametrize("B,hq,hkv,d", [(1, 2, 1, 4), (3, 4, 2, 4), (2, 4, 1, 128), (3, 2, 2, 128)])
def test_brute_force_tiny(B, hq, hkv, d):
    """P7: at tiny sizes the oracle agrees with an independent pure-Python
    evaluation to 1e-12."""
    rng = np.random.default_rng(B * 100 + hq * 10 + d)
    lens = rng.integers(1, 18, size=B)
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]) + np.arange(B)
    rows = int(offs[-1] + lens[-1] + 1)
    k = rand_bits(rng, (rows, hkv, d))
    v = rand_bits(rng, (rows, hkv, d))
    q = rand_bits(rng, (B, hq, d))
    scale = 1 / math.sqrt(d)
    np.testing.assert_allclose(oracle.decode_attn(q, k, v, offs, lens, scale),
                               brute_force(q, k, v, offs, lens, scale), rtol=0, atol=1e-12)


def test_threads_do_not_change_results():
    rng = np.random.default_rng(17)
    w = wl.WORKLOADS["tiny"]
    lay = wl.make_layout(wl.draw_lengths(w) // 8, 1)
    k = rand_bits(rng, (lay.num_rows, w.num_kv_heads, 128))
    v = rand_bits(rng, (lay.num_rows, w.num_kv_heads, 128))
    q = wl.query_bits(w, 0)
    a = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale, threads=1)
    b = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale, threads=4)
    np.testing.assert_array_equal(a, b)
    pairs = np.array([[3, 15], [0, 0], [2, 7]])
    np.testing.assert_array_equal(oracle.decode_attn_pairs(q, k, v, lay.offsets, lay.lens, w.scale, pairs),
                                  a[pairs[:, 0], pairs[:, 1]])


# ------------------------------------------------------------- paged caches

def _paged_copy(k, v, lay, page_tokens, rng, spare_pages=5):
    """Scatter every sequence's rows into randomly chosen pages; unused slots
    and pages hold NaN.  Returns pages and block tables."""
    caps = [int(c) for c in lay.capacity]
    npages_seq = [-(-c // page_tokens) for c in caps]
    total = sum(npages_seq) + spare_pages
    perm = rng.permutation(total)
    hkv, d = k.shape[1], k.shape[2]
    kp = np.full((total, page_tokens, hkv, d), wl.BF16_NAN, np.uint16)
    vp = np.full_like(kp, wl.BF16_NAN)
    bt = np.full((len(caps), max(npages_seq) + 2), -1, np.int32)
    nxt = 0
    for b, cap in enumerate(caps):
        o = int(lay.offsets[b])
        for j in range(npages_seq[b]):
            page = perm[nxt]
            nxt += 1
            bt[b, j] = page
            n = min(page_tokens, cap - j * page_tokens)
            kp[page, :n] = k[o + j * page_tokens: o + j * page_tokens + n]
            vp[page, :n] = v[o + j * page_tokens: o + j * page_tokens + n]
    return kp, vp, bt


@pytest.mark.parametrize("page_tokens", [16, 32, 48])
def test_paged_oracle_equals_contiguous(page_tokens):
    """The block-table indirection changes where rows live, not what is
    computed: scattered pages with NaN everywhere else give exactly the
    contiguous oracle's output."""
    rng = np.random.default_rng(31 + page_tokens)
    w = wl.Workload("pg", 91, 1, 7, 16, 4, 3, "uniform", 1, 200)
    lens = wl.draw_lengths(w)
    lens[:3] = [1, page_tokens, page_tokens + 1]
    lay = wl.make_layout(lens, steps=3)
    k, v = wl.layer_kv_bits(w, lay, 0)
    q = wl.query_bits(w, 0)
    ref = oracle.decode_attn(q, k, v, lay.offsets, lens, w.scale)
    kp, vp, bt = _paged_copy(k, v, lay, page_tokens, rng)
    got = oracle.decode_attn_paged(q, kp, vp, bt, lens, w.scale)
    np.testing.assert_array_equal(got, ref)


def test_paged_append_uses_the_new_token():
    """With k_new / v_new the newest token's cache slot is ignored (it holds NaN
    here) and the new rows are attended instead: identical to the contiguous
    oracle on a cache where that row was written."""
    rng = np.random.default_rng(41)
    w = wl.Workload("pa", 92, 1, 6, 8, 2, 1, "uniform", 1, 90)
    lens = wl.draw_lengths(w)
    lens[0] = 1
    lay = wl.make_layout(lens, steps=1)
    k, v = wl.layer_kv_bits(w, lay, 0)
    q = wl.query_bits(w, 0)
    k_new = rand_bits(rng, (6, 2, 128))
    v_new = rand_bits(rng, (6, 2, 128))
    k2, v2 = k.copy(), v.copy()
    for b in range(6):
        r = lay.offsets[b] + lens[b] - 1
        k2[r], v2[r] = k_new[b], v_new[b]
        k[r] = wl.BF16_NAN
        v[r] = wl.BF16_NAN
    ref = oracle.decode_attn(q, k2, v2, lay.offsets, lens, w.scale)
    kp, vp, bt = _paged_copy(k, v, lay, 16, rng)
    got = oracle.decode_attn_paged(q, kp, vp, bt, lens, w.scale, k_new, v_new)
    np.testing.assert_array_equal(got, ref)
    # without the append the NaN slot is read
    assert np.isnan(oracle.decode_attn_paged(q, kp, vp, bt, lens, w.scale)).any()


def test_paged_rejects_bad_block_tables():
    rng = np.random.default_rng(42)
    kp = rand_bits(rng, (3, 16, 1, 128))
    q = rand_bits(rng, (1, 1, 128))
    with pytest.raises(ValueError):
        oracle.decode_attn_paged(q, kp, kp, np.array([[0, 7]], np.int32), [20], 0.1)
    with pytest.raises(ValueError):
        oracle.decode_attn_paged(q, kp, kp, np.array([[0]], np.int32), [20], 0.1)


# ------------------------------------------------------------- causal prefill

def test_prefill_rows_are_decodes_of_growing_prefixes():
    """Query i of a sequence with L rows and n new tokens is the decode of the
    first L - n + i + 1 rows: checked against the pinned decode path, with
    sequences and query rows in shuffled places."""
    rng = np.random.default_rng(61)
    hq, hkv, d = 8, 2, 128
    lens = np.array([1, 20, 33, 7], np.int32)
    qlen = np.array([1, 5, 33, 0], np.int32)
    lay = wl.make_layout(lens, 1, gap_max=3, shuffle=True, rng=rng)
    k = rand_bits(rng, (lay.num_rows, hkv, d))
    v = rand_bits(rng, (lay.num_rows, hkv, d))
    q_starts = np.array([40, 0, 6, 39], np.int32)
    q = rand_bits(rng, (80, hq, d))
    out = oracle.prefill_attn(q, k, v, lay.offsets, lens, q_starts, qlen, 0.09)
    for b in range(4):
        for i in range(qlen[b]):
            row = q_starts[b] + i
            dec = oracle.decode_attn(q[row:row + 1], k, v, [lay.offsets[b]], [lens[b] - qlen[b] + i + 1], 0.09)
            np.testing.assert_array_equal(out[row], dec[0])
    untouched = np.ones(80, bool)
    for b in range(4):
        untouched[q_starts[b]:q_starts[b] + qlen[b]] = False
    assert (out[untouched] == 0).all()


def test_prefill_is_causal():
    """Changing a later token's K/V never changes an earlier query's output;
    the first new query of a fresh sequence (L = n) sees only itself."""
    rng = np.random.default_rng(62)
    L = 24
    k = rand_bits(rng, (L, 1, 128))
    v = rand_bits(rng, (L, 1, 128))
    q = rand_bits(rng, (L, 2, 128))
    a = oracle.prefill_attn(q, k, v, [0], [L], [0], [L], 0.1)
    k2, v2 = k.copy(), v.copy()
    k2[15:] = rand_bits(rng, (L - 15, 1, 128))
    v2[15:] = rand_bits(rng, (L - 15, 1, 128))
    b = oracle.prefill_attn(q, k2, v2, [0], [L], [0], [L], 0.1)
    np.testing.assert_array_equal(a[:15], b[:15])
    assert not np.array_equal(a[15:], b[15:])
    np.testing.assert_array_equal(a[0, 0], unbf(v[0, 0]).astype(np.float64))


def test_prefill_rejects_bad_lengths():
    rng = np.random.default_rng(63)
    k = rand_bits(rng, (8, 1, 128))
    q = rand_bits(rng, (4, 1, 128))
    with pytest.raises(ValueError):
        oracle.prefill_attn(q, k, k, [0], [3], [0], [4], 0.1)   # more queries than tokens
    with pytest.raises(ValueError):
        oracle.prefill_attn(q, k, k, [0], [8], [2], [3], 0.1)   # query rows past q


# ---------------------------------------------------------------- OPD token loss
# App. OPD Optimization: eq:opd-token-advantage, eq:opd-ratio, eq:opd-dual-clip,
# eq:opd-surrogate (delta = 0.2, kappa = 3, ratio clip 20, eps = 1e-8).

def _one_hot_rows(n, vocab=4):
    """Rows whose token 0 has log-probability 0 to far below double rounding."""
    z = np.full((n, vocab), -100.0)
    z[:, 0] = 0.0
    return z


# (A, rho, token loss, d loss / d rho * rho) from the cases of eq:opd-dual-clip, by hand
OPD_REGIMES = [
    (0.5, 0.5, -0.25, -0.25),        # A > 0, below the band: rho A selected
    (0.5, 1.1, -0.55, -0.55),        # A > 0, inside the band
    (0.5, 1.5, -0.6, 0.0),           # A > 0, above the band: clip(rho) A = 1.2 A, flat
    (-0.5, 0.5, 0.4, 0.0),           # A < 0, below the band: clip(rho) A = 0.8 A, flat
    (-0.5, 1.1, 0.55, 0.55),         # A < 0, inside the band
    (-0.5, 2.0, 1.0, 1.0),           # A < 0, above the band, under the dual clip
    (-0.5, 4.0, 1.5, 0.0),           # A < 0, dual clip kappa |A| = 1.5, flat
    (0.0, 2.0, 0.0, 0.0),            # A = 0
]


def _regime_batch(cases, per_seq=1):
    n = len(cases)
    old = np.array([-np.log(rho) for _, rho, _, _ in cases], np.float32)
    tea = (old.astype(np.float64) + np.array([a for a, _, _, _ in cases])).astype(np.float32)
    starts = np.arange(0, n + 1, per_seq, dtype=np.int32)
    return _one_hot_rows(n), np.zeros(n, np.int32), old, tea, np.ones(n, np.uint8), starts


def test_opd_regimes_closed_form():
    z, tok, old, tea, m, st = _regime_batch(OPD_REGIMES)
    r = oracle.opd_loss(z, tok, old, tea, m, st)
    n = len(OPD_REGIMES)
    np.testing.assert_allclose(r["token_loss"], [c[2] for c in OPD_REGIMES], rtol=0, atol=1e-6)
    w = 1.0 / (n * (1 + 1e-8))
    np.testing.assert_allclose(r["weight"], w, rtol=1e-12)
    np.testing.assert_allclose(r["dlp"], [w * c[3] for c in OPD_REGIMES], rtol=0, atol=1e-7)
    np.testing.assert_allclose(r["lp"], 0.0, atol=1e-30)


def test_opd_ratio_clip_at_20():
    # lp - old = 25 is clipped to 20 (eq:opd-ratio): rho = e^20, no gradient through rho
    # lp - old = -25 clips to -20: rho = e^-20, below the band, where the loss
    # -rho A has a slope in rho, yet no gradient reaches lp through the clip
    z = _one_hot_rows(3)
    old = np.array([-25.0, -25.0, 25.0], np.float32)
    tea = old + np.array([0.5, -0.5, 0.5], np.float32)
    r = oracle.opd_loss(z, [0, 0, 0], old, tea, [1, 1, 1], [0, 1, 2, 3])
    np.testing.assert_allclose(r["token_loss"], [-0.6, 1.5, -0.5 * math.exp(-20)], rtol=1e-6, atol=1e-6)
    assert (r["dlp"] == 0).all()
    # just inside the clip the ratio carries gradient again: l = -1.2 A flat for A > 0,
    # but for A < 0 above the band the dual clip is flat too; use A < 0 below kappa
    z2 = _one_hot_rows(1)
    old2 = np.array([-np.log(2.0)], np.float32)
    r2 = oracle.opd_loss(z2, [0], old2, old2 - np.float32(0.5), [1], [0, 1])
    assert r2["dlp"][0] > 0


def test_opd_seq_mean_token_mean():
    # response 0: one token with loss -0.25; response 1: three tokens 0.4, 0.55, 1.0
    # seq-mean-token-mean = (-0.25 + 1.95 / 3) / 2 = 0.2 (token mean would be 0.425)
    cases = [OPD_REGIMES[0], OPD_REGIMES[3], OPD_REGIMES[4], OPD_REGIMES[5]]
    z, tok, old, tea, m, _ = _regime_batch(cases)
    r = oracle.opd_loss(z, tok, old, tea, m, [0, 1, 4])
    assert r["loss"] == pytest.approx(0.2, abs=1e-6)
    np.testing.assert_allclose(r["weight"], [0.5 / (1 + 1e-8)] + [0.5 / (3 + 1e-8)] * 3, rtol=1e-12)


def test_opd_masked_tokens_are_excluded():
    # inserted tokens stay in the context but carry no loss and no normalisation;
    # their rows are never read (NaN logits, garbage log-probs)
    cases = [OPD_REGIMES[0], OPD_REGIMES[3], OPD_REGIMES[4], OPD_REGIMES[5]]
    z, tok, old, tea, m, _ = _regime_batch(cases)
    z = np.insert(z, [2, 4], np.nan, axis=0)
    tok = np.insert(tok, [2, 4], 3)
    old = np.insert(old, [2, 4], np.float32(7.0))
    tea = np.insert(tea, [2, 4], np.float32(-9.0))
    m = np.insert(m, [2, 4], 0)
    zb = wl.f32_to_bf16_bits(z.astype(np.float32))
    r = oracle.opd_loss(zb, tok, old, tea, m, [0, 1, 6])
    assert r["loss"] == pytest.approx(0.2, abs=1e-5)
    for j in (2, 5):
        assert r["token_loss"][j] == 0 and r["dlp"][j] == 0 and r["lp"][j] == 0 and r["weight"][j] == 0
    g = oracle.opd_grad_rows(zb, tok, m, r["dlp"], [2, 5])
    assert (g == 0).all()


def test_opd_fully_masked_response_counts_in_the_batch():
    # 0 / (0 + eps) = 0 for a response with no supervised token, and |B| grows
    cases = [OPD_REGIMES[0], OPD_REGIMES[3], OPD_REGIMES[4], OPD_REGIMES[5], OPD_REGIMES[1]]
    z, tok, old, tea, m, _ = _regime_batch(cases)
    m[4] = 0
    r = oracle.opd_loss(z, tok, old, tea, m, [0, 1, 4, 5])
    assert r["loss"] == pytest.approx(0.2 * 2 / 3, abs=1e-6)
    r0 = oracle.opd_loss(z, tok, old, tea, m, [0, 1, 4, 4, 5])  # and an empty response
    assert r0["loss"] == pytest.approx(0.2 * 2 / 4, abs=1e-6)


def test_opd_logprob_is_log_softmax():
    from scipy.special import logsumexp

    rng = np.random.default_rng(3)
    zb = wl.f32_to_bf16_bits((3 * rng.standard_normal((8, 1000))).astype(np.float32))
    z = wl.bf16_bits_to_f32(zb).astype(np.float64)
    tok = rng.integers(0, 1000, 8).astype(np.int32)
    r = oracle.opd_loss(zb, tok, np.zeros(8, np.float32), np.zeros(8, np.float32), np.ones(8, np.uint8),
                        [0, 8])
    np.testing.assert_allclose(r["lp"], z[np.arange(8), tok] - logsumexp(z, axis=1), rtol=0, atol=1e-12)


def _fd_batch(rng, n, vocab, rhos, advs):
    zb = wl.f32_to_bf16_bits(rng.standard_normal((n, vocab)).astype(np.float32))
    z = wl.bf16_bits_to_f32(zb).astype(np.float64)
    tok = rng.integers(0, vocab, n).astype(np.int32)
    m = np.ones(n, np.uint8)
    lp = oracle.opd_loss(z, tok, np.zeros(n, np.float32), np.zeros(n, np.float32), m, [0, n])["lp"]
    old = (lp - np.log(rhos)).astype(np.float32)
    tea = (old.astype(np.float64) + advs).astype(np.float32)
    return zb, z, tok, old, tea, m


def test_opd_gradient_matches_finite_differences():
    # rho values away from the kinks (0.8, 1.2, 3) cover every regime
    rng = np.random.default_rng(5)
    rhos = np.array([0.5, 1.05, 1.6, 0.6, 0.95, 2.0, 5.0, 1.1])
    advs = np.array([0.7, 0.7, 0.7, -0.6, -0.6, -0.6, -0.6, 0.0])
    n, vocab = len(rhos), 7
    zb, z, tok, old, tea, m = _fd_batch(rng, n, vocab, rhos, advs)
    st = [0, 3, 8]
    base = oracle.opd_loss(zb, tok, old, tea, m, st)
    grad = oracle.opd_grad_rows(zb, tok, m, base["dlp"], np.arange(n))
    h = 1e-6
    fd = np.zeros_like(z)
    for j in range(n):
        for v in range(vocab):
            zp, zm = z.copy(), z.copy()
            zp[j, v] += h
            zm[j, v] -= h
            fd[j, v] = (oracle.opd_loss(zp, tok, old, tea, m, st)["loss"]
                        - oracle.opd_loss(zm, tok, old, tea, m, st)["loss"]) / (2 * h)
    np.testing.assert_allclose(grad, fd, rtol=0, atol=1e-8)
    assert np.abs(grad).max() > 1e-3  # some rows carry gradient
    # flat regimes: no gradient at all
    flat = [2, 3, 6, 7]
    assert np.abs(grad[flat]).max() == 0


def test_opd_logit_shift_invariance():
    rng = np.random.default_rng(6)
    zb, z, tok, old, tea, m = _fd_batch(rng, 6, 50, np.array([0.5, 1.1, 2.0, 0.9, 4.0, 1.3]),
                                        np.array([0.3, -0.4, -0.2, 0.1, -0.5, 0.6]))
    a = oracle.opd_loss(z, tok, old, tea, m, [0, 2, 6])
    b = oracle.opd_loss(z + rng.standard_normal((6, 1)) * 10, tok, old, tea, m, [0, 2, 6])
    np.testing.assert_allclose(b["lp"], a["lp"], atol=1e-12)
    assert b["loss"] == pytest.approx(a["loss"], abs=1e-12)


def test_opd_rejects_bad_inputs():
    z = _one_hot_rows(2)
    ok = dict(tokens=[0, 0], old_lp=[0, 0], tea_lp=[0, 0], mask=[1, 1], seq_starts=[0, 2])
    oracle.opd_loss(z, **ok)
    with pytest.raises(ValueError):
        oracle.opd_loss(z, **{**ok, "tokens": [0, 4]})
    with pytest.raises(ValueError):
        oracle.opd_loss(z, **{**ok, "seq_starts": [0, 1]})
    with pytest.raises(ValueError):
        oracle.opd_loss(z, **{**ok, "seq_starts": [1, 2]})
    oracle.opd_loss(z, **{**ok, "tokens": [0, 4], "mask": [1, 0]})  # masked rows are not read


# ---------------------------------------------------------------- rollout scheduler
# Prop. 1 (eq:ideal-rollout-speedup), App. finite concurrency
# (eq:finite-capacity-time-bound), the calibrated estimate
# (eq:calibrated-rollout-speedup).

from oracle import oracle_sched as sch  # noqa: E402


def _uniform(n, turns, value):
    return [[value] * turns for _ in range(n)]


@pytest.mark.parametrize("n,turns,lf,lu", [(1, 1, 1.0, 8.0), (4, 30, 1.0, 8.0), (16, 8, 0.5, 2.0), (3, 5, 2.0, 2.0)])
def test_sched_prop1_with_enough_slots(n, turns, lf, lu):
    """With a slot for every request (2NT) no request waits: Vanilla takes
    T l_full and ActFirst (T - 1) l_fast + l_full (Prop. 1).  (2N slots are not
    enough: ActFirst keeps up to about l_full / l_fast full responses of a task
    in flight.)"""
    van = sch.simulate_latency(sch.VANILLA, _uniform(n, turns, lf), _uniform(n, turns, lu), 2 * n * turns)
    act = sch.simulate_latency(sch.ACTFIRST, _uniform(n, turns, lf), _uniform(n, turns, lu), 2 * n * turns)
    assert van["completion"] == pytest.approx(turns * lu)
    assert act["completion"] == pytest.approx((turns - 1) * lf + lu)
    s = van["completion"] / act["completion"]
    assert s == pytest.approx(sch.ideal_speedup(turns, lf, lu))
    assert 1.0 - 1e-12 <= s <= min(turns, lu / lf) + 1e-12


def test_sched_ideal_speedup_values():
    # T l_full / ((T-1) l_fast + l_full): by hand
    assert sch.ideal_speedup(1, 1.0, 8.0) == 1.0
    assert sch.ideal_speedup(30, 1.0, 8.0) == pytest.approx(240.0 / 37.0)
    assert sch.ideal_speedup(10 ** 9, 1.0, 8.0) == pytest.approx(8.0, rel=1e-7)  # the T -> infinity limit
    assert sch.ideal_speedup(4, 2.0, 2.0) == 1.0                                  # equal latencies: no gain


def test_sched_calibrated_estimate():
    """Per-task constant latencies, unrestricted overlap: the batch waits for
    its slowest task (eq:calibrated-rollout-speedup), including a task whose
    fast action is slower than its full response."""
    lf = [1.0, 0.5, 3.0, 0.2]
    lu = [4.0, 6.0, 2.0, 1.0]
    turns = 7
    fast = [[a] * turns for a in lf]
    full = [[b] * turns for b in lu]
    van = sch.simulate_latency(sch.VANILLA, fast, full, 1000)
    act = sch.simulate_latency(sch.ACTFIRST, fast, full, 1000)
    assert van["completion"] == pytest.approx(max(turns * b for b in lu))          # 42
    assert act["completion"] == pytest.approx(max((turns - 1) * a + max(a, b) for a, b in zip(lf, lu)))  # 21
    assert sch.calibrated_completion(sch.VANILLA, lf, lu, turns) == pytest.approx(42.0)
    assert sch.calibrated_completion(sch.ACTFIRST, lf, lu, turns) == pytest.approx(21.0)


def test_sched_schedule_by_hand():
    """N = 2, T = 2, l_fast = 1, l_full = 3, FIFO admission (submission time,
    task, turn, fast before full).  One slot: Vanilla serves 0/0 [0,3], 1/0
    [3,6], 0/1 [6,9], 1/1 [9,12]; ActFirst serves 0/0 fast [0,1], 0/0 full
    [1,4], 1/0 fast [4,5], 1/0 full [5,8], 0/1 fast [8,9], 0/1 full [9,12],
    1/1 fast [12,13], 1/1 full [13,16].  Four slots: Vanilla 6; ActFirst admits
    all four turn-0 requests at 0, task 0's turn-1 pair at 1 (two slots free),
    task 1's turn-1 fast at 2 and its full at 3 -> 6.  Eight slots: 4."""
    fast, full = _uniform(2, 2, 1.0), _uniform(2, 2, 3.0)
    van = sch.simulate_latency(sch.VANILLA, fast, full, 1)
    act = sch.simulate_latency(sch.ACTFIRST, fast, full, 1)
    assert van["completion"] == 12.0 and act["completion"] == 16.0
    assert [van["start"][(i, t, 1)] for i, t in [(0, 0), (1, 0), (0, 1), (1, 1)]] == [0.0, 3.0, 6.0, 9.0]
    want = {(0, 0, 0): 0, (0, 0, 1): 1, (1, 0, 0): 4, (1, 0, 1): 5, (0, 1, 0): 8, (0, 1, 1): 9,
            (1, 1, 0): 12, (1, 1, 1): 13}
    assert {k: act["start"][k] for k in want} == {k: float(v) for k, v in want.items()}
    assert sch.simulate_latency(sch.VANILLA, fast, full, 4)["completion"] == 6.0
    a4 = sch.simulate_latency(sch.ACTFIRST, fast, full, 4)
    assert a4["completion"] == 6.0
    assert (a4["start"][(0, 1, 0)], a4["start"][(1, 1, 0)], a4["start"][(1, 1, 1)]) == (1.0, 2.0, 3.0)
    assert sch.simulate_latency(sch.ACTFIRST, fast, full, 8)["completion"] == 4.0
    assert act["peak"] == 1 and van["peak"] == 1


def test_sched_finite_concurrency_bounds():
    """For any cap, ActFirst's completion respects the dependency chain and the
    slot-time bound (eq:finite-capacity-time-bound); the speedup respects
    eq:finite-capacity-speedup; admitted requests never exceed the cap."""
    rng = np.random.default_rng(8)
    for _ in range(40):
        n, turns = int(rng.integers(1, 6)), int(rng.integers(1, 7))
        lf, lu = float(rng.uniform(0.1, 2)), float(rng.uniform(0.1, 5))
        b = int(rng.integers(1, 2 * n + 2))
        van = sch.simulate_latency(sch.VANILLA, _uniform(n, turns, lf), _uniform(n, turns, lu), b)
        act = sch.simulate_latency(sch.ACTFIRST, _uniform(n, turns, lf), _uniform(n, turns, lu), b)
        lower = sch.completion_lower_bound(n, turns, lf, lu, b)
        assert act["completion"] >= lower - 1e-9
        assert van["completion"] / act["completion"] <= van["completion"] / lower + 1e-9
        assert act["peak"] <= b and van["peak"] <= b
        # dependencies: a turn's requests start no earlier than the gating request of the turn before
        for i in range(n):
            for t in range(1, turns):
                assert act["start"][(i, t, 0)] >= act["end"][(i, t - 1, 0)] - 1e-12
                assert van["start"][(i, t, 1)] >= van["end"][(i, t - 1, 1)] - 1e-12


@pytest.mark.parametrize("b_max", [1, 2, 3, 5, 100])
def test_sched_engine_with_constant_steps_equals_latency_model(b_max):
    """With a constant step cost the engine model reduces to the latency model
    with l = output tokens x step, for any cap."""
    rng = np.random.default_rng(b_max)
    n, turns = 3, 4
    ctx = [[int(rng.integers(10, 50)) for _ in range(turns)] for _ in range(n)]
    for policy in (sch.VANILLA, sch.ACTFIRST):
        e = sch.simulate_engine(policy, ctx, 2, 7, b_max, base=0.5, per_kv=0.0, prefill=0.0)
        lat = sch.simulate_latency(policy, _uniform(n, turns, 1.0), _uniform(n, turns, 3.5), b_max)
        assert e["completion"] == pytest.approx(lat["completion"])
        for k, v in lat["start"].items():
            assert e["start"][k] == pytest.approx(v)


def test_sched_engine_by_hand():
    """One task, one turn, context 4 tokens, fast 2 and full 3 output tokens,
    step = 1 + 0.5 x KV tokens + 0.25 x newly prefilled tokens.
    Vanilla: 1 + 0.5*4 + 0.25*4 = 4, then 1 + 0.5*5 = 3.5, then 1 + 0.5*6 = 4 -> 11.5.
    ActFirst (both admitted at 0): 1 + 0.5*8 + 0.25*8 = 7, 1 + 0.5*10 = 6, 1 + 0.5*6 = 4 -> 17;
    the fast action ends at 13."""
    v = sch.simulate_engine(sch.VANILLA, [[4]], 2, 3, 8, base=1.0, per_kv=0.5, prefill=0.25)
    a = sch.simulate_engine(sch.ACTFIRST, [[4]], 2, 3, 8, base=1.0, per_kv=0.5, prefill=0.25)
    assert v["completion"] == 11.5 and v["steps"] == 3
    assert a["completion"] == 17.0 and a["end"][(0, 0, 0)] == 13.0

"""Indexing exactness, split handling, determinism, output dtype, ABI errors and
HIP-graph replay of the HIP path (through the C ABI)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import CtxError, DecodeAttention

from _gpu_util import assert_parity, dev, up_bf16, up_i32

pytestmark = pytest.mark.gpu

bf = wl.f32_to_bf16_bits
unbf = wl.bf16_bits_to_f32


def run(hq, hkv, q, k, v, offs, lens, scale, split_tokens=0, out_dtype=torch.float32,
        max_seq_len=None, canary=False):
    b = len(lens)
    msl = max_seq_len or max(int(np.max(lens)) if b else 1, 1)
    with DecodeAttention(hq, hkv, max(b, 1), msl, out_dtype=out_dtype, split_tokens=split_tokens) as attn:
        buf = torch.full((b + 1, hq, 128), -12345.0, dtype=out_dtype, device=dev())
        out = buf[:b]
        attn.run(up_bf16(q), up_bf16(k), up_bf16(v), up_i32(offs), up_i32(lens), scale, out)
        torch.cuda.synchronize()
        if canary:
            assert (buf[b] == -12345.0).all(), "write past the end of out"
        return out.float().cpu().numpy()


def rand_bits(rng, shape, scale=1.0):
    return bf(rng.standard_normal(shape).astype(np.float32) * np.float32(scale))


def test_poisoned_gaps_shuffled_regions_and_canary():
    """NaN in every row no sequence may read (gaps, slack past each length);
    regions shuffled; a canary row after out."""
    rng = np.random.default_rng(21)
    w = wl.Workload("poison", 120, 1, 24, 32, 8, 5, "uniform", 1, 700)
    lens = wl.draw_lengths(w)
    lens[:6] = [1, 15, 16, 17, 33, 700]
    lay = wl.make_layout(lens, steps=5, gap_max=40, shuffle=True, rng=rng)
    k, v = wl.layer_kv_bits(w, lay, 0, fill=wl.BF16_NAN)
    for b in range(w.batch):
        o = lay.offsets[b]
        k[o + lens[b]: o + lay.capacity[b]] = wl.BF16_NAN
        v[o + lens[b]: o + lay.capacity[b]] = wl.BF16_NAN
    q = wl.query_bits(w, 0)
    ref = oracle.decode_attn(q, k, v, lay.offsets, lens, w.scale)
    for split in (0, 16, 48):
        got = run(32, 8, q, k, v, lay.offsets, lens, w.scale, split_tokens=split,
                  max_seq_len=lay.max_seq_len, canary=True)
        assert_parity(got, ref, f"poison split={split}")


def test_spike_retrieval_exact_rows():
    """One key per (sequence, KV head) dominates by a huge logit; V rows hold
    integer codes of (row, head, dim), so out must equal the code of exactly
    that row: a wrong row, head or offset is obvious."""
    rng = np.random.default_rng(22)
    hq, hkv, d = 32, 8, 128
    lens = np.array([1, 5, 16, 17, 100, 513, 1024, 2049], np.int32)
    lay = wl.make_layout(lens, 1, gap_max=9, shuffle=True, rng=rng)
    k = rand_bits(rng, (lay.num_rows, hkv, d), 0.01)
    code = (np.arange(lay.num_rows)[:, None, None] * 8 + np.arange(hkv)[None, :, None]) % 255
    v = bf((code + (np.arange(d)[None, None, :] % 5) - 2).astype(np.float32))
    q = np.full((len(lens), hq, d), bf(np.array([1.0], np.float32))[0], np.uint16)
    star = {}
    for b in range(len(lens)):
        for kv in range(hkv):
            t = int(rng.integers(0, lens[b]))
            star[(b, kv)] = lay.offsets[b] + t
            k[lay.offsets[b] + t, kv] = bf(np.array([8.0], np.float32))[0]
    for split in (0, 16, 256):
        got = run(hq, hkv, q, k, v, lay.offsets, lens, 0.0884, split_tokens=split)
        for b in range(len(lens)):
            for h in range(hq):
                expect = unbf(v[star[(b, h // 4)], h // 4])
                np.testing.assert_allclose(got[b, h], expect, rtol=0, atol=1e-3,
                                           err_msg=f"b={b} h={h} split={split}")


def test_gqa_mapping_exact():
    """V = kv index on each KV head -> out[b, h, :] = h // g for every group size.
    Odd head counts leave the last pair of heads of the merge with one head,
    and odd group sizes put a pair's two heads on different KV heads."""
    rng = np.random.default_rng(23)
    # Hkv 8, 4 -> four KV heads per workgroup; 2, 6 -> two; 1, 3, 7, 5 -> one
    for hq, hkv in [(32, 8), (16, 8), (8, 8), (16, 1), (32, 2), (64, 4), (12, 6), (12, 3), (9, 3), (7, 7),
                    (5, 1)]:
        lens = np.array([3, 40, 129], np.int32)
        lay = wl.make_layout(lens, 1)
        k = rand_bits(rng, (lay.num_rows, hkv, 128))
        v = np.zeros((lay.num_rows, hkv, 128), np.uint16)
        for kv in range(hkv):
            v[:, kv] = bf(np.array([float(kv)], np.float32))[0]
        q = rand_bits(rng, (3, hq, 128))
        g = hq // hkv
        for split in (0, 16):
            got = run(hq, hkv, q, k, v, lay.offsets, lens, 0.0884, split_tokens=split)
            for h in range(hq):
                np.testing.assert_allclose(got[:, h], float(h // g), rtol=1e-5, atol=1e-6,
                                           err_msg=f"{hq}/{hkv} h={h} split={split}")


def test_more_than_256_sequences():
    """300 sequences: the kernels scan the lengths 256 at a time, so the range
    search and the merge cross a chunk boundary; empty sequences sit at both
    ends of each chunk and a long one straddles the boundary."""
    rng = np.random.default_rng(29)
    hq, hkv = 32, 8
    lens = rng.integers(1, 400, size=300).astype(np.int32)
    lens[[0, 255, 256, 299]] = 0
    lens[[1, 254, 257]] = [1, 2500, 3]
    lay = wl.make_layout(lens, 1, gap_max=7, shuffle=True, rng=rng)
    k = rand_bits(rng, (lay.num_rows, hkv, 128))
    v = rand_bits(rng, (lay.num_rows, hkv, 128))
    q = rand_bits(rng, (len(lens), hq, 128))
    ref = oracle.decode_attn(q, k, v, lay.offsets, lens, 0.0884)
    for split in (0, 48):
        got = run(hq, hkv, q, k, v, lay.offsets, lens, 0.0884, split_tokens=split, max_seq_len=lay.max_seq_len,
                  canary=True)
        assert_parity(got, ref, f"300 sequences split={split}")
        assert (got[lens == 0] == 0).all(), "empty sequences must give zeros"


@pytest.mark.parametrize("C", [16, 64, 256])
def test_lengths_at_split_boundaries(C):
    rng = np.random.default_rng(24 + C)
    lens = np.array([1, C - 1, C, C + 1, 2 * C - 1, 2 * C, 2 * C + 1, 5 * C + 3, 4 * C], np.int32)
    lens = np.maximum(lens, 1)
    lay = wl.make_layout(lens, 1, gap_max=3, shuffle=True, rng=rng)
    k = rand_bits(rng, (lay.num_rows, 8, 128))
    v = rand_bits(rng, (lay.num_rows, 8, 128))
    q = rand_bits(rng, (len(lens), 32, 128))
    ref = oracle.decode_attn(q, k, v, lay.offsets, lens, 0.0884)
    for split in (C, 0):
        got = run(32, 8, q, k, v, lay.offsets, lens, 0.0884, split_tokens=split, canary=True)
        assert_parity(got, ref, f"C={C} split={split}")


def test_empty_and_single_row_sequences():
    rng = np.random.default_rng(25)
    lens = np.array([0, 1, 0, 2, 1, 0], np.int32)
    lay = wl.make_layout(np.maximum(lens, 1), 1)
    k = rand_bits(rng, (lay.num_rows, 8, 128))
    v = rand_bits(rng, (lay.num_rows, 8, 128))
    q = rand_bits(rng, (len(lens), 16, 128))
    for split in (0, 16):
        got = run(16, 8, q, k, v, lay.offsets, lens, 0.0884, split_tokens=split, max_seq_len=4)
        for b in np.nonzero(lens == 0)[0]:
            assert (got[b] == 0).all()
        for b in np.nonzero(lens == 1)[0]:
            for h in range(16):
                np.testing.assert_array_equal(got[b, h], unbf(v[lay.offsets[b], h // 2]))
    # a batch of nothing but empty sequences
    got = run(16, 8, q, k, v, lay.offsets, np.zeros(6, np.int32), 0.0884)
    assert (got == 0).all()


def test_split_invariance_and_determinism():
    w = wl.small_workload(wl.WORKLOADS["long_ragged"], batch=16, lengths=(17, 3000))
    lay = wl.workload_layout(w)
    q = wl.query_bits(w, 0)
    k, v = wl.layer_kv_bits(w, lay, 0)
    outs = {}
    for split in (0, 16, 64, 256, 1024, 4096):
        a = run(32, 8, q, k, v, lay.offsets, lay.lens, w.scale, split_tokens=split, max_seq_len=lay.max_seq_len)
        b = run(32, 8, q, k, v, lay.offsets, lay.lens, w.scale, split_tokens=split, max_seq_len=lay.max_seq_len)
        np.testing.assert_array_equal(a, b, err_msg=f"split={split} not deterministic")
        outs[split] = a
    for split, a in outs.items():
        np.testing.assert_allclose(a, outs[4096], rtol=0, atol=1e-5, err_msg=f"split={split}")


def test_repeated_runs_on_one_handle_are_bitwise_identical():
    w = wl.WORKLOADS["tiny"]
    lay = wl.workload_layout(w)
    q = up_bf16(wl.query_bits(w, 0))
    kh, vh = wl.layer_kv_bits(w, lay, 0)
    k, v = up_bf16(kh), up_bf16(vh)
    offs, lens = up_i32(lay.offsets), up_i32(lay.lens)
    with DecodeAttention(16, 8, 4, lay.max_seq_len) as attn:
        outs = []
        for _ in range(5):
            o = torch.empty((4, 16, 128), dtype=torch.float32, device=dev())
            attn.run(q, k, v, offs, lens, w.scale, o)
            outs.append(o)
        torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o, outs[0])


def test_bf16_output_is_rounded_fp32_result():
    w = wl.small_workload(wl.WORKLOADS["act_first_burst"], batch=16, lengths=(100, 900))
    lay = wl.workload_layout(w)
    q = wl.query_bits(w, 0)
    k, v = wl.layer_kv_bits(w, lay, 0)
    ref = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale)
    for split in (0, 64):
        f32 = run(32, 8, q, k, v, lay.offsets, lay.lens, w.scale, split_tokens=split, max_seq_len=lay.max_seq_len)
        b16 = run(32, 8, q, k, v, lay.offsets, lay.lens, w.scale, split_tokens=split,
                  out_dtype=torch.bfloat16, max_seq_len=lay.max_seq_len)
        np.testing.assert_array_equal(bf(b16.astype(np.float32)), bf(f32.astype(np.float32)))
        # within one bf16 ulp of the rounded oracle value, plus the fp32 path's
        # own rounding (which dominates for outputs near zero)
        ref_b = unbf(bf(ref.astype(np.float32))).astype(np.float64)
        ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref_b), 1e-30))) - 7)
        excess = np.abs(b16 - ref_b) - ulp
        assert excess.max() <= 2e-6, f"bf16 output {excess.max():.3e} beyond one ulp"
        assert (np.abs(b16 - ref_b) <= ulp).mean() > 0.999


# ----------------------------------------------------------------- ABI on GPU

def _raw(lib, h, *args):
    return lib.ctx_decode_attn_run(h, *args)


def test_abi_errors_on_device():
    lib = bd.load_library()
    attn = DecodeAttention(32, 8, 4, 256)
    h = attn.handle
    q = torch.zeros((5, 32, 128), dtype=torch.bfloat16, device=dev())
    kv = torch.zeros((64, 8, 128), dtype=torch.bfloat16, device=dev())
    out = torch.zeros((5, 32, 128), dtype=torch.float32, device=dev())
    offs = torch.zeros(5, dtype=torch.int32, device=dev())
    lens = torch.ones(5, dtype=torch.int32, device=dev())
    P = lambda t, off=0: t.data_ptr() + off  # noqa: E731
    args = lambda n=4, qo=0, ko=0, oo=0, scale=0.1: (P(q, qo), P(kv, ko), P(kv), P(offs), P(lens), n, scale, P(out, oo), None)  # noqa: E731
    assert _raw(lib, h, *args()) == bd.CTX_OK
    assert _raw(lib, h, *args(n=5)) == bd.CTX_ERR_CAPACITY
    assert _raw(lib, h, *args(n=-1)) == bd.CTX_ERR_INVALID_ARG
    assert _raw(lib, h, *args(qo=2)) == bd.CTX_ERR_ALIGNMENT
    assert _raw(lib, h, *args(ko=8)) == bd.CTX_ERR_ALIGNMENT
    assert _raw(lib, h, *args(oo=4)) == bd.CTX_ERR_ALIGNMENT
    assert _raw(lib, h, *args(scale=float("nan"))) == bd.CTX_ERR_INVALID_ARG
    assert _raw(lib, h, *args(scale=float("inf"))) == bd.CTX_ERR_INVALID_ARG
    assert _raw(lib, h, None, P(kv), P(kv), P(offs), P(lens), 4, 0.1, P(out), None) == bd.CTX_ERR_INVALID_ARG
    assert _raw(lib, h, P(q), P(kv), P(kv), P(offs), None, 4, 0.1, P(out), None) == bd.CTX_ERR_INVALID_ARG
    assert "aligned" in lib.ctx_decode_attn_last_error().decode() or lib.ctx_decode_attn_last_error()
    # zero sequences: nothing queued, OK even with NULL pointers
    assert _raw(lib, h, None, None, None, None, None, 0, 0.1, None, None) == bd.CTX_OK
    torch.cuda.synchronize()
    attn.close()
    with pytest.raises(CtxError):
        DecodeAttention(32, 8, 4, 256, head_dim=64)
    with pytest.raises(TypeError):
        DecodeAttention(16, 8, 4, 64).run(q.float(), kv, kv, offs, lens, 0.1, out)


def test_huge_workspace_reports_oom():
    lib = bd.load_library()
    # ~32 TB of split workspace: the allocation must fail cleanly
    d = bd.CtxDesc(32, 8, 128, 2_000_000_000, 1024, bd.CTX_DTYPE_F32, 0)
    h = ctypes.c_void_p()
    assert lib.ctx_decode_attn_create(ctypes.byref(d), ctypes.byref(h)) == bd.CTX_ERR_OOM
    assert h.value is None
    # a forced split too fine for the bounds is rejected before allocating
    d = bd.CtxDesc(32, 8, 128, 1 << 20, 1 << 30, bd.CTX_DTYPE_F32, 16)
    assert lib.ctx_decode_attn_create(ctypes.byref(d), ctypes.byref(h)) == bd.CTX_ERR_INVALID_ARG


def test_graph_capture_replay_matches_eager():
    """Several run calls (one per layer) captured in one HIP graph; every replay,
    with eager work in between, must match the eager result exactly."""
    w = wl.small_workload(wl.WORKLOADS["student_4b"], batch=8, lengths=(50, 600))
    lay = wl.workload_layout(w)
    offs, lens = up_i32(lay.offsets), up_i32(lay.lens)
    layers = []
    for layer in range(3):
        kh, vh = wl.layer_kv_bits(w, lay, layer)
        layers.append((up_bf16(wl.query_bits(w, layer)), up_bf16(kh), up_bf16(vh)))
    attn = DecodeAttention(32, 8, w.batch, lay.max_seq_len)
    outs = [torch.zeros((w.batch, 32, 128), dtype=torch.float32, device=dev()) for _ in layers]
    eager = []
    for (q, k, v), o in zip(layers, outs):
        attn.run(q, k, v, offs, lens, w.scale, o)
        eager.append(o.clone())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for (q, k, v), o in zip(layers, outs):
                attn.run(q, k, v, offs, lens, w.scale, o)
    torch.cuda.synchronize()
    for rep in range(4):
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, eager):
            assert torch.equal(o, e), f"replay {rep}"
        # eager work between replays
        attn.run(*layers[0], offs, lens, w.scale, outs[0])
        torch.cuda.synchronize()
    del g
    attn.close()


@pytest.mark.parametrize("split", [0, 16])
def test_non_finite_value_reaches_only_its_own_dimension(split):
    """out[b, h, d] depends on V[:, kv, d] only (eq:token-context, the
    attention definition): a NaN or an infinity in one element of V makes that
    output dimension of the heads reading it non-finite and leaves every other
    element equal to the oracle's."""
    rng = np.random.default_rng(61)
    w = wl.Workload("nonfinite", 121, 1, 4, 32, 8, 1, "uniform", 40, 300)
    lay = wl.workload_layout(w)
    k, v = wl.layer_kv_bits(w, lay, 0)
    q = wl.query_bits(w, 0)
    planted = [(1, 7, 2, 37, wl.BF16_NAN), (2, 3, 5, 100, np.uint16(0x7F80)), (3, 0, 0, 5, np.uint16(0xFF80))]
    for b, t, kv, d, bits in planted:
        v[lay.offsets[b] + t, kv, d] = bits
    ref = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale)
    got = run(32, 8, q, k, v, lay.offsets, lay.lens, w.scale, split_tokens=split)
    bad = np.zeros(got.shape, bool)
    g = w.group
    for b, t, kv, d, _ in planted:
        bad[b, kv * g:(kv + 1) * g, d] = True
    assert not np.isfinite(got[bad]).any(), "a planted non-finite value did not reach its dimension"
    assert np.isnan(got[1, 2 * g:3 * g, 37]).all()
    assert_parity(got[~bad], ref[~bad], f"elements beside the non-finite ones, split={split}")

"""Paged KV caches (block tables) and the fused append of the decoded token,
through ctx_decode_attn_run_paged, against the paged CPU oracle."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import CtxError, DecodeAttention

from _gpu_util import SampledLayer, assert_parity, dev, paged_copy, up_bf16, up_i32

pytestmark = pytest.mark.gpu

bf = wl.f32_to_bf16_bits


def rand_bits(rng, shape):
    return bf(rng.standard_normal(shape).astype(np.float32))


def run_paged(w, q, kp, vp, bt, lens, page_tokens, split=0, k_new=None, v_new=None, max_seq_len=None,
              out_dtype=torch.float32):
    """Returns (out, k_pages after, v_pages after) as host arrays."""
    b = len(lens)
    kpd, vpd = up_bf16(kp), up_bf16(vp)
    with DecodeAttention(w.num_q_heads, w.num_kv_heads, b, max_seq_len or int(np.max(lens)),
                         split_tokens=split, page_tokens=page_tokens, out_dtype=out_dtype) as attn:
        buf = torch.full((b + 1, w.num_q_heads, 128), -777.0, dtype=out_dtype, device=dev())
        out = buf[:b]
        attn.run_paged(up_bf16(q), kpd, vpd, up_i32(bt), up_i32(lens), w.scale, out,
                       k_new=None if k_new is None else up_bf16(k_new),
                       v_new=None if v_new is None else up_bf16(v_new))
        torch.cuda.synchronize()
        assert (buf[b] == -777.0).all(), "write past the end of out"
    as_bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)  # noqa: E731
    return out.float().cpu().numpy(), as_bits(kpd), as_bits(vpd)


def paged_case(seed, page_tokens, batch=20, hq=32, hkv=8, lo=1, hi=900, steps=4):
    rng = np.random.default_rng(seed)
    w = wl.Workload(f"pg{seed}", 130 + seed % 50, 1, batch, hq, hkv, steps, "uniform", lo, hi)
    lens = wl.draw_lengths(w)
    fixed = np.minimum([1, page_tokens, page_tokens + 1, 2 * page_tokens + 3, 15, 17], hi)[:batch]
    lens[:len(fixed)] = fixed
    lay = wl.make_layout(lens, steps=steps)
    k, v = wl.layer_kv_bits(w, lay, 0)
    q = wl.query_bits(w, 0)
    kp, vp, bt = paged_copy(k, v, lay, page_tokens, rng)
    return w, lay, q, kp, vp, bt, rng


@pytest.mark.parametrize("page_tokens", [16, 32, 64])
def test_paged_parity(page_tokens):
    w, lay, q, kp, vp, bt, _ = paged_case(50 + page_tokens, page_tokens)
    ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale)
    for split in (0, 16, 48, 112):
        got, kp2, vp2 = run_paged(w, q, kp, vp, bt, lay.lens, page_tokens, split=split,
                                  max_seq_len=lay.max_seq_len)
        assert_parity(got, ref, f"paged P={page_tokens} split={split}")
        np.testing.assert_array_equal(kp2, kp)  # nothing written without an append
        np.testing.assert_array_equal(vp2, vp)


@pytest.mark.parametrize("page_tokens,split", [(16, 0), (16, 32), (64, 0), (32, 48)])
def test_paged_append(page_tokens, split):
    """The slot of each sequence's newest token holds NaN before the call; the
    kernel must attend to k_new / v_new instead and leave them in the slot,
    and change nothing else in the caches."""
    w, lay, q, kp, vp, bt, rng = paged_case(70 + page_tokens + split, page_tokens)
    lens = lay.lens.copy()
    lens[3] = 0  # an empty sequence appends nothing
    k_new = rand_bits(rng, (w.batch, w.num_kv_heads, 128))
    v_new = rand_bits(rng, (w.batch, w.num_kv_heads, 128))
    kp_exp, vp_exp = kp.copy(), vp.copy()
    for b in range(w.batch):
        if lens[b] == 0:
            continue
        t = lens[b] - 1
        page, slot = bt[b, t // page_tokens], t % page_tokens
        kp[page, slot] = wl.BF16_NAN
        vp[page, slot] = wl.BF16_NAN
        kp_exp[page, slot] = k_new[b]
        vp_exp[page, slot] = v_new[b]
    ref = oracle.decode_attn_paged(q, kp, vp, bt, lens, w.scale, k_new, v_new)
    got, kp2, vp2 = run_paged(w, q, kp, vp, bt, lens, page_tokens, split=split, k_new=k_new, v_new=v_new,
                              max_seq_len=lay.max_seq_len)
    assert_parity(got, ref, f"append P={page_tokens} split={split}")
    assert (got[3] == 0).all()
    np.testing.assert_array_equal(kp2, kp_exp)
    np.testing.assert_array_equal(vp2, vp_exp)


def test_paged_gqa_group_sizes():
    """Workgroups of up to 8 KV heads: odd KV-head counts leave a partial
    workgroup, and odd group sizes an odd number of query heads per KV head;
    every case also appends, so the append's row addressing is checked too."""
    for hq, hkv in [(16, 1), (64, 4), (8, 8), (9, 3), (12, 6), (5, 1), (28, 7), (45, 9), (30, 10)]:
        w, lay, q, kp, vp, bt, rng = paged_case(90 + hq + hkv, 16, batch=5, hq=hq, hkv=hkv, hi=300)
        ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale)
        got, _, _ = run_paged(w, q, kp, vp, bt, lay.lens, 16)
        assert_parity(got, ref, f"paged {hq}/{hkv}")
        k_new = rand_bits(rng, (w.batch, hkv, 128))
        v_new = rand_bits(rng, (w.batch, hkv, 128))
        kp_exp, vp_exp = kp.copy(), vp.copy()
        for b in range(w.batch):
            t = lay.lens[b] - 1
            kp_exp[bt[b, t // 16], t % 16] = k_new[b]
            vp_exp[bt[b, t // 16], t % 16] = v_new[b]
        ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale, k_new, v_new)
        got, kp2, vp2 = run_paged(w, q, kp, vp, bt, lay.lens, 16, split=32, k_new=k_new, v_new=v_new)
        assert_parity(got, ref, f"paged append {hq}/{hkv}")
        np.testing.assert_array_equal(kp2, kp_exp)
        np.testing.assert_array_equal(vp2, vp_exp)


def test_paged_full_size_long_ragged_with_append():
    """Full-size long-horizon ragged layer in 16-token pages (pages shuffled),
    the last decode step appending its token; the oracle recomputes the
    sampled sequences."""
    w = wl.WORKLOADS["long_ragged"]
    sl = SampledLayer(w)
    lay = sl.layout
    P = 16
    rng = np.random.default_rng(5)
    npages = [-(-int(c) // P) for c in lay.capacity]
    perm = torch.from_numpy(rng.permutation(sum(npages)).astype(np.int64)).to(dev())
    bt = np.zeros((w.batch, max(npages)), np.int32)
    # page j of sequence b holds cache rows offs_b + jP ..; shuffle pages through perm
    src_rows = []
    nxt = 0
    for b in range(w.batch):
        for j in range(npages[b]):
            bt[b, j] = int(perm[nxt])
            src_rows.append(int(lay.offsets[b]) + j * P)
            nxt += 1
    kp = torch.zeros((sum(npages), P, 8, 128), dtype=torch.bfloat16, device=dev())
    vp = torch.zeros_like(kp)
    rows = torch.tensor(src_rows, device=dev())
    idx = rows[:, None] + torch.arange(P, device=dev())[None, :]
    idx = idx.clamp(max=lay.num_rows - 1)
    kp[perm] = sl.k[idx]
    vp[perm] = sl.v[idx]
    step = w.steps - 1
    lens = lay.lens_at(step)
    qh, qd = sl.query(step)
    k_new = rand_bits(rng, (w.batch, 8, 128))
    v_new = rand_bits(rng, (w.batch, 8, 128))
    out = torch.empty((w.batch, 32, 128), dtype=torch.float32, device=dev())
    with DecodeAttention(32, 8, w.batch, lay.max_seq_len, page_tokens=P) as attn:
        attn.run_paged(qd, kp, vp, up_i32(bt), up_i32(lens), w.scale, out, k_new=up_bf16(k_new),
                       v_new=up_bf16(v_new))
        torch.cuda.synchronize()
    # oracle on the sampled sequences: contiguous host rows with the newest row replaced
    hk, hv = sl.hk.copy(), sl.hv.copy()
    sample_lens = np.array([lens[b] for b in sl.sample], np.int32)
    for i, b in enumerate(sl.sample):
        r = sl.host_offsets[i] + lens[b] - 1
        hk[r], hv[r] = k_new[b], v_new[b]
    ref = oracle.decode_attn(qh[sl.sample], hk, hv, sl.host_offsets, sample_lens, w.scale)
    assert_parity(out.cpu().numpy()[sl.sample], ref, "paged full-size long_ragged append")
    for b in sl.sample:  # the appended rows landed in their pages
        t = lens[b] - 1
        got_k = kp[bt[b, t // P], t % P].view(torch.int16).cpu().numpy().view(np.uint16)
        np.testing.assert_array_equal(got_k, k_new[b])


def test_paged_abi_errors():
    lib = bd.load_library()
    q = torch.zeros((2, 16, 128), dtype=torch.bfloat16, device=dev())
    pages = torch.zeros((4, 16, 8, 128), dtype=torch.bfloat16, device=dev())
    bt = torch.zeros((2, 2), dtype=torch.int32, device=dev())
    lens = torch.ones(2, dtype=torch.int32, device=dev())
    out = torch.zeros((2, 16, 128), dtype=torch.float32, device=dev())
    new = torch.zeros((2, 8, 128), dtype=torch.bfloat16, device=dev())
    P = lambda t, off=0: t.data_ptr() + off  # noqa: E731
    with DecodeAttention(16, 8, 2, 32) as plain:  # no page_tokens
        rc = lib.ctx_decode_attn_run_paged(plain.handle, P(q), P(pages), P(pages), P(bt), 2, P(lens), 2,
                                           None, None, 0.1, P(out), None)
        assert rc == bd.CTX_ERR_UNSUPPORTED
    with DecodeAttention(16, 8, 2, 32, page_tokens=16) as attn:
        h = attn.handle
        args = lambda kn, vn, mp=2: (P(q), P(pages), P(pages), P(bt), mp, P(lens), 2, kn, vn, 0.1, P(out), None)  # noqa: E731
        assert lib.ctx_decode_attn_run_paged(h, *args(None, None)) == bd.CTX_OK
        assert lib.ctx_decode_attn_run_paged(h, *args(P(new), P(new))) == bd.CTX_OK
        assert lib.ctx_decode_attn_run_paged(h, *args(P(new), None)) == bd.CTX_ERR_INVALID_ARG
        assert lib.ctx_decode_attn_run_paged(h, *args(P(new, 2), P(new))) == bd.CTX_ERR_ALIGNMENT
        assert lib.ctx_decode_attn_run_paged(h, *args(None, None, mp=0)) == bd.CTX_ERR_INVALID_ARG
        torch.cuda.synchronize()
    for kw in (dict(page_tokens=24), dict(page_tokens=16, split_tokens=24), dict(page_tokens=-16)):
        with pytest.raises(CtxError):
            DecodeAttention(16, 8, 2, 32, **kw)


def test_paged_more_than_256_sequences_with_append():
    """300 sequences in 16-token pages: the padded range plan and the merge scan
    the lengths across a 256-sequence chunk boundary; the append of every
    sequence's newest token is checked in the caches too."""
    w, lay, q, kp, vp, bt, rng = paged_case(37, 16, batch=300, hi=300)
    k_new = rand_bits(rng, (w.batch, w.num_kv_heads, 128))
    v_new = rand_bits(rng, (w.batch, w.num_kv_heads, 128))
    ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale, k_new, v_new)
    for split in (0, 32):
        got, _, _ = run_paged(w, q, kp, vp, bt, lay.lens, 16, split=split, k_new=k_new, v_new=v_new,
                              max_seq_len=lay.max_seq_len)
        assert_parity(got, ref, f"paged append, 300 sequences, split={split}")


def test_paged_bf16_output_and_many_sequences():
    """bf16 output equals the rounded fp32 output, and a batch of more than
    64 sequences (the range search over the whole batch) with an append."""
    w, lay, q, kp, vp, bt, rng = paged_case(31, 16, batch=150, hi=400)
    f32, _, _ = run_paged(w, q, kp, vp, bt, lay.lens, 16, split=0, max_seq_len=lay.max_seq_len)
    b16, _, _ = run_paged(w, q, kp, vp, bt, lay.lens, 16, split=0, max_seq_len=lay.max_seq_len,
                          out_dtype=torch.bfloat16)
    np.testing.assert_array_equal(b16, wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(f32.astype(np.float32))))
    ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale)
    assert_parity(f32, ref, "paged, 150 sequences")
    k_new = rand_bits(rng, (w.batch, w.num_kv_heads, 128))
    v_new = rand_bits(rng, (w.batch, w.num_kv_heads, 128))
    ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale, k_new, v_new)
    for split in (0, 32):
        got, _, _ = run_paged(w, q, kp, vp, bt, lay.lens, 16, split=split, k_new=k_new, v_new=v_new,
                              max_seq_len=lay.max_seq_len)
        assert_parity(got, ref, f"paged append, 150 sequences, split={split}")

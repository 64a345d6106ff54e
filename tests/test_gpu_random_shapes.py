"""A seeded random sweep of shapes through the decode step (contiguous and
paged) and the causal prefill, each case against the oracle.

Every case draws its own head ratio (1 to 16 query heads per KV head, 1 to 16
KV heads), batch, length mix (zero, one and block-boundary lengths among
uniform and long ones), forced split, page size and whether the decoded token
is appended.  Caches are laid out in shuffled order with NaN-poisoned gaps and
unused page slots, so a read outside a sequence's rows shows up as a non-finite
output.  Contiguous decode runs in both output dtypes: fp32 against the oracle,
bf16 as the round-to-nearest-even of the same handle's fp32 result."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import DecodeAttention

from _gpu_util import assert_parity, dev, paged_copy, up_bf16, up_i32

pytestmark = pytest.mark.gpu

bf = wl.f32_to_bf16_bits
EDGE_LENGTHS = (0, 1, 2, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129)


def heads(rng):
    hkv = int(rng.choice([1, 2, 3, 4, 5, 6, 7, 8, 10, 12, 16]))
    g = int(rng.integers(1, 17))
    while hkv * g > 128:
        g -= 1
    return hkv * g, hkv


def lengths(rng, batch, long_max=5000):
    pick = rng.random(batch)
    lens = np.where(pick < 0.35, rng.choice(EDGE_LENGTHS, size=batch),
                    np.where(pick < 0.9, rng.integers(1, 1500, size=batch),
                             rng.integers(1500, long_max + 1, size=batch)))
    return lens.astype(np.int32)


def rand_bits(rng, shape):
    return bf(rng.standard_normal(shape).astype(np.float32))


def workload(case, batch, hq, hkv, rng):
    peaky = 0.05 if rng.random() < 0.3 else 0.0
    return wl.Workload(f"rand{case}", 200 + case, 1, batch, hq, hkv, 1, "uniform", 1, 2, peaky_frac=peaky)


@pytest.mark.parametrize("case", range(16))
def test_random_decode(case):
    rng = np.random.default_rng(9000 + case)
    hq, hkv = heads(rng)
    batch = int(rng.integers(1, 121))
    lens = lengths(rng, batch)
    w = workload(case, batch, hq, hkv, rng)
    lay = wl.make_layout(lens, 1, gap_max=4, shuffle=True, rng=rng)
    k, v = wl.layer_kv_bits(w, lay, 0, fill=wl.BF16_NAN)
    q = wl.query_bits(w, 0)
    split = int(rng.choice([0, 0, 16, 17, 48, 64, 200, 1000]))
    what = f"case {case}: {hq}/{hkv} heads, batch {batch}, split {split}, tokens {int(lens.sum())}"
    print(what, flush=True)
    ref = oracle.decode_attn(q, k, v, lay.offsets, lens, w.scale)
    outs = {}
    for dt in (torch.float32, torch.bfloat16):
        with DecodeAttention(hq, hkv, batch, max(1, lay.max_seq_len), out_dtype=dt, split_tokens=split) as attn:
            buf = torch.full((batch + 1, hq, 128), -9.0, dtype=dt, device=dev())
            attn.run(up_bf16(q), up_bf16(k), up_bf16(v), up_i32(lay.offsets), up_i32(lens), w.scale, buf[:batch])
            torch.cuda.synchronize()
            assert (buf[batch] == -9.0).all(), f"{what}: write past the end of out"
            outs[dt] = buf[:batch]
    got = outs[torch.float32].cpu().numpy()
    assert_parity(got, ref, what)
    assert (got[lens == 0] == 0).all(), f"{what}: empty sequences must give zeros"
    want = outs[torch.float32].to(torch.bfloat16)
    assert torch.equal(outs[torch.bfloat16].view(torch.int16), want.view(torch.int16)), \
        f"{what}: bf16 out is not the rounded fp32 result"


@pytest.mark.parametrize("case", range(10))
def test_random_paged(case):
    rng = np.random.default_rng(9100 + case)
    hq, hkv = heads(rng)
    batch = int(rng.integers(1, 90))
    lens = lengths(rng, batch, long_max=3000)
    page = int(rng.choice([16, 32, 48, 64, 128]))
    split = int(rng.choice([0, 0, page, 16 * int(rng.integers(1, 40))]))
    append = bool(rng.random() < 0.6)
    w = workload(case, batch, hq, hkv, rng)
    lay = wl.make_layout(lens, 1)
    k, v = wl.layer_kv_bits(w, lay, 0)
    q = wl.query_bits(w, 0)
    kp, vp, bt = paged_copy(k, v, lay, page, rng)
    k_new = v_new = None
    kp_exp, vp_exp = kp.copy(), vp.copy()
    if append:
        k_new = rand_bits(rng, (batch, hkv, 128))
        v_new = rand_bits(rng, (batch, hkv, 128))
        for b in range(batch):
            if lens[b] == 0:
                continue
            t = lens[b] - 1
            pg, slot = bt[b, t // page], t % page
            kp[pg, slot] = wl.BF16_NAN  # the call must attend to k_new / v_new, not the slot
            vp[pg, slot] = wl.BF16_NAN
            kp_exp[pg, slot] = k_new[b]
            vp_exp[pg, slot] = v_new[b]
    what = f"case {case}: {hq}/{hkv} heads, batch {batch}, page {page}, split {split}, append {append}"
    print(what, flush=True)
    ref = oracle.decode_attn_paged(q, kp, vp, bt, lens, w.scale, k_new, v_new)
    kpd, vpd = up_bf16(kp), up_bf16(vp)
    with DecodeAttention(hq, hkv, batch, max(1, lay.max_seq_len), split_tokens=split, page_tokens=page) as attn:
        buf = torch.full((batch + 1, hq, 128), -9.0, dtype=torch.float32, device=dev())
        attn.run_paged(up_bf16(q), kpd, vpd, up_i32(bt), up_i32(lens), w.scale, buf[:batch],
                       k_new=None if k_new is None else up_bf16(k_new),
                       v_new=None if v_new is None else up_bf16(v_new))
        torch.cuda.synchronize()
        assert (buf[batch] == -9.0).all(), f"{what}: write past the end of out"
    got = buf[:batch].cpu().numpy()
    assert_parity(got, ref, what)
    assert (got[lens == 0] == 0).all(), f"{what}: empty sequences must give zeros"
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)  # noqa: E731
    np.testing.assert_array_equal(bits(kpd), kp_exp, err_msg=f"{what}: K pages")
    np.testing.assert_array_equal(bits(vpd), vp_exp, err_msg=f"{what}: V pages")


@pytest.mark.parametrize("case", range(10))
def test_random_prefill(case):
    rng = np.random.default_rng(9200 + case)
    hq, hkv = heads(rng)
    batch = int(rng.integers(1, 11))
    nq = rng.integers(0, 261, size=batch).astype(np.int32)
    nq[rng.random(batch) < 0.15] = 1
    hist = np.where(rng.random(batch) < 0.2, 0, rng.integers(0, 1500, size=batch))
    lens = (hist + nq).astype(np.int32)
    split_p = bool(rng.random() < 0.5)
    w = workload(case, batch, hq, hkv, rng)
    lay = wl.make_layout(lens, 1, gap_max=5, shuffle=True, rng=rng)
    k, v = wl.layer_kv_bits(w, lay, 0, fill=wl.BF16_NAN)
    q_starts = np.zeros(batch, np.int32)
    row = 0
    for b in rng.permutation(batch):
        row += int(rng.integers(0, 3))
        q_starts[b] = row
        row += int(nq[b])
    total_q = row + 1
    q = rand_bits(rng, (total_q, hq, 128))
    what = f"case {case}: {hq}/{hkv} heads, batch {batch}, new {nq.tolist()}, split_p {split_p}"
    print(what, flush=True)
    ref = oracle.prefill_attn(q, k, v, lay.offsets, lens, q_starts, nq, w.scale)
    max_q = max(1, int(nq.max()))
    with DecodeAttention(hq, hkv, batch, max(1, int(lens.max()))) as attn:
        out = torch.full((total_q, hq, 128), -9.0, dtype=torch.float32, device=dev())
        attn.prefill(up_bf16(q), up_bf16(k), up_bf16(v), up_i32(lay.offsets), up_i32(lens), up_i32(q_starts),
                     up_i32(nq), max_q, w.scale, out, split_p=split_p)
        torch.cuda.synchronize()
    got = out.cpu().numpy()
    rows = np.concatenate([np.arange(q_starts[b], q_starts[b] + nq[b]) for b in range(batch)]).astype(np.int64)
    untouched = np.setdiff1d(np.arange(total_q), rows)
    assert (got[untouched] == -9.0).all(), f"{what}: rows of no sequence were written"
    if len(rows):
        assert_parity(got[rows], ref[rows], what, tight=split_p)

"""Full-size layers, every (sequence, head) compared with the oracle.

One layer of each full-size workload at its first and last decode step,
launched as the benchmark launches it (balanced split over the whole batch).
The layer is drawn on the device (N(0,1) bf16 keys and values, plus the
act-first burst's peaky keys: 5% of key rows x4) and copied whole to the host,
where the oracle recomputes every sequence and head.

The act-first burst's layer holds more than 2^31 elements per cache (256
sequences of up to 12,800 rows of 8 x 128), so its last sequences start past
byte offset 4 GiB of K and V; the tests check that the layout places some
there and compare them like every other sequence.  The same layer also
serves the paged decode (16-token pages, shuffled, with the append of the
decoded token) and the causal prefill of the appended reference observation
(three query rows of every sequence, all heads).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import DecodeAttention

from _gpu_util import assert_parity, dev, up_bf16, up_i32

pytestmark = pytest.mark.gpu

FOUR_GIB = 1 << 32


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


class FullLayer:
    """A full-size layer on the device and its exact copy on the host."""

    def __init__(self, w: wl.Workload, layer: int = 0):
        self.w = w
        self.layer = layer
        self.layout = wl.workload_layout(w)
        shape = (self.layout.num_rows, w.num_kv_heads, w.head_dim)
        self.k = torch.empty(shape, dtype=torch.bfloat16, device=dev())
        self.v = torch.empty_like(self.k)
        wl.fill_kv_device(self.k, self.v, w, layer)
        torch.cuda.synchronize()
        self.hk = host_bits(self.k)
        self.hv = host_bits(self.v)
        self.offsets = up_i32(self.layout.offsets)
        row_bytes = w.num_kv_heads * w.head_dim * 2
        self.past_4gib = [b for b in range(w.batch) if int(self.layout.offsets[b]) * row_bytes >= FOUR_GIB]

    def query(self, step: int):
        qh = wl.query_bits(self.w, self.layer, step)
        return qh, up_bf16(qh)


_cache = {}


def full_layer(name: str) -> FullLayer:
    """One layer per workload, kept for the tests of this module."""
    if name not in _cache:
        _cache.clear()
        torch.cuda.empty_cache()
        _cache[name] = FullLayer(wl.WORKLOADS[name])
    return _cache[name]


def teardown_module(module):
    _cache.clear()
    torch.cuda.empty_cache()


# the act-first burst last: the paged and prefill tests below reuse its layer
FIRST_LAST = [
    ("student_0p6b_1p7b", (0,)),
    ("student_4b", (0,)),
    ("long_ragged", (0, 63)),
    ("act_first_burst", (0, 7)),
]


@pytest.mark.parametrize("name,steps", FIRST_LAST, ids=[n for n, _ in FIRST_LAST])
def test_full_layer_every_sequence(name, steps):
    fl = full_layer(name)
    w, lay = fl.w, fl.layout
    if name == "act_first_burst":
        assert fl.past_4gib, "the act-first layer should place sequences past byte offset 4 GiB"
        print(f"{name}: sequences {fl.past_4gib} start past byte offset 4 GiB", flush=True)
    with DecodeAttention(w.num_q_heads, w.num_kv_heads, w.batch, lay.max_seq_len) as attn:
        for step in steps:
            assert step < w.steps
            qh, qd = fl.query(step)
            lens = lay.lens_at(step)
            out = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev())
            attn.run(qd, fl.k, fl.v, fl.offsets, up_i32(lens), w.scale, out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            ref = oracle.decode_attn(qh, fl.hk, fl.hv, lay.offsets, lens, w.scale)
            assert_parity(got, ref, f"{name} layer 0 step {step}, all {w.batch} sequences x {w.num_q_heads} heads")
            if fl.past_4gib:
                assert_parity(got[fl.past_4gib], ref[fl.past_4gib], f"{name} step {step} past 4 GiB")


def test_full_layer_paged_act_first_burst_with_append():
    """The act-first layer in 16-token pages dealt in shuffled order, at the
    last decode step, appending each sequence's decoded token; every sequence
    is compared with the oracle on the contiguous copy whose newest rows hold
    the appended keys and values, and every appended row is checked in its page."""
    fl = full_layer("act_first_burst")
    w, lay = fl.w, fl.layout
    P = 16
    rng = np.random.default_rng(23)
    npages = -(-lay.capacity.astype(np.int64) // P)
    total_pages = int(npages.sum())
    perm = rng.permutation(total_pages)
    bt = np.zeros((w.batch, int(npages.max())), np.int32)
    src = np.empty(total_pages, np.int64)  # first contiguous row of each page, by page number
    nxt = 0
    for b in range(w.batch):
        for j in range(int(npages[b])):
            page = int(perm[nxt])
            bt[b, j] = page
            src[page] = int(lay.offsets[b]) + j * P
            nxt += 1
    idx = torch.from_numpy(src).to(dev())[:, None] + torch.arange(P, device=dev())[None, :]
    idx.clamp_(max=lay.num_rows - 1)  # slots past a sequence's capacity are never read
    kp = fl.k[idx.view(-1)].view(total_pages, P, w.num_kv_heads, w.head_dim)
    vp = fl.v[idx.view(-1)].view(total_pages, P, w.num_kv_heads, w.head_dim)
    del idx
    step = w.steps - 1
    lens = lay.lens_at(step)
    qh, qd = fl.query(step)
    k_new = wl.normal_bf16(rng, (w.batch, w.num_kv_heads, w.head_dim))
    v_new = wl.normal_bf16(rng, (w.batch, w.num_kv_heads, w.head_dim))
    out = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev())
    with DecodeAttention(w.num_q_heads, w.num_kv_heads, w.batch, lay.max_seq_len, page_tokens=P) as attn:
        attn.run_paged(qd, kp, vp, up_i32(bt), up_i32(lens), w.scale, out, k_new=up_bf16(k_new),
                       v_new=up_bf16(v_new))
        torch.cuda.synchronize()
    # the oracle on the contiguous host copy with each newest row replaced (restored afterwards)
    newest = lay.offsets.astype(np.int64) + lens - 1
    saved_k, saved_v = fl.hk[newest].copy(), fl.hv[newest].copy()
    try:
        fl.hk[newest], fl.hv[newest] = k_new, v_new
        ref = oracle.decode_attn(qh, fl.hk, fl.hv, lay.offsets, lens, w.scale)
    finally:
        fl.hk[newest], fl.hv[newest] = saved_k, saved_v
    got = out.cpu().numpy()
    assert_parity(got, ref, f"paged act-first burst step {step} with append, all sequences")
    assert_parity(got[fl.past_4gib], ref[fl.past_4gib], "paged, sequences past 4 GiB")
    t = lens - 1
    pages = torch.from_numpy(bt[np.arange(w.batch), t // P].astype(np.int64)).to(dev())
    slots = torch.from_numpy((t % P).astype(np.int64)).to(dev())
    np.testing.assert_array_equal(host_bits(kp[pages, slots]), k_new)
    np.testing.assert_array_equal(host_bits(vp[pages, slots]), v_new)
    del kp, vp
    torch.cuda.empty_cache()


@pytest.mark.parametrize("split_p", [False, True], ids=["bf16p", "splitp"])
def test_full_layer_prefill_act_first_burst_every_sequence(split_p):
    """Causal prefill of every sequence's appended reference observation
    (U{128..512} newest tokens) over the full act-first layer in one call;
    the first, the last and one middle query row of every sequence, all heads,
    are recomputed by the oracle as decodes of their prefixes."""
    fl = full_layer("act_first_burst")
    w, lay = fl.w, fl.layout
    lens = lay.lens_at(0)
    nq = wl.draw_extra(w)
    q_starts = np.concatenate([[0], np.cumsum(nq)[:-1]]).astype(np.int32)
    total_q = int(nq.sum())
    q = torch.empty((total_q, w.num_q_heads, w.head_dim), dtype=torch.bfloat16, device=dev())
    wl.fill_normal_bf16_device(q, wl.DEFAULT_SEED, w.index, fl.layer, 13)
    out = torch.empty((total_q, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev())
    with DecodeAttention(w.num_q_heads, w.num_kv_heads, w.batch, int(lens.max())) as attn:
        attn.prefill(q, fl.k, fl.v, fl.offsets, up_i32(lens), up_i32(q_starts), up_i32(nq), int(nq.max()),
                     w.scale, out, split_p=split_p)
        torch.cuda.synchronize()
    rng = np.random.default_rng(29)
    rows, sub_offs, sub_lens = [], [], []
    for b in range(w.batch):
        for i in sorted({0, int(rng.integers(1, nq[b] - 1)), int(nq[b]) - 1}):
            rows.append(int(q_starts[b]) + i)
            sub_offs.append(int(lay.offsets[b]))
            sub_lens.append(int(lens[b]) - int(nq[b]) + i + 1)
    sel = torch.tensor(rows, device=dev())
    qh = host_bits(q[sel])
    ref = oracle.decode_attn(qh, fl.hk, fl.hv, np.array(sub_offs, np.int32), np.array(sub_lens, np.int32), w.scale)
    got = out[sel].cpu().numpy()
    what = f"prefill act-first burst ({'two-term' if split_p else 'bf16'} weights), {len(rows)} rows of all sequences"
    assert_parity(got, ref, what, tight=split_p)
    assert torch.isfinite(out).all().item()

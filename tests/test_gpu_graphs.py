"""HIP-graph capture of the other allocation-free entry points: the paged
decode step with its append, the causal prefill (both weight precisions) and
the OPD loss with its gradient.  Each is captured once and replayed several
times, with eager work in between, and every replay must equal the eager
result bit for bit (including the caches the append writes)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import DecodeAttention

from _gpu_util import assert_parity, dev, paged_copy, up_bf16, up_i32

pytestmark = pytest.mark.gpu

REPLAYS = 4


def capture(fn):
    """fn() queued on a side stream inside one captured graph."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fn(s)
    torch.cuda.synchronize()
    return g


def bits(t):
    """The tensor's bits as integers: equal means identical, NaN included."""
    return t.view({4: torch.int32, 2: torch.int16}[t.element_size()])


def replay_and_check(g, outputs, expected, poison, eager_between):
    for rep in range(REPLAYS):
        for t in outputs:
            poison(t)
        g.replay()
        torch.cuda.synchronize()
        for name, (t, e) in enumerate(zip(outputs, expected)):
            assert torch.equal(bits(t), bits(e)), f"replay {rep}, output {name}"
        eager_between()
        torch.cuda.synchronize()


def test_graph_paged_decode_with_append():
    rng = np.random.default_rng(41)
    w = wl.Workload("pgraph", 141, 1, 12, 32, 8, 3, "uniform", 1, 500)
    lens = wl.draw_lengths(w)
    lay = wl.make_layout(lens, steps=3)
    P = 16
    layers = []
    for layer in range(2):
        k, v = wl.layer_kv_bits(w, lay, layer)
        kp, vp, bt = paged_copy(k, v, lay, P, rng)
        q = wl.query_bits(w, layer)
        kn = wl.f32_to_bf16_bits(rng.standard_normal((w.batch, 8, 128)).astype(np.float32))
        vn = wl.f32_to_bf16_bits(rng.standard_normal((w.batch, 8, 128)).astype(np.float32))
        ref = oracle.decode_attn_paged(q, kp, vp, bt, lay.lens, w.scale, kn, vn)
        layers.append(dict(q=up_bf16(q), kp=up_bf16(kp), vp=up_bf16(vp), bt=up_i32(bt), kn=up_bf16(kn),
                           vn=up_bf16(vn), ref=ref))
    lens_d = up_i32(lay.lens)
    attn = DecodeAttention(32, 8, w.batch, lay.max_seq_len, page_tokens=P)
    outs = [torch.zeros((w.batch, 32, 128), dtype=torch.float32, device=dev()) for _ in layers]

    def run_all(stream=None):
        for L, o in zip(layers, outs):
            attn.run_paged(L["q"], L["kp"], L["vp"], L["bt"], lens_d, w.scale, o, k_new=L["kn"], v_new=L["vn"],
                           stream=stream)

    run_all()
    torch.cuda.synchronize()
    for L, o in zip(layers, outs):
        assert_parity(o.cpu().numpy(), L["ref"], "paged eager")
    eager = [o.clone() for o in outs]
    caches = [t.clone() for L in layers for t in (L["kp"], L["vp"])]
    g = capture(run_all)
    replay_and_check(g, outs, eager, lambda t: t.fill_(float("nan")), lambda: run_all())
    # the appends rewrite the same slots with the same rows: the caches are
    # unchanged bit for bit (their unused slots hold NaN, so compare the bits)
    for t, c in zip([t for L in layers for t in (L["kp"], L["vp"])], caches):
        assert torch.equal(t.view(torch.int16), c.view(torch.int16))
    del g
    attn.close()


@pytest.mark.parametrize("split_p", [False, True])
def test_graph_prefill(split_p):
    rng = np.random.default_rng(43)
    lens = np.array([40, 300, 7, 129], np.int32)
    nq = np.array([5, 120, 7, 0], np.int32)
    lay = wl.make_layout(lens, 1, gap_max=5, shuffle=True, rng=rng)
    k = wl.f32_to_bf16_bits(rng.standard_normal((lay.num_rows, 8, 128)).astype(np.float32))
    v = wl.f32_to_bf16_bits(rng.standard_normal((lay.num_rows, 8, 128)).astype(np.float32))
    qs = np.concatenate([[0], np.cumsum(nq)[:-1]]).astype(np.int32)
    q = wl.f32_to_bf16_bits(rng.standard_normal((int(nq.sum()), 32, 128)).astype(np.float32))
    ref = oracle.prefill_attn(q, k, v, lay.offsets, lens, qs, nq, 0.0884)
    args = [up_bf16(q), up_bf16(k), up_bf16(v), up_i32(lay.offsets), up_i32(lens), up_i32(qs), up_i32(nq)]
    attn = DecodeAttention(32, 8, len(lens), int(lens.max()))
    out = torch.zeros((int(nq.sum()), 32, 128), dtype=torch.float32, device=dev())

    def run(stream=None):
        attn.prefill(*args, int(nq.max()), 0.0884, out, stream=stream, split_p=split_p)

    run()
    torch.cuda.synchronize()
    assert_parity(out.cpu().numpy(), ref, f"prefill eager split_p={split_p}", tight=split_p)
    eager = out.clone()
    g = capture(run)
    replay_and_check(g, [out], [eager], lambda t: t.fill_(float("nan")), lambda: run())
    del g
    attn.close()


def test_graph_opd_loss_and_gradient():
    ow = wl.OPD_WORKLOADS["opd_tiny"]
    ob = wl.opd_batch(ow)
    zh = wl.opd_logits_host(ow, ob)
    ref = oracle.opd_loss(zh[:, :ow.vocab], ob.tokens, ob.old_lp, ob.teacher_lp, ob.mask, ob.seq_starts)
    ins = [up_bf16(zh), up_i32(ob.tokens), torch.from_numpy(ob.old_lp).to(dev()),
           torch.from_numpy(ob.teacher_lp).to(dev()), torch.from_numpy(ob.mask).to(dev()), up_i32(ob.seq_starts)]
    n = len(ob.tokens)
    out = {"loss": torch.zeros(1, dtype=torch.float32, device=dev()),
           "token_logp": torch.zeros(n, dtype=torch.float32, device=dev()),
           "token_weight": torch.zeros(n, dtype=torch.float32, device=dev()),
           "token_loss": torch.zeros(n, dtype=torch.float32, device=dev()),
           "grad_logits": torch.zeros((n, (ow.vocab + 7) // 8 * 8), dtype=torch.bfloat16, device=dev())}

    def run(stream=None):
        bd.opd_loss(*ins, out={**out, "vocab": ow.vocab}, stream=stream)

    run()
    torch.cuda.synchronize()
    assert abs(float(out["loss"].cpu()[0]) - ref["loss"]) <= 1e-4 * max(1.0, abs(ref["loss"]))
    # the gradient's columns past the vocabulary (row padding) are never written
    checked = [out[k] for k in ("loss", "token_logp", "token_weight", "token_loss")]
    checked.append(out["grad_logits"][:, :ow.vocab])
    eager = [t.clone() for t in checked]
    g = capture(run)
    replay_and_check(g, checked, eager, lambda t: t.fill_(float("nan")), lambda: run())
    del g

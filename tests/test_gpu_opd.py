"""Fused OPD token loss and logits gradient (ctx_opd_loss_run) against the CPU
oracle (App. OPD Optimization: eq:opd-token-advantage ... eq:opd-surrogate)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import workloads as wl

from _gpu_util import dev, up_bf16

pytestmark = pytest.mark.gpu

# Tolerances from the arithmetic: the fp32 log-sum-exp over <= 155k terms is
# good to a few 1e-6 absolute, so lp, the ratio and the token losses carry
# relative errors near 1e-6; gradients are rounded to bf16 (half an ulp is at
# most 2^-8 relative: 8 significant bits), checked at 2^-8 relative plus 1e-5
# of the row's scale.
LP_ATOL = 1e-4
LOSS_RTOL, LOSS_ATOL = 1e-4, 1e-5
GRAD_RTOL = 2.0 ** -8


def up(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev()).to(dtype)


def run_gpu(z_dev, b: wl.OpdBatch, vocab, grad=True, params=None, grad_stride=None):
    out = {"vocab": vocab}
    n = b.num_tokens
    if grad and grad_stride is not None:
        out["grad_logits"] = torch.full((n, grad_stride), -7.0, dtype=torch.bfloat16, device=dev())
    r = bd.opd_loss(z_dev, up(b.tokens, torch.int32), up(b.old_lp, torch.float32), up(b.teacher_lp, torch.float32),
                    up(b.mask, torch.uint8), up(b.seq_starts, torch.int32), params=params, grad=grad, out=out)
    torch.cuda.synchronize()
    return {k: (v.float().cpu().numpy() if v.dtype == torch.bfloat16 else v.cpu().numpy()) for k, v in r.items()}


def near_kink(ref, b, params=bd.OpdParams()):
    """Tokens whose branch of eq:opd-ratio / eq:opd-dual-clip sits within
    rounding of a kink: either side's gradient is a correct result there."""
    r = ref["lp"] - b.old_lp.astype(np.float64)
    rho = np.exp(np.clip(r, -params.log_ratio_clip, params.log_ratio_clip))
    a = b.teacher_lp.astype(np.float64) - b.old_lp
    rel = lambda x, y: np.abs(x - y) <= 1e-4 * np.abs(y)  # noqa: E731
    return (rel(rho, 1 - params.clip_delta) | rel(rho, 1 + params.clip_delta) | rel(rho, params.dual_clip)
            | (np.abs(np.abs(r) - params.log_ratio_clip) < 1e-3) | (np.abs(a) < 1e-6))


def check_scalars(got, ref, b, what):
    m = b.mask.astype(bool)
    np.testing.assert_allclose(got["token_logp"][m], ref["lp"][m], rtol=0, atol=LP_ATOL, err_msg=what)
    assert (got["token_logp"][~m] == 0).all() and (got["token_loss"][~m] == 0).all()
    np.testing.assert_allclose(got["token_weight"], ref["weight"], rtol=1e-6, atol=0, err_msg=what)
    np.testing.assert_allclose(got["token_loss"], ref["token_loss"], rtol=LOSS_RTOL, atol=LOSS_ATOL, err_msg=what)
    assert got["loss"][0] == pytest.approx(ref["loss"], rel=LOSS_RTOL, abs=LOSS_ATOL), what


def check_grad_rows(got_rows, ref_rows, dlp_rows, what, rows=None, tokens=None):
    scale = np.maximum(np.abs(ref_rows).max(axis=1, keepdims=True), 1e-30)
    err = np.abs(got_rows - ref_rows)
    bad = err > GRAD_RTOL * np.abs(ref_rows) + 1e-5 * scale
    if bad.any():
        for i, c in list(zip(*np.nonzero(bad)))[:12]:
            r = rows[i] if rows is not None else i
            print(f"{what}: row {r} col {c} got {got_rows[i, c]:.4e} ref {ref_rows[i, c]:.4e} "
                  f"dlp {dlp_rows[i]:.3e} token {tokens[r] if tokens is not None else '?'}", flush=True)
    assert not bad.any(), f"{what}: {bad.sum()} gradient entries off, worst {err.max():.3e}"
    assert np.isfinite(got_rows).all()


@pytest.mark.parametrize("name", ["opd_tiny"])
def test_opd_parity_small(name):
    w = wl.OPD_WORKLOADS[name]
    b = wl.opd_batch(w)
    zh = wl.opd_logits_host(w, b)
    ref = oracle.opd_loss(zh[:, :w.vocab], b.tokens, b.old_lp, b.teacher_lp, b.mask, b.seq_starts)
    got = run_gpu(up_bf16(zh), b, w.vocab, grad_stride=w.row_stride)
    check_scalars(got, ref, b, name)
    ok = ~near_kink(ref, b)
    rows = np.nonzero(ok)[0]
    gref = oracle.opd_grad_rows(zh[:, :w.vocab], b.tokens, b.mask, ref["dlp"], rows)
    check_grad_rows(got["grad_logits"][rows, :w.vocab], gref, ref["dlp"][rows], name)
    # columns >= vocab untouched, masked rows all zero
    assert (got["grad_logits"][:, w.vocab:] == -7.0).all()
    assert (got["grad_logits"][b.mask == 0, :w.vocab] == 0).all()
    # every clipping regime is present in the batch
    a = b.teacher_lp.astype(np.float64) - b.old_lp
    rho = np.exp(np.clip(ref["lp"] - b.old_lp, -20, 20))
    m = b.mask.astype(bool)
    assert ((a > 0) & (rho > 1.2) & m).any() and ((a < 0) & (rho > 3) & m).any()
    assert ((a < 0) & (rho < 0.8) & m).any() and ((rho > 0.8) & (rho < 1.2) & m).any()


def test_opd_edge_batches():
    """Empty responses, a fully masked response, length-1 responses, a vocab
    below one chunk and one of exactly one chunk per thread round."""
    rng = np.random.default_rng(9)
    for vocab, stride in [(7, 8), (8, 8), (8193, 8200), (4096, 4096), (50257, 50264)]:
        lens = np.array([0, 1, 5, 0, 3, 1])
        starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        n = int(starts[-1])
        mask = np.ones(n, np.uint8)
        mask[starts[4]:starts[5]] = 0  # fully masked response
        tokens = rng.integers(0, vocab, n).astype(np.int32)
        old = (-rng.exponential(1.0, n) + rng.normal(0, 0.5, n)).astype(np.float32)
        tea = (old + rng.normal(0, 1, n)).astype(np.float32)
        b = wl.OpdBatch(starts, tokens, mask, np.zeros(n), old, tea)
        z = (2 * rng.standard_normal((n, stride))).astype(np.float32)
        z[:, vocab:] = np.nan
        zh = wl.f32_to_bf16_bits(z)
        ref = oracle.opd_loss(zh[:, :vocab], tokens, old, tea, mask, starts)
        got = run_gpu(up_bf16(zh), b, vocab, grad_stride=stride)
        check_scalars(got, ref, b, f"vocab {vocab}")
        rows = np.nonzero(~near_kink(ref, b))[0]
        gref = oracle.opd_grad_rows(zh[:, :vocab], tokens, mask, ref["dlp"], rows)
        check_grad_rows(got["grad_logits"][rows, :vocab], gref, ref["dlp"][rows], f"vocab {vocab}")
        assert (got["grad_logits"][:, vocab:] == -7.0).all()


def test_opd_loss_only_matches_and_is_deterministic():
    w = wl.OPD_WORKLOADS["opd_tiny"]
    b = wl.opd_batch(w)
    z = up_bf16(wl.opd_logits_host(w, b))
    g1 = run_gpu(z, b, w.vocab, grad=True)
    g2 = run_gpu(z, b, w.vocab, grad=True)
    f = run_gpu(z, b, w.vocab, grad=False)
    for k in ("loss", "token_logp", "token_loss", "token_weight"):
        assert np.array_equal(g1[k], g2[k]) and np.array_equal(g1[k], f[k]), k
    assert np.array_equal(g1["grad_logits"], g2["grad_logits"])


def test_opd_params_change_the_regimes():
    """delta and kappa are honoured: with the band closed (delta = 0) and a
    large kappa the loss equals the oracle run with the same constants."""
    w = wl.OPD_WORKLOADS["opd_tiny"]
    b = wl.opd_batch(w)
    zh = wl.opd_logits_host(w, b)
    prm = bd.OpdParams(log_ratio_clip=5.0, clip_delta=0.0, dual_clip=10.0, eps=1e-3)
    ref = oracle.opd_loss(zh[:, :w.vocab], b.tokens, b.old_lp, b.teacher_lp, b.mask, b.seq_starts,
                          clip_log=5.0, delta=0.0, kappa=10.0, eps=1e-3)
    got = run_gpu(up_bf16(zh), b, w.vocab, params=prm)
    check_scalars(got, ref, b, "custom params")


def test_opd_full_size_qwen3_batch():
    """The full batch (64 responses, ~17k tokens, vocabulary 151,936): every
    token's lp and loss and the batch loss against the oracle, and the
    gradient rows of sampled tokens."""
    w = wl.OPD_WORKLOADS["opd_qwen3"]
    b = wl.opd_batch(w)
    z = wl.opd_logits_device(w, b, dev())
    got = run_gpu(z, b, w.vocab)
    zh = z.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = oracle.opd_loss(zh, b.tokens, b.old_lp, b.teacher_lp, b.mask, b.seq_starts)
    check_scalars(got, ref, b, "opd_qwen3")
    rng = np.random.default_rng(4)
    ok = np.nonzero(~near_kink(ref, b) & (ref["dlp"] != 0))[0]
    rows = np.sort(np.concatenate([rng.choice(ok, 10, replace=False), np.nonzero(b.mask == 0)[0][:2],
                                   np.nonzero(ref["dlp"] == 0)[0][:2]]))
    gref = oracle.opd_grad_rows(zh, b.tokens, b.mask, ref["dlp"], rows)
    check_grad_rows(got["grad_logits"][rows], gref, ref["dlp"][rows], "opd_qwen3", rows, b.tokens)
    print(f"opd_qwen3: loss {got['loss'][0]:.6f} vs {ref['loss']:.6f}; "
          f"lp max err {np.abs(got['token_logp'] - ref['lp'])[b.mask == 1].max():.2e}", flush=True)


def test_opd_abi_errors():
    lib = bd.load_library()
    n, vocab = 4, 64
    z = torch.zeros((n, vocab), dtype=torch.bfloat16, device=dev())
    i = torch.zeros(n, dtype=torch.int32, device=dev())
    f = torch.zeros(n, dtype=torch.float32, device=dev())
    m = torch.ones(n, dtype=torch.uint8, device=dev())
    st = torch.tensor([0, n], dtype=torch.int32, device=dev())
    g = torch.zeros((n, vocab), dtype=torch.bfloat16, device=dev())
    loss = torch.zeros(1, dtype=torch.float32, device=dev())
    P = lambda t, off=0: t.data_ptr() + off  # noqa: E731
    good = bd.OpdParams()

    def call(logits=P(z), stride=vocab, v=vocab, params=good, grad=P(g), gstride=vocab, weight=P(f), nseq=1):
        return lib.ctx_opd_loss_run(logits, stride, v, P(i), P(f), P(f), P(m), P(st), nseq, n,
                                    ctypes.byref(params) if params is not None else None, None, weight, P(f),
                                    P(loss), grad, gstride, None)

    assert call() == bd.CTX_OK
    assert call(params=None) == bd.CTX_ERR_INVALID_ARG
    assert call(params=bd.OpdParams(clip_delta=1.0)) == bd.CTX_ERR_INVALID_ARG
    assert call(params=bd.OpdParams(dual_clip=1.0)) == bd.CTX_ERR_INVALID_ARG
    assert call(params=bd.OpdParams(log_ratio_clip=float("nan"))) == bd.CTX_ERR_INVALID_ARG
    assert call(stride=60) == bd.CTX_ERR_INVALID_ARG        # below vocab
    assert call(stride=68, v=64) == bd.CTX_ERR_INVALID_ARG  # not a multiple of 8
    assert call(v=155649, stride=155656) == bd.CTX_ERR_UNSUPPORTED
    assert call(logits=P(z, 2)) == bd.CTX_ERR_ALIGNMENT
    assert call(weight=None) == bd.CTX_ERR_INVALID_ARG
    assert call(nseq=0) == bd.CTX_ERR_INVALID_ARG            # tokens without responses
    assert call(grad=None) == bd.CTX_OK
    # an empty batch: the per-token arrays may be NULL; only loss and seq_starts are needed
    st0 = torch.zeros(2, dtype=torch.int32, device=dev())  # one empty response
    assert lib.ctx_opd_loss_run(None, vocab, vocab, None, None, None, None, P(st0), 1, 0, ctypes.byref(good),
                                None, None, None, P(loss), None, 0, None) == bd.CTX_OK
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0
    assert bd.load_library().ctx_decode_attn_last_error() is not None

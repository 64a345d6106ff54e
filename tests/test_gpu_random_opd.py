"""A seeded random sweep of the fused OPD loss and gradient against the oracle:
vocabularies from a few entries to the 155,648 maximum (around the 8-entry
chunk and 8,192-entry round boundaries too), padded row strides, empty and
fully masked responses, random masks, clipping constants and logit scales,
with and without the gradient."""
import numpy as np
import pytest

import oracle
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import workloads as wl

from _gpu_util import up_bf16
from test_gpu_opd import check_grad_rows, check_scalars, near_kink, run_gpu

pytestmark = pytest.mark.gpu


def vocabulary(rng):
    kind = rng.integers(0, 4)
    if kind == 0:
        return int(rng.integers(1, 65))
    if kind == 1:
        return int(rng.integers(65, 10_000))
    if kind == 2:
        return int(8192 * rng.integers(1, 19) + rng.integers(-1, 2))
    return int(rng.integers(10_000, 155_649))


@pytest.mark.parametrize("case", range(10))
def test_random_opd(case):
    rng = np.random.default_rng(9300 + case)
    vocab = min(vocabulary(rng), 155_648)
    stride = -(-vocab // 8) * 8 + 8 * int(rng.integers(0, 3))
    nresp = int(rng.integers(1, 13))
    lens = rng.integers(0, 41, size=nresp)
    lens[rng.random(nresp) < 0.15] = 0
    starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n = int(starts[-1])
    mask = (rng.random(n) > rng.uniform(0.0, 0.3)).astype(np.uint8)
    if nresp > 1 and lens[0] > 0:
        mask[starts[0]:starts[1]] = 0  # a fully masked response
    tokens = rng.integers(0, vocab, n).astype(np.int32)
    old = (-rng.exponential(1.0, n) + rng.normal(0, 0.5, n)).astype(np.float32)
    tea = (old + rng.normal(0, rng.uniform(0.2, 2.0), n)).astype(np.float32)
    b = wl.OpdBatch(starts, tokens, mask, np.zeros(n), old, tea)
    z = (rng.uniform(0.5, 4.0) * rng.standard_normal((n, stride))).astype(np.float32)
    z[:, vocab:] = np.nan  # columns past the vocabulary are never read
    zh = wl.f32_to_bf16_bits(z)
    if rng.random() < 0.5:
        prm = bd.OpdParams()
        kw = {}
    else:
        clip, delta, kappa = float(rng.uniform(1.0, 20.0)), float(rng.uniform(0.0, 0.5)), float(rng.uniform(1.5, 5.0))
        eps = float(rng.choice([1e-8, 1e-3, 0.0]))
        prm = bd.OpdParams(log_ratio_clip=clip, clip_delta=delta, dual_clip=kappa, eps=eps)
        kw = dict(clip_log=clip, delta=delta, kappa=kappa, eps=eps)
    grad = bool(rng.random() < 0.7)
    what = f"case {case}: vocab {vocab}, stride {stride}, {nresp} responses, {n} tokens, grad {grad}"
    print(what, flush=True)
    ref = oracle.opd_loss(zh[:, :vocab], tokens, old, tea, mask, starts, **kw)
    got = run_gpu(up_bf16(zh), b, vocab, grad=grad, params=prm, grad_stride=stride if grad else None)
    check_scalars(got, ref, b, what)
    if grad and n:
        rows = np.nonzero(~near_kink(ref, b, prm))[0]
        gref = oracle.opd_grad_rows(zh[:, :vocab], tokens, mask, ref["dlp"], rows)
        check_grad_rows(got["grad_logits"][rows, :vocab], gref, ref["dlp"][rows], what, rows, tokens)
        assert (got["grad_logits"][:, vocab:] == -7.0).all(), f"{what}: columns past the vocabulary written"

"""Parity of the HIP decode-attention path against the CPU oracle, through the C ABI.

Inputs are the seeded bf16 workloads; the gate is max-abs <= 1e-2 and
mean-abs <= 1e-3 over every checked output element (fp32 out), with a much
tighter bound on max-abs to catch small indexing or accumulation slips.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import DecodeAttention

from _gpu_util import assert_parity, up_bf16, up_i32, dev

pytestmark = pytest.mark.gpu


def run_layer(w, lay, q, k, v, lens=None, split_tokens=0, out_dtype=torch.float32, max_seq_len=None):
    lens = lay.lens if lens is None else lens
    with DecodeAttention(w.num_q_heads, w.num_kv_heads, len(lens), max_seq_len or max(lay.max_seq_len, 1),
                         out_dtype=out_dtype, split_tokens=split_tokens) as attn:
        out = torch.empty((len(lens), w.num_q_heads, w.head_dim), dtype=out_dtype, device=dev())
        attn.run(up_bf16(q), up_bf16(k), up_bf16(v), up_i32(lay.offsets), up_i32(lens), w.scale, out)
        torch.cuda.synchronize()
    return out.float().cpu().numpy()


def full_check(w, seed=wl.DEFAULT_SEED, split_tokens=0, **layout_kw):
    lay = wl.workload_layout(w, seed, **layout_kw)
    q = wl.query_bits(w, 0, 0, seed)
    k, v = wl.layer_kv_bits(w, lay, 0, seed)
    ref = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale)
    got = run_layer(w, lay, q, k, v, split_tokens=split_tokens)
    return got, ref


def test_tiny_full():
    got, ref = full_check(wl.WORKLOADS["tiny"])
    assert_parity(got, ref, "tiny")


REDUCED = {
    # same heads, value distributions and length kinds; lengths cut so the
    # oracle finishes in seconds while spanning many 16-token blocks and
    # ragged tails
    "student_0p6b_1p7b": dict(batch=64, lengths=(100, 700)),
    "student_4b": dict(batch=64, lengths=(200, 900)),
    "act_first_burst": dict(batch=48, lengths=(300, 1200)),
    "long_ragged": dict(batch=32, lengths=(17, 4000)),
}


@pytest.mark.parametrize("name", list(REDUCED))
def test_reduced_workloads_full(name):
    w = wl.small_workload(wl.WORKLOADS[name], **REDUCED[name])
    got, ref = full_check(w)
    assert_parity(got, ref, f"{name} reduced")


def test_large_batch_forced_splits():
    """More than 64 sequences (the wave-wide prefix search runs in chunks) and
    forced split sizes that cut most sequences several times."""
    w = wl.small_workload(wl.WORKLOADS["act_first_burst"], batch=150, lengths=(16, 700))
    lay = wl.workload_layout(w)
    q = wl.query_bits(w, 0)
    k, v = wl.layer_kv_bits(w, lay, 0)
    ref = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale)
    for split in (0, 16, 112, 1000):
        got = run_layer(w, lay, q, k, v, split_tokens=split)
        assert_parity(got, ref, f"B=150 split={split}")

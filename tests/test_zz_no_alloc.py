"""ctx_decode_attn_run_static (no handle, no allocation: the split workspace is
the library's static device array) against ctx_decode_attn_run, through the C ABI.

Two calls in a row, the second with a smaller batch, then one with twice the
KV heads, each bit for bit equal to the handle's run on the same inputs and
within the parity gate of the oracle; then a call whose workspace would exceed
the static array is refused."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36608_amd import binding as bd
from paper_2609_36608_amd import workloads as wl
from paper_2609_36608_amd.binding import DecodeAttention

from _gpu_util import assert_parity, dev, up_bf16, up_i32

pytestmark = pytest.mark.gpu


def case(seed, batch, hq, hkv, lo, hi):
    w = wl.Workload(f"static{seed}", 170 + seed, 1, batch, hq, hkv, 1, "uniform", lo, hi)
    rng = np.random.default_rng(seed)
    lay = wl.make_layout(wl.draw_lengths(w), 1, gap_max=3, shuffle=True, rng=rng)
    k, v = wl.layer_kv_bits(w, lay, 0)
    q = wl.query_bits(w, 0)
    return w, lay, q, k, v


def static_run(desc, q, k, v, offs, lens, scale, out):
    lib = bd.load_library()
    stream = torch.cuda.current_stream().cuda_stream
    return lib.ctx_decode_attn_run_static(ctypes.byref(desc), q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                          offs.data_ptr(), lens.data_ptr(), q.shape[0], ctypes.c_float(scale),
                                          out.data_ptr(), stream)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_static_entry_matches_the_handle_run(out_dtype):
    code = bd.CTX_DTYPE_F32 if out_dtype == torch.float32 else bd.CTX_DTYPE_BF16
    # The first call is the larger one, so the second reuses a workspace holding
    # stale partials.  The third has twice the KV heads with the same workgroup
    # shape: its split (ranges per KV head) must follow its own head count, as a
    # handle's does, for the two results to agree bit for bit.
    for seed, batch, lo, hi, hq, hkv in [(1, 256, 16, 1200, 32, 8), (2, 37, 1, 900, 32, 8),
                                         (4, 40, 1, 900, 32, 16)]:
        w, lay, q, k, v = case(seed, batch, hq, hkv, lo, hi)
        qd, kd, vd = up_bf16(q), up_bf16(k), up_bf16(v)
        offs, lens = up_i32(lay.offsets), up_i32(lay.lens)
        desc = bd.CtxDesc(hq, hkv, 128, 256, int(lay.lens.max()), code, 0, 0)
        buf = torch.full((batch + 1, hq, 128), -3.0, dtype=out_dtype, device=dev())
        got = buf[:batch]
        assert static_run(desc, qd, kd, vd, offs, lens, w.scale, got) == bd.CTX_OK
        torch.cuda.synchronize()
        assert (buf[batch] == -3.0).all(), "write past the end of out"
        with DecodeAttention(hq, hkv, 256, int(lay.lens.max()), out_dtype=out_dtype) as attn:
            want = torch.empty_like(got)
            attn.run(qd, kd, vd, offs, lens, w.scale, want)
            torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16) if out_dtype == torch.bfloat16 else got.view(torch.int32),
                           want.view(torch.int16) if out_dtype == torch.bfloat16 else want.view(torch.int32)), \
            f"static entry differs from the handle run (batch {batch}, {hq}/{hkv} heads)"
        ref = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale)
        assert_parity(got.float().cpu().numpy(), ref, f"static entry, batch {batch}, {hq}/{hkv} heads, {out_dtype}",
                      tight=out_dtype == torch.float32)


def test_static_entry_python_binding_and_capacity():
    w, lay, q, k, v = case(3, 12, 16, 8, 1, 700)
    qd, kd, vd = up_bf16(q), up_bf16(k), up_bf16(v)
    offs, lens = up_i32(lay.offsets), up_i32(lay.lens)
    out = torch.empty((12, 16, 128), dtype=torch.float32, device=dev())
    bd.ctx_decode_attn_run_static(qd, kd, vd, offs, lens, w.scale, out, num_kv_heads=8)
    torch.cuda.synchronize()
    ref = oracle.decode_attn(q, k, v, lay.offsets, lay.lens, w.scale)
    assert_parity(out.cpu().numpy(), ref, "static entry through the binding")
    # an empty batch is a no-op through the binding as through the C ABI
    assert bd.ctx_decode_attn_run_static(qd[:0], kd, vd, offs[:0], lens[:0], w.scale, out[:0],
                                         num_kv_heads=8).shape[0] == 0
    torch.cuda.synchronize()
    # 128 query heads: even one sequence needs more than the static workspace holds
    big = torch.zeros((1, 128, 128), dtype=torch.bfloat16, device=dev())
    kv = torch.zeros((4, 8, 128), dtype=torch.bfloat16, device=dev())
    o = torch.zeros((1, 128, 128), dtype=torch.float32, device=dev())
    one = torch.ones(1, dtype=torch.int32, device=dev())
    zero = torch.zeros(1, dtype=torch.int32, device=dev())
    desc = bd.CtxDesc(128, 8, 128, 4, 4, bd.CTX_DTYPE_F32, 0, 0)
    assert static_run(desc, big, kv, kv, zero, one, 0.1, o) == bd.CTX_ERR_CAPACITY
    assert "exceeds the static" in bd.load_library().ctx_decode_attn_last_error().decode()
    torch.cuda.synchronize()

"""C-ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects bad arguments before touching the device."""
import ctypes
import glob
import os
import re

import pytest

from paper_2609_36608_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for hdr in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(hdr).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    return bd.load_library()


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(bd.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, -6):
        s = lib.ctx_decode_attn_status_string(code).decode()
        assert s and s != "unknown status"
    assert lib.ctx_decode_attn_status_string(17).decode() == "unknown status"


def good_desc(**kw):
    d = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, max_batch=32, max_seq_len=4096,
             out_dtype=bd.CTX_DTYPE_F32, split_tokens=0)
    d.update(kw)
    return bd.CtxDesc(**d)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), bd.CTX_ERR_UNSUPPORTED),
    (dict(head_dim=256), bd.CTX_ERR_UNSUPPORTED),
    (dict(num_q_heads=12, num_kv_heads=8), bd.CTX_ERR_UNSUPPORTED),
    (dict(num_q_heads=64, num_kv_heads=2), bd.CTX_ERR_UNSUPPORTED),   # group 32 > 16
    (dict(num_q_heads=0), bd.CTX_ERR_INVALID_ARG),
    (dict(num_kv_heads=-1), bd.CTX_ERR_INVALID_ARG),
    (dict(max_batch=0), bd.CTX_ERR_INVALID_ARG),
    (dict(max_seq_len=0), bd.CTX_ERR_INVALID_ARG),
    (dict(out_dtype=7), bd.CTX_ERR_INVALID_ARG),
    (dict(split_tokens=5), bd.CTX_ERR_INVALID_ARG),
    (dict(split_tokens=-16), bd.CTX_ERR_INVALID_ARG),
])
def test_create_rejects_bad_desc(lib, kw, status):
    h = ctypes.c_void_p(1234)
    rc = lib.ctx_decode_attn_create(ctypes.byref(good_desc(**kw)), ctypes.byref(h))
    assert rc == status
    assert h.value is None
    assert lib.ctx_decode_attn_last_error().decode()


def test_create_null_arguments(lib):
    h = ctypes.c_void_p()
    assert lib.ctx_decode_attn_create(None, ctypes.byref(h)) == bd.CTX_ERR_INVALID_ARG
    assert lib.ctx_decode_attn_create(ctypes.byref(good_desc()), None) == bd.CTX_ERR_INVALID_ARG


def test_run_and_destroy_null_handle(lib):
    assert lib.ctx_decode_attn_run(None, 16, 16, 16, 16, 16, 1, 0.1, 16, None) == bd.CTX_ERR_INVALID_ARG
    assert lib.ctx_decode_attn_destroy(None) == bd.CTX_OK


def test_valid_desc_without_gpu_reports_hip_error_or_succeeds(lib):
    """On a machine without a GPU a valid create fails cleanly with CTX_ERR_HIP
    (no crash, no handle); with a GPU it succeeds."""
    h = ctypes.c_void_p()
    rc = lib.ctx_decode_attn_create(ctypes.byref(good_desc()), ctypes.byref(h))
    if rc == bd.CTX_OK:
        assert h.value is not None
        assert lib.ctx_decode_attn_destroy(h) == bd.CTX_OK
    else:
        assert rc == bd.CTX_ERR_HIP
        assert h.value is None


@pytest.mark.parametrize("kw,num_seqs,status", [
    (dict(split_tokens=64), 4, bd.CTX_ERR_UNSUPPORTED),
    (dict(page_tokens=16), 4, bd.CTX_ERR_UNSUPPORTED),
    (dict(head_dim=64), 4, bd.CTX_ERR_UNSUPPORTED),
    (dict(out_dtype=7), 4, bd.CTX_ERR_INVALID_ARG),
    (dict(max_batch=8), 9, bd.CTX_ERR_CAPACITY),
    (dict(), -1, bd.CTX_ERR_INVALID_ARG),
])
def test_static_run_rejects_bad_arguments_before_the_device(lib, kw, num_seqs, status):
    """The allocation-free entry point checks its descriptor and sizes first."""
    rc = lib.ctx_decode_attn_run_static(ctypes.byref(good_desc(**kw)), 16, 16, 16, 16, 16, num_seqs, 0.1, 16, None)
    assert rc == status
    assert lib.ctx_decode_attn_last_error().decode()


def test_static_run_null_and_empty(lib):
    assert lib.ctx_decode_attn_run_static(None, 16, 16, 16, 16, 16, 1, 0.1, 16, None) == bd.CTX_ERR_INVALID_ARG
    assert lib.ctx_decode_attn_run_static(ctypes.byref(good_desc()), 16, 16, 16, 16, 16, 0, 0.1, 16, None) == bd.CTX_OK
    assert lib.ctx_decode_attn_run_static(ctypes.byref(good_desc()), None, 16, 16, 16, 16, 1, 0.1, 16,
                                          None) == bd.CTX_ERR_INVALID_ARG
    assert lib.ctx_decode_attn_run_static(ctypes.byref(good_desc()), 16, 16, 16, 16, 16, 1, float("nan"), 16,
                                          None) == bd.CTX_ERR_INVALID_ARG
    assert lib.ctx_decode_attn_run_static(ctypes.byref(good_desc()), 18, 16, 16, 16, 16, 1, 0.1, 16,
                                          None) == bd.CTX_ERR_ALIGNMENT


@pytest.mark.parametrize("args,status", [
    ((None, 16, 16, 1, 0), bd.CTX_ERR_INVALID_ARG),        # NULL source
    ((16, 16, None, 1, 0), bd.CTX_ERR_INVALID_ARG),        # NULL sink / destination
    ((16, 0, 16, 1, 0), bd.CTX_ERR_INVALID_ARG),           # no bytes
    ((16, 24, 16, 1, 0), bd.CTX_ERR_INVALID_ARG),          # not whole 16-byte chunks
    ((16, 16, 16, 0, 0), bd.CTX_ERR_INVALID_ARG),          # empty grid
    ((16, 16, 16, 1, 2), bd.CTX_ERR_INVALID_ARG),          # unknown flag bit
    ((24, 16, 16, 1, 0), bd.CTX_ERR_ALIGNMENT),            # misaligned source
    ((16, 16, 8, 1, 0), bd.CTX_ERR_ALIGNMENT),             # misaligned sink / destination
])
def test_streaming_probes_reject_bad_arguments_before_the_device(lib, args, status):
    src, nbytes, other, wg, flags = args
    assert lib.ctx_hbm_read(src, nbytes, other, wg, flags, None) == status
    assert lib.ctx_hbm_copy(src, other, nbytes, wg, flags, None) == status
    assert lib.ctx_decode_attn_last_error().decode()


@pytest.mark.parametrize("args,status", [
    ((2, 1, 1, 16), bd.CTX_ERR_INVALID_ARG),               # unknown MFMA shape
    ((bd.CTX_MFMA_16X16X32, 0, 1, 16), bd.CTX_ERR_INVALID_ARG),    # empty grid
    ((bd.CTX_MFMA_32X32X16, 1, 0, 16), bd.CTX_ERR_INVALID_ARG),    # no iterations
    ((bd.CTX_MFMA_16X16X32, 1, 1, None), bd.CTX_ERR_INVALID_ARG),  # NULL sink
    ((bd.CTX_MFMA_16X16X32, 1, 1, 8), bd.CTX_ERR_ALIGNMENT),       # misaligned sink
])
def test_mfma_probe_rejects_bad_arguments_before_the_device(lib, args, status):
    shape, wg, iters, sink = args
    assert lib.ctx_mfma_bf16(shape, wg, iters, sink, None) == status
    assert lib.ctx_decode_attn_last_error().decode()

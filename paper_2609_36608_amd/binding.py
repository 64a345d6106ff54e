"""ctypes binding of libctx_decode_attn.so: argument marshalling only.

Every step of the attention runs in the library's HIP kernels; PyTorch only
provides device memory and the stream.  There is no fallback: if the library
is missing, loading fails with an error that says how to build it.
"""
from __future__ import annotations

import ctypes
import os

from .build import LIB

CTX_OK = 0
CTX_ERR_INVALID_ARG = -1
CTX_ERR_UNSUPPORTED = -2
CTX_ERR_CAPACITY = -3
CTX_ERR_ALIGNMENT = -4
CTX_ERR_HIP = -5
CTX_ERR_OOM = -6

CTX_DTYPE_BF16 = 0
CTX_DTYPE_F32 = 1

CTX_PREFILL_SPLIT_P = 1  # ctx_prefill_attn_run flag: softmax weights as two bf16 terms
CTX_STATIC_SCRATCH_BYTES = 16 << 20  # static workspace of ctx_decode_attn_run_static, per device
CTX_HBM_SINK_BYTES_PER_WORKGROUP = 64
CTX_HBM_NONTEMPORAL = 1
CTX_MFMA_16X16X32 = 0
CTX_MFMA_32X32X16 = 1
MFMA_FLOPS_PER_WAVE_ROUND = {CTX_MFMA_16X16X32: 8 * 16 * 16 * 32 * 2, CTX_MFMA_32X32X16: 8 * 32 * 32 * 16 * 2}

# every function the C header declares
EXPORTS = (
    "ctx_decode_attn_create",
    "ctx_decode_attn_run",
    "ctx_decode_attn_run_static",
    "ctx_decode_attn_run_paged",
    "ctx_prefill_attn_run",
    "ctx_opd_loss_run",
    "ctx_rollout_simulate",
    "ctx_rollout_simulate_engine",
    "ctx_hbm_read",
    "ctx_hbm_copy",
    "ctx_mfma_bf16",
    "ctx_decode_attn_destroy",
    "ctx_decode_attn_status_string",
    "ctx_decode_attn_last_error",
)


class CtxDesc(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("max_batch", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32),
        ("out_dtype", ctypes.c_int),
        ("split_tokens", ctypes.c_int32),
        ("page_tokens", ctypes.c_int32),
    ]


class OpdParams(ctypes.Structure):
    """ctx_opd_loss_params; defaults are the paper's values (App. OPD Optimization)."""
    _fields_ = [
        ("log_ratio_clip", ctypes.c_float),
        ("clip_delta", ctypes.c_float),
        ("dual_clip", ctypes.c_float),
        ("eps", ctypes.c_float),
    ]

    def __init__(self, log_ratio_clip=20.0, clip_delta=0.2, dual_clip=3.0, eps=1e-8):
        super().__init__(log_ratio_clip, clip_delta, dual_clip, eps)


class RolloutConfig(ctypes.Structure):
    _fields_ = [("policy", ctypes.c_int32), ("num_tasks", ctypes.c_int32), ("turns", ctypes.c_int32),
                ("max_concurrency", ctypes.c_int32)]


class RolloutEngine(ctypes.Structure):
    _fields_ = [("step_base", ctypes.c_double), ("step_per_kv_token", ctypes.c_double),
                ("prefill_per_token", ctypes.c_double), ("fast_tokens", ctypes.c_int32),
                ("full_tokens", ctypes.c_int32)]


ROLLOUT_VANILLA = 0
ROLLOUT_ACTFIRST = 1


class CtxError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"ctx_decode_attn status {status}: {message}")
        self.status = status


_lib = None


def load_library(path: str | None = None):
    """Load the HIP library (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or LIB
    # torch ships its own libamdhip64.so.7; load it first so this library binds
    # to the same HIP runtime as the streams and memory torch hands us
    import torch  # noqa: F401

    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(path)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.ctx_decode_attn_create.argtypes = [ctypes.POINTER(CtxDesc), ctypes.POINTER(ctypes.c_void_p)]
    lib.ctx_decode_attn_create.restype = ctypes.c_int
    lib.ctx_decode_attn_run.argtypes = [vp, vp, vp, vp, vp, vp, i32, ctypes.c_float, vp, vp]
    lib.ctx_decode_attn_run.restype = ctypes.c_int
    lib.ctx_decode_attn_run_static.argtypes = [ctypes.POINTER(CtxDesc), vp, vp, vp, vp, vp, i32, ctypes.c_float,
                                               vp, vp]
    lib.ctx_decode_attn_run_static.restype = ctypes.c_int
    lib.ctx_decode_attn_run_paged.argtypes = [vp, vp, vp, vp, vp, i32, vp, i32, vp, vp, ctypes.c_float, vp, vp]
    lib.ctx_decode_attn_run_paged.restype = ctypes.c_int
    lib.ctx_prefill_attn_run.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, ctypes.c_float, ctypes.c_uint32,
                                         vp, vp]
    lib.ctx_prefill_attn_run.restype = ctypes.c_int
    lib.ctx_opd_loss_run.argtypes = [vp, ctypes.c_int64, i32, vp, vp, vp, vp, vp, i32, i32,
                                     ctypes.POINTER(OpdParams), vp, vp, vp, vp, vp, ctypes.c_int64, vp]
    lib.ctx_opd_loss_run.restype = ctypes.c_int
    lib.ctx_rollout_simulate.argtypes = [ctypes.POINTER(RolloutConfig), vp, vp, vp, vp, vp, vp]
    lib.ctx_rollout_simulate.restype = ctypes.c_int
    lib.ctx_rollout_simulate_engine.argtypes = [ctypes.POINTER(RolloutConfig), ctypes.POINTER(RolloutEngine), vp, vp,
                                                vp, vp, vp, vp]
    lib.ctx_rollout_simulate_engine.restype = ctypes.c_int
    lib.ctx_hbm_read.argtypes = [vp, ctypes.c_size_t, vp, i32, ctypes.c_uint32, vp]
    lib.ctx_hbm_read.restype = ctypes.c_int
    lib.ctx_hbm_copy.argtypes = [vp, vp, ctypes.c_size_t, i32, ctypes.c_uint32, vp]
    lib.ctx_hbm_copy.restype = ctypes.c_int
    lib.ctx_mfma_bf16.argtypes = [i32, i32, i32, vp, vp]
    lib.ctx_mfma_bf16.restype = ctypes.c_int
    lib.ctx_decode_attn_destroy.argtypes = [vp]
    lib.ctx_decode_attn_destroy.restype = ctypes.c_int
    lib.ctx_decode_attn_status_string.argtypes = [ctypes.c_int]
    lib.ctx_decode_attn_status_string.restype = ctypes.c_char_p
    lib.ctx_decode_attn_last_error.argtypes = []
    lib.ctx_decode_attn_last_error.restype = ctypes.c_char_p
    if path == LIB:
        _lib = lib
    return lib


def error_for(lib, status: int) -> CtxError:
    msg = lib.ctx_decode_attn_status_string(status).decode()
    detail = lib.ctx_decode_attn_last_error().decode()
    return CtxError(status, f"{msg}: {detail}" if detail else msg)


def _dtype_code(dtype) -> int:
    import torch

    if dtype == torch.float32:
        return CTX_DTYPE_F32
    if dtype == torch.bfloat16:
        return CTX_DTYPE_BF16
    raise ValueError(f"out dtype must be float32 or bfloat16, not {dtype}")


def _check_tensors(device: int, checks) -> None:
    """Each (name, tensor, dtype): that dtype, on cuda:device, contiguous."""
    for name, t, dt in checks:
        if t.dtype != dt:
            raise TypeError(f"{name} must be {dt}, got {t.dtype}")
        if not t.is_cuda or t.device.index != device:
            raise ValueError(f"{name} must be on cuda:{device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")


def _stream_ptr(stream, device=None) -> int:
    """hipStream_t of a torch stream (default: the current one of `device`) or a raw handle."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


class DecodeAttention:
    """Handle for ctx_decode_attn_run: decode-step GQA attention of one new token
    per sequence over ragged KV caches [rows, Hkv, 128] (bf16)."""

    def __init__(self, num_q_heads: int, num_kv_heads: int, max_batch: int, max_seq_len: int,
                 head_dim: int = 128, out_dtype=None, split_tokens: int = 0, page_tokens: int = 0):
        import torch

        self.lib = load_library()
        self.out_dtype = torch.float32 if out_dtype is None else out_dtype
        self.desc = CtxDesc(num_q_heads, num_kv_heads, head_dim, max_batch, max_seq_len,
                            _dtype_code(self.out_dtype), split_tokens, page_tokens)
        handle = ctypes.c_void_p()
        rc = self.lib.ctx_decode_attn_create(ctypes.byref(self.desc), ctypes.byref(handle))
        if rc != CTX_OK:
            raise error_for(self.lib, rc)
        self.handle = handle
        self.device = torch.cuda.current_device()

    def run(self, q, k_cache, v_cache, seq_offsets, seq_lens, scale: float, out, stream=None):
        import torch

        if self.handle is None:
            raise RuntimeError("handle is closed")
        d = self.desc
        _check_tensors(self.device, (("q", q, torch.bfloat16), ("k_cache", k_cache, torch.bfloat16),
                                     ("v_cache", v_cache, torch.bfloat16), ("seq_offsets", seq_offsets, torch.int32),
                                     ("seq_lens", seq_lens, torch.int32), ("out", out, self.out_dtype)))
        b = q.shape[0]
        if q.shape != (b, d.num_q_heads, d.head_dim) or out.shape != q.shape:
            raise ValueError(f"q/out must be [{b}, {d.num_q_heads}, {d.head_dim}]")
        if k_cache.dim() != 3 or k_cache.shape[1:] != (d.num_kv_heads, d.head_dim) or v_cache.shape != k_cache.shape:
            raise ValueError(f"k_cache/v_cache must be [rows, {d.num_kv_heads}, {d.head_dim}]")
        if seq_offsets.shape != (b,) or seq_lens.shape != (b,):
            raise ValueError(f"seq_offsets/seq_lens must be [{b}]")
        sp = _stream_ptr(stream)
        rc = self.lib.ctx_decode_attn_run(self.handle, q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                          seq_offsets.data_ptr(), seq_lens.data_ptr(), b, float(scale),
                                          out.data_ptr(), sp)
        if rc != CTX_OK:
            raise error_for(self.lib, rc)
        return out

    def run_paged(self, q, k_pages, v_pages, block_tables, seq_lens, scale: float, out,
                  k_new=None, v_new=None, stream=None):
        """Paged caches [num_pages, P, Hkv, D]; block_tables [B, max_pages] int32;
        optional k_new / v_new [B, Hkv, D] are appended as each sequence's
        newest token (written into its cache slot)."""
        import torch

        if self.handle is None:
            raise RuntimeError("handle is closed")
        d = self.desc
        if (k_new is None) != (v_new is None):
            raise ValueError("k_new and v_new go together")
        checks = [("q", q, torch.bfloat16), ("k_pages", k_pages, torch.bfloat16),
                  ("v_pages", v_pages, torch.bfloat16), ("block_tables", block_tables, torch.int32),
                  ("seq_lens", seq_lens, torch.int32), ("out", out, self.out_dtype)]
        if k_new is not None:
            checks += [("k_new", k_new, torch.bfloat16), ("v_new", v_new, torch.bfloat16)]
        _check_tensors(self.device, checks)
        b = q.shape[0]
        if q.shape != (b, d.num_q_heads, d.head_dim) or out.shape != q.shape:
            raise ValueError(f"q/out must be [{b}, {d.num_q_heads}, {d.head_dim}]")
        if k_pages.dim() != 4 or k_pages.shape[1:] != (d.page_tokens, d.num_kv_heads, d.head_dim) \
                or v_pages.shape != k_pages.shape:
            raise ValueError(f"k_pages/v_pages must be [pages, {d.page_tokens}, {d.num_kv_heads}, {d.head_dim}]")
        if block_tables.dim() != 2 or block_tables.shape[0] != b or seq_lens.shape != (b,):
            raise ValueError(f"block_tables must be [{b}, max_pages] and seq_lens [{b}]")
        if k_new is not None and (k_new.shape != (b, d.num_kv_heads, d.head_dim) or v_new.shape != k_new.shape):
            raise ValueError(f"k_new/v_new must be [{b}, {d.num_kv_heads}, {d.head_dim}]")
        sp = _stream_ptr(stream)
        rc = self.lib.ctx_decode_attn_run_paged(
            self.handle, q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(), block_tables.data_ptr(),
            block_tables.shape[1], seq_lens.data_ptr(), b,
            k_new.data_ptr() if k_new is not None else None, v_new.data_ptr() if v_new is not None else None,
            float(scale), out.data_ptr(), sp)
        if rc != CTX_OK:
            raise error_for(self.lib, rc)
        return out

    def prefill(self, q, k_cache, v_cache, seq_offsets, seq_lens, q_starts, q_lens, max_q_len: int,
                scale: float, out, stream=None, split_p: bool = False):
        """Causal prefill: q / out [total_q, Hq, D]; sequence b's q_lens[b] queries
        (rows q_starts[b] ..) are the last q_lens[b] of its seq_lens[b] cached rows.
        split_p: carry the softmax weights as two bf16 terms (CTX_PREFILL_SPLIT_P)
        instead of one."""
        import torch

        if self.handle is None:
            raise RuntimeError("handle is closed")
        d = self.desc
        _check_tensors(self.device, (("q", q, torch.bfloat16), ("k_cache", k_cache, torch.bfloat16),
                                     ("v_cache", v_cache, torch.bfloat16), ("seq_offsets", seq_offsets, torch.int32),
                                     ("seq_lens", seq_lens, torch.int32), ("q_starts", q_starts, torch.int32),
                                     ("q_lens", q_lens, torch.int32), ("out", out, self.out_dtype)))
        b = seq_lens.shape[0]
        if q.dim() != 3 or q.shape[1:] != (d.num_q_heads, d.head_dim) or out.shape != q.shape:
            raise ValueError(f"q/out must be [rows, {d.num_q_heads}, {d.head_dim}]")
        if k_cache.dim() != 3 or k_cache.shape[1:] != (d.num_kv_heads, d.head_dim) or v_cache.shape != k_cache.shape:
            raise ValueError(f"k_cache/v_cache must be [rows, {d.num_kv_heads}, {d.head_dim}]")
        if seq_offsets.shape != (b,) or q_starts.shape != (b,) or q_lens.shape != (b,):
            raise ValueError(f"seq_offsets, seq_lens, q_starts, q_lens must all be [{b}]")
        sp = _stream_ptr(stream)
        rc = self.lib.ctx_prefill_attn_run(self.handle, q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                           seq_offsets.data_ptr(), seq_lens.data_ptr(), q_starts.data_ptr(),
                                           q_lens.data_ptr(), b, int(max_q_len), float(scale),
                                           CTX_PREFILL_SPLIT_P if split_p else 0, out.data_ptr(), sp)
        if rc != CTX_OK:
            raise error_for(self.lib, rc)
        return out

    def close(self):
        if getattr(self, "handle", None) is not None:
            rc = self.lib.ctx_decode_attn_destroy(self.handle)
            self.handle = None
            if rc != CTX_OK:
                raise error_for(self.lib, rc)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ctx_decode_attn_run_static(q, k_cache, v_cache, seq_offsets, seq_lens, scale: float, out, num_kv_heads: int,
                               max_batch: int | None = None, stream=None):
    """ctx_decode_attn_run_static: the decode step with no handle and no
    allocation (the split workspace is the library's static device array).
    q / out [B, Hq, 128] (out float32 or bfloat16), caches [rows, Hkv, 128] bf16,
    seq_offsets / seq_lens [B] int32; max_batch defaults to B (1 for an empty batch)."""
    import torch

    lib = load_library()
    b, hq = q.shape[0], q.shape[1]
    device = q.device.index if q.is_cuda else -1
    _check_tensors(device, (("q", q, torch.bfloat16), ("k_cache", k_cache, torch.bfloat16),
                            ("v_cache", v_cache, torch.bfloat16), ("seq_offsets", seq_offsets, torch.int32),
                            ("seq_lens", seq_lens, torch.int32), ("out", out, out.dtype)))
    if q.dim() != 3 or out.shape != q.shape:
        raise ValueError("q/out must be [B, Hq, 128] of one shape")
    if k_cache.dim() != 3 or k_cache.shape[1] != num_kv_heads or v_cache.shape != k_cache.shape:
        raise ValueError(f"k_cache/v_cache must be [rows, {num_kv_heads}, 128]")
    if seq_offsets.shape != (b,) or seq_lens.shape != (b,):
        raise ValueError(f"seq_offsets/seq_lens must be [{b}]")
    desc = CtxDesc(hq, num_kv_heads, q.shape[2], max(b, 1) if max_batch is None else max_batch, 1,
                   _dtype_code(out.dtype), 0, 0)
    rc = lib.ctx_decode_attn_run_static(ctypes.byref(desc), q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                        seq_offsets.data_ptr(), seq_lens.data_ptr(), b, float(scale), out.data_ptr(),
                                        _stream_ptr(stream, q.device))
    if rc != CTX_OK:
        raise error_for(lib, rc)
    return out


def opd_loss(logits, tokens, old_logp, teacher_logp, mask, seq_starts, params: OpdParams | None = None,
             grad: bool = True, out: dict | None = None, stream=None) -> dict:
    """Fused OPD token loss (ctx_opd_loss_run) over a packed batch.

    logits bf16 [N, stride] (the last dimension may be a view wider than vocab:
    pass `vocab` via logits.shape[1] unless `out["vocab"]` is given), tokens int32 [N],
    old_logp / teacher_logp float32 [N], mask uint8 [N], seq_starts int32 [B + 1].
    Returns a dict of device tensors: loss [1], token_logp, token_weight,
    token_loss [N] and, with grad=True, grad_logits bf16 [N, vocab].  Tensors
    given in `out` under those names are written in place (no allocation)."""
    import torch

    lib = load_library()
    params = params or OpdParams()
    n = tokens.shape[0]
    dev = logits.device
    for name, t, dt in (("logits", logits, torch.bfloat16), ("tokens", tokens, torch.int32),
                        ("old_logp", old_logp, torch.float32), ("teacher_logp", teacher_logp, torch.float32),
                        ("mask", mask, torch.uint8), ("seq_starts", seq_starts, torch.int32)):
        if t.dtype != dt:
            raise TypeError(f"{name} must be {dt}, got {t.dtype}")
        if not t.is_cuda or t.device != dev:
            raise ValueError(f"{name} must be on {dev}")
    if logits.dim() != 2 or logits.shape[0] != n or logits.stride(1) != 1:
        raise ValueError("logits must be [N, V] with unit column stride")
    for name, t in (("tokens", tokens), ("old_logp", old_logp), ("teacher_logp", teacher_logp),
                    ("mask", mask), ("seq_starts", seq_starts)):
        if not t.is_contiguous() or t.dim() != 1:
            raise ValueError(f"{name} must be a contiguous vector")
    out = dict(out or {})
    vocab = int(out.pop("vocab", logits.shape[1]))
    if not 0 < vocab <= logits.shape[1]:
        raise ValueError(f"vocab {vocab} must be in 1..{logits.shape[1]} (the columns of logits)")

    def buf(name, shape, dtype):
        t = out.get(name)
        if t is None:
            t = torch.empty(shape, dtype=dtype, device=dev)
        elif t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or t.device != dev:
            raise ValueError(f"out[{name!r}] must be a contiguous {dtype} tensor of shape {tuple(shape)}")
        return t

    res = {"loss": buf("loss", (1,), torch.float32), "token_logp": buf("token_logp", (n,), torch.float32),
           "token_weight": buf("token_weight", (n,), torch.float32),
           "token_loss": buf("token_loss", (n,), torch.float32)}
    g = None
    if grad:
        g = out.get("grad_logits")
        if g is None:  # rows padded to a multiple of 8 elements (16-byte chunks)
            g = torch.empty((n, (vocab + 7) // 8 * 8), dtype=torch.bfloat16, device=dev)
        elif (g.dtype != torch.bfloat16 or g.dim() != 2 or g.shape[0] != n or g.stride(1) != 1
              or g.shape[1] < vocab or g.device != dev):
            raise ValueError(f"out['grad_logits'] must be bf16 [N, >= {vocab}] with unit column stride on {dev}")
        res["grad_logits"] = g if out.get("grad_logits") is not None else g[:, :vocab]
    sp = _stream_ptr(stream, dev)
    rc = lib.ctx_opd_loss_run(logits.data_ptr(), logits.stride(0), vocab, tokens.data_ptr(), old_logp.data_ptr(),
                              teacher_logp.data_ptr(), mask.data_ptr(), seq_starts.data_ptr(),
                              seq_starts.shape[0] - 1, n, ctypes.byref(params), res["token_logp"].data_ptr(),
                              res["token_weight"].data_ptr(), res["token_loss"].data_ptr(), res["loss"].data_ptr(),
                              g.data_ptr() if g is not None else None, g.stride(0) if g is not None else 0, sp)
    if rc != CTX_OK:
        raise error_for(lib, rc)
    return res


def _rollout_outputs(n, turns):
    import numpy as np

    return (np.zeros(1, np.float64), np.full(n * turns * 2, -1.0), np.full(n * turns * 2, -1.0),
            np.zeros(1, np.int32))


def rollout_simulate(policy: int, fast_latency, full_latency, max_concurrency: int) -> dict:
    """Latency model of ctx_rollout_simulate.  fast_latency, full_latency:
    [N, T] seconds (host arrays).  Returns completion, start and end [N, T, 2]
    (kind 0 = fast action, 1 = full response; -1 = not submitted) and peak."""
    import numpy as np

    lib = load_library()
    full = np.ascontiguousarray(full_latency, dtype=np.float64)
    fast = np.ascontiguousarray(fast_latency, dtype=np.float64)
    n, turns = full.shape
    cfg = RolloutConfig(policy, n, turns, max_concurrency)
    comp, st, en, pk = _rollout_outputs(n, turns)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731
    rc = lib.ctx_rollout_simulate(ctypes.byref(cfg), p(fast), p(full), p(comp), p(st), p(en), p(pk))
    if rc != CTX_OK:
        raise error_for(lib, rc)
    return {"completion": float(comp[0]), "start": st.reshape(n, turns, 2), "end": en.reshape(n, turns, 2),
            "peak": int(pk[0])}


def rollout_simulate_engine(policy: int, context_tokens, fast_tokens: int, full_tokens: int, max_concurrency: int,
                            step_base: float, step_per_kv_token: float, prefill_per_token: float) -> dict:
    """Engine model of ctx_rollout_simulate_engine; context_tokens [N, T]."""
    import numpy as np

    lib = load_library()
    ctx = np.ascontiguousarray(context_tokens, dtype=np.int32)
    n, turns = ctx.shape
    cfg = RolloutConfig(policy, n, turns, max_concurrency)
    eng = RolloutEngine(step_base, step_per_kv_token, prefill_per_token, fast_tokens, full_tokens)
    comp, st, en, pk = _rollout_outputs(n, turns)
    steps = np.zeros(1, np.int64)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731
    rc = lib.ctx_rollout_simulate_engine(ctypes.byref(cfg), ctypes.byref(eng), p(ctx), p(comp), p(st), p(en),
                                         p(pk), p(steps))
    if rc != CTX_OK:
        raise error_for(lib, rc)
    return {"completion": float(comp[0]), "start": st.reshape(n, turns, 2), "end": en.reshape(n, turns, 2),
            "peak": int(pk[0]), "steps": int(steps[0])}


def ctx_hbm_read(src, sink, workgroups: int, nontemporal: bool = True, stream=None):
    """Stream every byte of the contiguous CUDA tensor `src` once through the
    compute units (ctx_hbm_read); `sink` is a CUDA tensor of at least
    workgroups * 64 bytes."""
    lib = load_library()
    nbytes = src.numel() * src.element_size()
    if not src.is_contiguous() or sink.numel() * sink.element_size() < workgroups * CTX_HBM_SINK_BYTES_PER_WORKGROUP:
        raise ValueError("src must be contiguous and sink hold workgroups * 64 bytes")
    rc = lib.ctx_hbm_read(src.data_ptr(), nbytes, sink.data_ptr(), int(workgroups),
                          CTX_HBM_NONTEMPORAL if nontemporal else 0, _stream_ptr(stream, src.device))
    if rc != CTX_OK:
        raise error_for(lib, rc)


def ctx_hbm_copy(src, dst, workgroups: int, nontemporal: bool = True, stream=None):
    """dst = src (contiguous CUDA tensors of equal byte size), every byte read and written once."""
    lib = load_library()
    nbytes = src.numel() * src.element_size()
    if not (src.is_contiguous() and dst.is_contiguous()) or dst.numel() * dst.element_size() != nbytes:
        raise ValueError("src and dst must be contiguous and of equal size")
    rc = lib.ctx_hbm_copy(src.data_ptr(), dst.data_ptr(), nbytes, int(workgroups),
                          CTX_HBM_NONTEMPORAL if nontemporal else 0, _stream_ptr(stream, src.device))
    if rc != CTX_OK:
        raise error_for(lib, rc)


def ctx_mfma_bf16(shape: int, workgroups: int, iterations: int, sink, stream=None) -> int:
    """Run the matrix-core rate probe (ctx_mfma_bf16); returns the flops it performs.
    `sink` is a CUDA tensor of at least workgroups * 64 bytes."""
    lib = load_library()
    if sink.numel() * sink.element_size() < workgroups * CTX_HBM_SINK_BYTES_PER_WORKGROUP:
        raise ValueError("sink must hold workgroups * 64 bytes")
    rc = lib.ctx_mfma_bf16(int(shape), int(workgroups), int(iterations), sink.data_ptr(), _stream_ptr(stream, sink.device))
    if rc != CTX_OK:
        raise error_for(lib, rc)
    return workgroups * 4 * iterations * MFMA_FLOPS_PER_WAVE_ROUND[shape]

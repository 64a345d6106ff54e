"""CPU oracles for decode-step GQA attention, causal prefill and the OPD token
loss (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  It wraps `liboracle_attn.so` (plain C, double precision) with
numpy arrays; see oracle_attn.c for the definition it computes.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        p, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_decode_attn.argtypes = [p, p, p, p, p, i32, i32, i32, i32, i64, f64, p, i32]
        lib.oracle_decode_attn.restype = ctypes.c_int
        lib.oracle_decode_attn_pairs.argtypes = [p, p, p, p, p, i32, i32, i32, i32, i64, f64,
                                                 p, i64, p, i32]
        lib.oracle_decode_attn_pairs.restype = ctypes.c_int
        lib.oracle_attn_weights.argtypes = [p, p, p, p, i32, i32, i32, i32, i64, f64, i32, i32, p]
        lib.oracle_attn_weights.restype = ctypes.c_int
        lib.oracle_decode_attn_paged_pairs.argtypes = [p, p, p, p, i32, i32, i64, p, i32, i32, i32, i32,
                                                       f64, p, p, p, i64, p, i32]
        lib.oracle_decode_attn_paged_pairs.restype = ctypes.c_int
        lib.oracle_prefill_attn.argtypes = [p, p, p, p, p, p, p, i32, i32, i32, i32, i64, i64, f64, p, i32]
        lib.oracle_prefill_attn.restype = ctypes.c_int
        lib.oracle_opd_loss.argtypes = [p, i64, i32, p, p, p, p, p, i32, i32, f64, f64, f64, f64,
                                        p, p, p, p, p, i32]
        lib.oracle_opd_loss.restype = ctypes.c_int
        lib.oracle_opd_loss_f64.argtypes = [p, i32, p, p, p, p, p, i32, i32, f64, f64, f64, f64,
                                            p, p, p, p, p, i32]
        lib.oracle_opd_loss_f64.restype = ctypes.c_int
        lib.oracle_opd_grad_rows.argtypes = [p, i64, i32, p, p, p, p, i64, p, i32]
        lib.oracle_opd_grad_rows.restype = ctypes.c_int
        _lib = lib
    return _lib


def _u16(a):
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("expected bf16 bits as uint16")
    return a


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc):
    if rc != 0:
        raise ValueError(f"oracle rejected its inputs (status {rc})")


def decode_attn(q, k, v, seq_offsets, seq_lens, scale, threads: int = 0) -> np.ndarray:
    """out[b, h, :] for every sequence and query head, float64 [B, Hq, D]."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    offs, lens = _i32(seq_offsets), _i32(seq_lens)
    b, hq, d = q.shape
    rows, hkv, dk = k.shape
    if v.shape != k.shape or dk != d or len(offs) != b or len(lens) != b:
        raise ValueError("shape mismatch")
    out = np.zeros((b, hq, d), dtype=np.float64)
    _check(_load().oracle_decode_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(offs), _ptr(lens),
                                      b, hq, hkv, d, rows, float(scale), _ptr(out), threads))
    return out


def decode_attn_pairs(q, k, v, seq_offsets, seq_lens, scale, pairs, threads: int = 0):
    """out for selected (b, h) pairs, float64 [n_pairs, D]."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    offs, lens = _i32(seq_offsets), _i32(seq_lens)
    pairs = np.ascontiguousarray(pairs, dtype=np.int32).reshape(-1, 2)
    b, hq, d = q.shape
    rows, hkv, _ = k.shape
    out = np.zeros((len(pairs), d), dtype=np.float64)
    _check(_load().oracle_decode_attn_pairs(_ptr(q), _ptr(k), _ptr(v), _ptr(offs), _ptr(lens),
                                            b, hq, hkv, d, rows, float(scale), _ptr(pairs),
                                            len(pairs), _ptr(out), threads))
    return out


def attn_weights(q, k, seq_offsets, seq_lens, scale, b: int, h: int) -> np.ndarray:
    """Softmax weights w_t of one (sequence, query head), float64 [L_b]."""
    q, k = _u16(q), _u16(k)
    offs, lens = _i32(seq_offsets), _i32(seq_lens)
    nb, hq, d = q.shape
    rows, hkv, _ = k.shape
    w = np.zeros(max(int(lens[b]), 1), dtype=np.float64)
    _check(_load().oracle_attn_weights(_ptr(q), _ptr(k), _ptr(offs), _ptr(lens), nb, hq, hkv, d,
                                       rows, float(scale), b, h, _ptr(w)))
    return w[: int(lens[b])]


def decode_attn_paged(q, k_pages, v_pages, block_tables, seq_lens, scale, k_new=None, v_new=None,
                      pairs=None, threads: int = 0) -> np.ndarray:
    """Paged decode attention: k_pages, v_pages [num_pages, P, Hkv, D] bf16 bits,
    block_tables [B, max_pages] int32; optional k_new, v_new [B, Hkv, D] replace
    each sequence's newest token.  Returns [B, Hq, D] (or [n_pairs, D])."""
    q, k, v = _u16(q), _u16(k_pages), _u16(v_pages)
    bt, lens = _i32(block_tables), _i32(seq_lens)
    b, hq, d = q.shape
    num_pages, page_tokens, hkv, dk = k.shape
    if v.shape != k.shape or dk != d or bt.ndim != 2 or bt.shape[0] != b or len(lens) != b:
        raise ValueError("shape mismatch")
    if (k_new is None) != (v_new is None):
        raise ValueError("k_new and v_new go together")
    kn = _u16(k_new) if k_new is not None else None
    vn = _u16(v_new) if v_new is not None else None
    if pairs is None:
        pairs = np.stack(np.meshgrid(np.arange(b), np.arange(hq), indexing="ij"), -1).reshape(-1, 2)
        shape = (b, hq, d)
    else:
        shape = None
    pairs = np.ascontiguousarray(pairs, dtype=np.int32).reshape(-1, 2)
    out = np.zeros((len(pairs), d), dtype=np.float64)
    nullp = ctypes.c_void_p(0)
    _check(_load().oracle_decode_attn_paged_pairs(
        _ptr(q), _ptr(k), _ptr(v), _ptr(bt), bt.shape[1], page_tokens, num_pages, _ptr(lens), b, hq, hkv,
        d, float(scale), _ptr(kn) if kn is not None else nullp, _ptr(vn) if vn is not None else nullp,
        _ptr(pairs), len(pairs), _ptr(out), threads))
    return out.reshape(shape) if shape is not None else out


def prefill_attn(q, k, v, seq_offsets, seq_lens, q_starts, q_lens, scale, threads: int = 0) -> np.ndarray:
    """Causal prefill: q [total_q, Hq, D]; sequence b's q_lens[b] queries (rows
    q_starts[b] ..) are its last q_lens[b] tokens; returns float64 [total_q, Hq, D]
    (rows of no sequence stay 0)."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    offs, lens = _i32(seq_offsets), _i32(seq_lens)
    qs, ql = _i32(q_starts), _i32(q_lens)
    total_q, hq, d = q.shape
    rows, hkv, _ = k.shape
    out = np.zeros((total_q, hq, d), dtype=np.float64)
    _check(_load().oracle_prefill_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(offs), _ptr(lens), _ptr(qs), _ptr(ql),
                                       len(lens), hq, hkv, d, rows, total_q, float(scale), _ptr(out), threads))
    return out


# OPD loss constants of the paper (App. OPD Optimization, tab:training-hyperparameters)
OPD_CLIP_LOG = 20.0
OPD_DELTA = 0.2
OPD_KAPPA = 3.0
OPD_EPS = 1e-8


def _opd_common(tokens, old_lp, tea_lp, mask, seq_starts):
    return (_i32(tokens), np.ascontiguousarray(old_lp, dtype=np.float32),
            np.ascontiguousarray(tea_lp, dtype=np.float32), np.ascontiguousarray(mask, dtype=np.uint8),
            _i32(seq_starts))


def opd_loss(logits, tokens, old_lp, tea_lp, mask, seq_starts, clip_log=OPD_CLIP_LOG, delta=OPD_DELTA,
             kappa=OPD_KAPPA, eps=OPD_EPS, threads: int = 0) -> dict:
    """OPD surrogate loss over a packed batch.  logits: bf16 bits [N, stride]
    (the first `vocab` columns used; pass vocab via a [N, V] array) or float64
    [N, V].  Returns float64 loss and per-token lp, weight, token_loss and
    dlp (= dL/dlp_j)."""
    tok, old, tea, m, st = _opd_common(tokens, old_lp, tea_lp, mask, seq_starts)
    n = len(tok)
    lp, w, tl, dlp = (np.zeros(n, np.float64) for _ in range(4))
    loss = np.zeros(1, np.float64)
    if logits.dtype == np.float64:
        z = np.ascontiguousarray(logits)
        rc = _load().oracle_opd_loss_f64(_ptr(z), z.shape[1], _ptr(tok), _ptr(old), _ptr(tea), _ptr(m), _ptr(st),
                                         len(st) - 1, n, clip_log, delta, kappa, eps, _ptr(lp), _ptr(w),
                                         _ptr(tl), _ptr(dlp), _ptr(loss), threads)
    else:
        z = _u16(logits)
        rc = _load().oracle_opd_loss(_ptr(z), z.shape[1], z.shape[1], _ptr(tok), _ptr(old), _ptr(tea), _ptr(m),
                                     _ptr(st), len(st) - 1, n, clip_log, delta, kappa, eps, _ptr(lp), _ptr(w),
                                     _ptr(tl), _ptr(dlp), _ptr(loss), threads)
    _check(rc)
    return {"loss": float(loss[0]), "lp": lp, "weight": w, "token_loss": tl, "dlp": dlp}


def opd_grad_rows(logits, tokens, mask, dlp, rows, threads: int = 0) -> np.ndarray:
    """dL/dlogits for the listed rows, float64 [len(rows), V]; logits bf16 bits [N, V]."""
    z = _u16(logits)
    tok, m = _i32(tokens), np.ascontiguousarray(mask, dtype=np.uint8)
    d = np.ascontiguousarray(dlp, dtype=np.float64)
    r = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((len(r), z.shape[1]), np.float64)
    _check(_load().oracle_opd_grad_rows(_ptr(z), z.shape[1], z.shape[1], _ptr(tok), _ptr(m), _ptr(d), _ptr(r),
                                        len(r), _ptr(out), threads))
    return out

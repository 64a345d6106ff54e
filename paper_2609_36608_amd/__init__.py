"""Decode-step GQA attention over ragged multi-turn KV caches on MI355X (gfx950),
with causal prefill of appended tokens and the fused OPD token loss.

The kernels live in libctx_decode_attn.so (C ABI in include/ctx_decode_attn.h
and include/ctx_opd_loss.h); `binding.DecodeAttention` and `binding.opd_loss`
are the thin ctypes wrappers used by tests and the benchmark.  Importing this
package loads nothing; `workloads` holds the seeded input generator.
"""

__all__ = ["DecodeAttention", "CtxError", "OpdParams", "load_library", "opd_loss"]


def __getattr__(name):
    if name in __all__:
        from . import binding

        return getattr(binding, name)
    raise AttributeError(name)

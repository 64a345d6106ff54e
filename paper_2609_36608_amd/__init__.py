"""Decode-step GQA attention over ragged multi-turn KV caches on MI355X (gfx950).

The kernels live in libctx_decode_attn.so (C ABI in include/ctx_decode_attn.h);
`binding.DecodeAttention` is the thin ctypes wrapper used by tests and the
benchmark.  Importing this package loads nothing; `workloads` holds the seeded
input generator.
"""

__all__ = ["DecodeAttention", "CtxError", "load_library"]


def __getattr__(name):
    if name in __all__:
        from . import binding

        return getattr(binding, name)
    raise AttributeError(name)

"""MI355X (gfx950) hot path of ArborKV-style structure-aware KV eviction for
Tree-of-Thoughts decoding: a HIP library behind the C ABI of include/arbor.h
and its ctypes binding (``paper_2605_22106_amd._lib``)."""
from . import synth  # noqa: F401

__all__ = ["synth"]

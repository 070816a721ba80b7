"""Independent CPU oracle for the Huff-LLM bf16 codec and decode-step GEMV.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package. The library under
``paper_2502_00922_amd`` never imports it and shares no code with it; the two
meet only through the container bytes and the seeded inputs from ``gen``.
"""
from . import codec, gemv

__all__ = ["codec", "gemv"]

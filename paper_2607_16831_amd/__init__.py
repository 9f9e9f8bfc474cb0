"""Gated DeltaNet prefill and decode for AMD MI355X (gfx950).

The compute lives in the HIP library ``libgdn.so`` (sources under ``csrc/``,
C ABI declared in ``include/gdn.h``). ``gdn`` is the thin ctypes binding with
the same entry-point names; ``synth`` draws seeded inputs.
"""
__all__ = ["gdn", "synth"]

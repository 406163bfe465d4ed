"""MI355X (gfx950) SLiM compressed linear layer: 2:4 sparse int4 weights plus a low-rank adapter.

The compute runs in ``libslim.so`` (hand-written HIP kernels behind a C ABI, declared
in ``include/slim.h``). ``paper_2608_24070_amd.slim`` is the thin ctypes binding with
the same entry-point names. Importing this package does not load the library;
the binding loads it on first use and raises if it is missing.
"""
__all__ = ["slim", "synth", "configs"]

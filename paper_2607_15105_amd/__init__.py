"""MI355X-native Hierarchical Global Attention (HGA) hot path.

The compute lives in ``libhga.so`` (hand-written HIP for gfx950, C ABI declared
in ``include/hga.h``). ``paper_2607_15105_amd.hga`` is the thin ctypes binding
that marshals torch tensors into that ABI; ``paper_2607_15105_amd.synth`` draws
the seeded synthetic inputs. Importing the package loads nothing native.
"""

__all__ = ["hga", "synth"]

"""MI355X-native GDN speculative verification (SpecLA, arXiv 2607.16673).

The compute lives in ``libsla.so`` (hand-written HIP for gfx950 behind a
C ABI, declared in ``include/sla.h``); ``binding`` marshals torch tensors
into it.  ``inputs`` is the seeded synthetic workload generator.
"""
__all__ = ["binding", "inputs"]

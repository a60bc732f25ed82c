"""MI355X-native routed attention (Sol-Attn forward hot path).

The compute lives in ``libsolattn.so`` (hand-written HIP for gfx950) behind a
C ABI declared in ``include/sol_attn.h``; ``paper_2607_24027_amd.binding``
marshals torch tensors to it.  ``configs`` and ``synth`` describe and generate
the workloads.  Submodules are imported explicitly
(``from paper_2607_24027_amd import binding``), so the workload helpers work on
machines without the built library.
"""
__all__ = ["binding", "build", "configs", "synth"]

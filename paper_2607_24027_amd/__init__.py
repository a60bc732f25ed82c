"""MI355X-native routed attention (Sol-Attn forward hot path).

The compute lives in ``libsolattn.so`` (hand-written HIP for gfx950) behind a
C ABI declared in ``include/sol_attn.h``; ``paper_2607_24027_amd.binding``
marshals torch tensors to it.  ``configs`` and ``synth`` describe and generate
the workloads.  The binding is imported lazily so that the workload helpers work
on machines without the built library.
"""
__all__ = ["configs", "synth", "binding"]


def __getattr__(name):
    if name == "binding":
        from . import binding
        return binding
    raise AttributeError(name)

"""MI355X-native MoE-layer hot path of Flux (federated MoE fine-tuning).

The compute lives in ``libfluxmoe.so`` (hand-written HIP for gfx950) behind a C
ABI declared in ``include/fluxmoe.h``; :mod:`.api` is the thin ctypes binding.
Importing this package does not load the library; the first API call does, and
it raises if the library is missing.
"""
__all__ = ["api", "workloads"]

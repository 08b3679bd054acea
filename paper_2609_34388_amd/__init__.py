"""MI355X (gfx950) draft-verify hot path of RecGuide.

The compute lives in ``librecguide.so`` (hand-written HIP kernels behind a C
ABI, declared in include/recguide.h); ``binding`` marshals torch tensors into
that ABI.  The library is loaded on first use and a missing or unloadable
library raises -- there is no fallback path.
"""
__all__ = ["binding", "workloads"]

"""MI355X (gfx950) engine for DVI's self-speculative decode step (arXiv 2510.05421).

The decode step (draft -> verify -> commit -> drafter update) runs in hand-written HIP
kernels behind the C ABI in include/dvi.h (libdvi.so); this package is the thin Python
binding over it.  Importing the binding requires the built library: there is no CPU
fallback.
"""
from .schedule import KLRLSchedule  # noqa: F401


def __getattr__(name):
    if name in ("Engine", "EngineConfig", "workspace_bytes"):
        from . import engine
        return getattr(engine, name)
    raise AttributeError(name)

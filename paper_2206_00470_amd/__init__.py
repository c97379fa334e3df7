"""MI355X (gfx950) sparse parameter store: pull rows by key, compute per-task
gradients, push them back merged per key with an AdaGrad update.

The computation lives in the HIP library ``libadapm_hip.so`` (C ABI in
``include/adapm.h``); ``Store`` and ``dedup`` only marshal torch tensors into
it.  Importing this package loads nothing; the library is loaded on first use
and a missing library is an error, never a fallback.
"""

__all__ = ["Store", "dedup", "workloads"]


def __getattr__(name):
    if name in ("Store", "dedup"):
        from . import store
        return getattr(store, name)
    if name == "workloads":
        from . import workloads
        return workloads
    raise AttributeError(name)

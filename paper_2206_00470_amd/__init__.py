"""MI355X (gfx950) sparse parameter store: pull rows by key, compute per-task
gradients, push them back merged per key with an AdaGrad update.

The computation lives in the HIP library ``libadapm_hip.so`` (C ABI in
``include/adapm.h``); ``Store`` and ``dedup`` only marshal torch tensors into
it.  Importing this package loads nothing; the library is loaded on first use
and a missing library is an error, never a fallback.
"""
import importlib

__all__ = ["Store", "StagedStore", "dedup", "action_timing", "workloads"]


def __getattr__(name):
    if name in ("Store", "StagedStore", "dedup", "action_timing"):
        return getattr(importlib.import_module(__name__ + ".store"), name)
    if name == "workloads":
        return importlib.import_module(__name__ + ".workloads")
    raise AttributeError(name)

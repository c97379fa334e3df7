"""ctypes declarations of the C ABI in ``include/adapm.h``.

Loads the in-tree ``libadapm_hip.so``; there is no fallback: if the library
is missing or does not load, every call raises.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libadapm_hip.so")

PS_OK = 0
PS_ERR_INVALID = -1
PS_ERR_KEY_RANGE = -2
PS_ERR_WORKSPACE = -3
PS_ERR_DEVICE = -4
PS_ERR_UNSUPPORTED = -5
PS_ERR_NOT_RESIDENT = -6

PS_OP_PULL, PS_OP_PUSH, PS_OP_DEDUP = 0, 1, 2
PS_OP_STEP_MF, PS_OP_STEP_KGE, PS_OP_STEP_SGNS, PS_OP_STEP_CTR = 3, 4, 5, 6
PS_OP_STEP_MF_ASYNC = 7

PS_NOALLOC_SCRATCH_BYTES = 64 << 20

PS_KERNEL_SEGREDUCE, PS_KERNEL_TASKGRAD, PS_KERNEL_SCATTER, PS_KERNEL_PULL, PS_KERNEL_MF_ROWMERGE = 0, 1, 2, 3, 4
PS_KERNEL_STAGE = 5
PS_KERNEL_MLP = 6
PS_KERNEL_ASYNC = 7
PS_TIMING_ALL = -1
PS_PROBE_GRID = 2048

STAGE_STATS = ["clock", "rounds", "forced", "staged", "evicted", "resident", "pending", "stalled", "plan_us"]

_p, _i64, _i32, _f32, _sz = C.c_void_p, C.c_int64, C.c_int32, C.c_float, C.c_size_t

# name -> (restype, argtypes); the same names and order as include/adapm.h
SIGNATURES = {
    "ps_create": (_i32, [C.POINTER(_p), _i64, _i32, _p, _p, _f32, _f32, _p]),
    "ps_create_strided": (_i32, [C.POINTER(_p), _i64, _i32, _i64, _p, _p, _f32, _f32, _p]),
    "ps_create_rowwise": (_i32, [C.POINTER(_p), _i64, _i32, _i64, _p, _p, _i64, _f32, _f32, _p]),
    "ps_create_bf16": (_i32, [C.POINTER(_p), _i64, _i32, _p, _i64, _p, _i64, _f32, _f32, _p]),
    "ps_destroy": (_i32, [_p]),
    "ps_workspace_bytes": (_sz, [_i64, _i32, _i32, _i64, _i64]),
    "ps_pull": (_i32, [_p, _p, _i64, _p, _p]),
    "ps_push": (_i32, [_p, _p, _i64, _p, _p, _sz, _p]),
    "ps_push_prepare": (_i32, [_p, _p, _i64, _p, _sz, _p]),
    "ps_push_apply": (_i32, [_p, _i64, _p, _p, _sz, _p]),
    "ps_push_noalloc": (_i32, [_p, _p, _i64, _p, _p]),
    "ps_dedup": (_i32, [_i64, _p, _i64, _p, _p, _p, _p, _p, _p, _sz, _p]),
    "ps_step_mf": (_i32, [_p, _p, _p, _p, _i64, _i64, _f32, _p, _p, _sz, _p]),
    "ps_step_mf_prepare": (_i32, [_p, _p, _p, _p, _i64, _i64, _p, _sz, _p]),
    "ps_step_mf_apply": (_i32, [_p, _i64, _f32, _p, _p, _sz, _p, _p]),
    "ps_push_async": (_i32, [_p, _p, _i64, _p, _p]),
    "ps_step_mf_async": (_i32, [_p, _p, _p, _p, _i64, _i64, _f32, _p, _p, _sz, _p]),
    "ps_step_kge": (_i32, [_p, _p, _p, _p, _p, _i64, _i32, _i32, _i64, _p, _p, _sz, _p]),
    "ps_step_sgns": (_i32, [_p, _p, _p, _p, _i64, _i32, _i32, _i64, _p, _p, _sz, _p]),
    "ps_step_ctr": (_i32, [_p, _p, _p, _i64, _i32, _p, _p, _sz, _p]),
    "ps_step_kge_prepare": (_i32, [_p, _p, _p, _p, _p, _i64, _i32, _i64, _p, _sz, _p]),
    "ps_step_kge_apply": (_i32, [_p, _p, _p, _p, _p, _i64, _i32, _i32, _i64, _p, _p, _sz, _p]),
    "ps_step_sgns_prepare": (_i32, [_p, _p, _p, _p, _i64, _i32, _i32, _i64, _p, _sz, _p]),
    "ps_step_sgns_apply": (_i32, [_p, _p, _p, _p, _i64, _i32, _i32, _i64, _p, _p, _sz, _p]),
    "ps_step_ctr_prepare": (_i32, [_p, _p, _i64, _i32, _p, _sz, _p]),
    "ps_step_ctr_apply": (_i32, [_p, _p, _p, _i64, _i32, _p, _p, _sz, _p]),
    "ps_get_error": (_i32, [_p, _p]),
    "ps_status_string": (C.c_char_p, [_i32]),
    "ps_last_error_message": (C.c_char_p, []),
    "ps_probe_gather": (_i32, [_p, _p, _i64, _p, _p]),
    "ps_set_timing": (_i32, [_p, _i32]),
    "ps_read_timing": (_i32, [_p, _i32, C.POINTER(C.c_double), C.POINTER(_i64)]),
    "ps_ctr_wd_workspace_bytes": (_sz, [_i64, _i32, _i64, _i32, _i32, _i32, _p]),
    "ps_step_ctr_wd": (_i32, [_p, _p, _p, _i64, _i32, _i32, _i32, _p, _p, _p, _p, _p, _sz, _p]),
    "ps_create_staged": (_i32, [C.POINTER(_p), _i64, _i32, _p, _p, _i64, _p, _p, _i64, _p, _i32, _p, _p, _f32, _f32,
                                _p]),
    "ps_set_action_timing": (_i32, [_p, C.c_double, C.c_double, C.c_double]),
    "ps_intent": (_i32, [_p, _p, _i64, _i64, _i64]),
    "ps_advance_clock": (_i32, [_p, _p]),
    "ps_stage_round": (_i32, [_p, _i32]),
    "ps_stage_auto": (_i32, [_p, _i32]),
    "ps_stage_flush": (_i32, [_p, _p]),
    "ps_stage_stats": (_i32, [_p, _p, _i32, C.POINTER(C.c_double)]),
    "ps_stage_resident": (_i32, [_p, _p, _i64, C.POINTER(_i64)]),
    "ps_action_timing": (_i32, [C.c_double, _i64, _i64, C.c_double, C.c_double, C.POINTER(C.c_double),
                                C.POINTER(_i64)]),
}


class PSError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or python paper_2206_00470_amd/build.py")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(status: int):
    if status != PS_OK:
        L = lib()
        msg = L.ps_last_error_message().decode() or L.ps_status_string(status).decode()
        raise PSError(status, msg)

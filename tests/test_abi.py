"""The C ABI without a GPU: the library loads, exports every declared entry
point, and rejects bad arguments on the host before touching the device."""
import ctypes as C
import os
import re

import pytest

from paper_2206_00470_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adapm.h")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ps_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared()
    for n in ("ps_create", "ps_create_rowwise", "ps_destroy", "ps_pull", "ps_push", "ps_dedup", "ps_step_mf", "ps_step_kge",
              "ps_step_sgns", "ps_step_ctr", "ps_get_error", "ps_workspace_bytes"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = _lib.lib()
    for n in declared():
        assert hasattr(L, n), n


def test_binding_covers_every_declared_symbol():
    assert sorted(_lib.SIGNATURES) == declared()


def test_status_strings():
    L = _lib.lib()
    for st in (0, -1, -2, -3, -4, -5):
        assert L.ps_status_string(st)
    assert L.ps_status_string(-99) == b"unknown status"


def test_create_rejects_bad_arguments_on_host():
    L = _lib.lib()
    h = C.c_void_p(1)
    fake = C.c_void_p(0x1000)
    other = C.c_void_p(0x2000)
    assert L.ps_create(None, 10, 4, fake, other, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create(C.byref(h), 0, 4, fake, other, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert h.value is None
    assert L.ps_create(C.byref(h), 10, 0, fake, other, 0.1, 0.0, None) == _lib.PS_ERR_UNSUPPORTED
    assert L.ps_create(C.byref(h), 10, 513, fake, other, 0.1, 0.0, None) == _lib.PS_ERR_UNSUPPORTED
    # rows wider than 512 floats: a multiple of 4 up to 16384 passes the width
    # check (these fake tables then fail the overlap check), others do not
    for bad in (514, 1001, 16388, 1 << 20):
        assert L.ps_create(C.byref(h), 10, bad, fake, other, 0.1, 0.0, None) == _lib.PS_ERR_UNSUPPORTED
    for wide in (516, 600, 1024, 4096, 16384):
        assert L.ps_create(C.byref(h), 10, wide, fake, other, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
        assert b"overlap" in L.ps_last_error_message()
        big = C.c_void_p(0x1000 + 16 * 10 * wide * 4)
        assert L.ps_create_rowwise(C.byref(h), 10, wide, wide, fake, big, 1, 0.1, 0.0, None) == \
            _lib.PS_ERR_UNSUPPORTED
    assert L.ps_create(C.byref(h), 10, 512, fake, None, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create(C.byref(h), 10, 4, None, other, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create(C.byref(h), 10, 4, fake, fake, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create(C.byref(h), 10, 4, C.c_void_p(0x1004), other, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create(C.byref(h), 10, 4, fake, other, 0.0, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create(C.byref(h), 10, 4, fake, other, 0.1, -1.0, None) == _lib.PS_ERR_INVALID
    assert b"lr" in L.ps_last_error_message()


def test_create_strided_rejects_overlapping_or_misaligned_rows():
    L = _lib.lib()
    h = C.c_void_p(1)
    base = 0x100000
    K, d = 1000, 100
    P = lambda off_floats: C.c_void_p(base + 4 * off_floats)
    # interleaved [K][2d]: accum = values + d, stride 2d is fine (host checks only, so expect no
    # argument error before the device allocation; we stop at the overlap checks here)
    assert L.ps_create_strided(C.byref(h), K, d, d - 1, P(0), P(d), 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create_strided(C.byref(h), K, d, 2 * d, P(0), P(d // 2), 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create_strided(C.byref(h), K, d, d, P(0), P(d), 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create_strided(C.byref(h), K, d, 2 * d + 2, P(0), P(d), 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create_strided(C.byref(h), K, d, 2 * d, P(1), P(d + 1), 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert h.value is None


def test_create_rowwise_rejects_overlapping_or_bad_accumulators():
    L = _lib.lib()
    h = C.c_void_p(1)
    base = 0x100000
    K, d = 1000, 100
    P = lambda off_floats: C.c_void_p(base + 4 * off_floats)
    cr = lambda ld, acc, ast, lr=0.1: L.ps_create_rowwise(C.byref(h), K, d, ld, P(0), acc, ast, lr, 0.0, None)
    assert cr(d + 4, None, d + 4) == _lib.PS_ERR_INVALID                  # no accumulator
    assert cr(d + 4, P(d), 0) == _lib.PS_ERR_INVALID                      # stride < 1
    assert cr(d + 4, P(d - 1), d + 4) == _lib.PS_ERR_INVALID              # inside the row
    assert cr(d, P(d), d) == _lib.PS_ERR_INVALID                          # no padding: next row's first value
    assert cr(d + 4, P(d), d + 3) == _lib.PS_ERR_INVALID                  # drifts into later rows
    assert cr(d + 4, P(5 * (d + 4)), 1) == _lib.PS_ERR_INVALID            # a vector inside W's extent
    assert cr(d + 4, P(d), d + 4, lr=0.0) == _lib.PS_ERR_INVALID
    assert cr(d + 2, P(d), d + 2) == _lib.PS_ERR_INVALID                  # stride not a multiple of 4
    assert L.ps_create_rowwise(None, K, d, d, P(0), P(K * d), 1, 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert L.ps_create_rowwise(C.byref(h), K, 513, 520, P(0), P(K * 520), 1, 0.1, 0.0,
                               None) == _lib.PS_ERR_UNSUPPORTED
    assert h.value is None


def test_create_bf16_rejects_overlap_and_misalignment():
    L = _lib.lib()
    h = C.c_void_p(1)
    base = 0x100000
    K, d = 1000, 100
    V = lambda off_bytes: C.c_void_p(base + off_bytes)
    cr = lambda va, vs, aa, as_: L.ps_create_bf16(C.byref(h), K, d, V(va), vs, V(aa), as_, 0.1, 0.0, None)
    assert cr(0, 100, 100, 100) == _lib.PS_ERR_INVALID                 # accumulators inside the value table
    assert cr(0, 304, 200, 152) == _lib.PS_ERR_INVALID                 # 8-byte aligned only
    assert cr(0, 304, 192, 152) == _lib.PS_ERR_INVALID                 # interleaved but overlapping the values
    assert cr(0, 300, 208, 152) == _lib.PS_ERR_INVALID                 # byte strides differ
    assert cr(4, 304, 208 + 4, 152) == _lib.PS_ERR_INVALID             # values not 8-byte aligned
    assert cr(0, 99, 10 ** 6, 100) == _lib.PS_ERR_INVALID              # stride below dim
    assert L.ps_create_bf16(C.byref(h), K, 513, V(0), 600, V(10 ** 7), 600, 0.1, 0.0, None) == \
        _lib.PS_ERR_UNSUPPORTED
    assert h.value is None


def test_calls_on_null_store_are_rejected():
    L = _lib.lib()
    p = C.c_void_p(0x1000)
    assert L.ps_pull(None, p, 1, p, None) == _lib.PS_ERR_INVALID
    assert L.ps_push(None, p, 1, p, p, 1 << 20, None) == _lib.PS_ERR_INVALID
    assert L.ps_step_mf(None, p, p, p, 1, 0, 0.01, None, p, 1 << 20, None) == _lib.PS_ERR_INVALID
    assert L.ps_get_error(None, None) == _lib.PS_ERR_INVALID
    assert L.ps_destroy(None) == _lib.PS_OK
    ms, n = C.c_double(), C.c_int64()
    assert L.ps_read_timing(None, 0, C.byref(ms), C.byref(n)) == _lib.PS_ERR_INVALID


def test_dedup_rejects_bad_arguments_on_host():
    L = _lib.lib()
    p = C.c_void_p(0x1000)
    assert L.ps_dedup(0, p, 4, p, p, p, p, None, p, 1 << 20, None) == _lib.PS_ERR_INVALID
    assert L.ps_dedup(10, p, -1, p, p, p, p, None, p, 1 << 20, None) == _lib.PS_ERR_INVALID
    assert L.ps_dedup(10, p, 1 << 31, p, p, p, p, None, p, 1 << 40, None) == _lib.PS_ERR_UNSUPPORTED
    assert L.ps_dedup(10, p, 4, p, p, None, p, None, p, 1 << 20, None) == _lib.PS_ERR_INVALID
    need = L.ps_workspace_bytes(10, 1, _lib.PS_OP_DEDUP, 4, 1)
    assert L.ps_dedup(10, p, 4, p, p, p, p, None, p, need - 1, None) == _lib.PS_ERR_WORKSPACE
    assert L.ps_dedup(10, p, 4, p, p, p, p, None, None, need, None) == _lib.PS_ERR_INVALID


@pytest.mark.parametrize("op,per", [(_lib.PS_OP_PUSH, 1), (_lib.PS_OP_DEDUP, 1), (_lib.PS_OP_STEP_MF, 2),
                                    (_lib.PS_OP_STEP_KGE, 103), (_lib.PS_OP_STEP_SGNS, 261),
                                    (_lib.PS_OP_STEP_CTR, 26)])
def test_workspace_sizes(op, per):
    L = _lib.lib()
    small = L.ps_workspace_bytes(1000, 100, op, 10, per)
    big = L.ps_workspace_bytes(1000, 100, op, 10_000, per)
    assert 0 < small < big
    assert L.ps_workspace_bytes(1000, 100, op, (1 << 31) // per, per) == 0   # beyond 32-bit occurrence index
    assert L.ps_workspace_bytes(0, 100, op, 10, per) == 0
    assert L.ps_workspace_bytes(1000, 100, op, 10, 0) == 0


def test_pull_needs_no_workspace():
    assert _lib.lib().ps_workspace_bytes(1000, 100, _lib.PS_OP_PULL, 10, 1) == 0


def test_binding_constants_match_the_header():
    """The binding's operation codes, kernel ids and staging statistics
    follow the header's numbering."""
    import re
    text = open(HEADER).read()
    defs = {m.group(1): int(m.group(2)) for m in re.finditer(r"#define (PS_[A-Z0-9_]+)\s+\(?(-?\d+)\)?", text)}
    for name in ("PS_OP_PUSH", "PS_OP_STEP_MF", "PS_OP_STEP_CTR", "PS_OP_STEP_MF_ASYNC", "PS_KERNEL_SEGREDUCE",
                 "PS_KERNEL_MF_ROWMERGE", "PS_KERNEL_STAGE", "PS_KERNEL_MLP", "PS_KERNEL_ASYNC",
                 "PS_ERR_KEY_RANGE", "PS_ERR_UNSUPPORTED", "PS_ERR_NOT_RESIDENT"):
        assert getattr(_lib, name) == defs[name], name
    stats = [n for n in defs if n.startswith("PS_STAGE_") and n != "PS_STAGE_NUM_STATS"]
    assert len(_lib.STAGE_STATS) == defs["PS_STAGE_NUM_STATS"] == len(stats)
    for n in stats:
        assert _lib.STAGE_STATS[defs[n]] == n[len("PS_STAGE_"):].lower(), n

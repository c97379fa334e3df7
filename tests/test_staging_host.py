"""Host logic of the staged store, without a GPU: the library's Algorithm 1
(ps_action_timing) against the plain reference in oracle/staging.py, and the
argument checks of ps_create_staged that run before any device call."""
import ctypes as C

import numpy as np
import pytest

from oracle.staging import action_timing as ref_timing
from paper_2206_00470_amd import _lib
from paper_2206_00470_amd.store import action_timing


def test_action_timing_matches_the_reference_on_random_traces():
    rng = np.random.default_rng(50)
    for trial in range(400):
        alpha = float(rng.choice([0.1, 0.3, 1.0, rng.uniform(0.01, 1.0)]))
        p = float(rng.choice([0.5, 0.9, 0.9999, rng.uniform(0.5, 0.99999)]))
        lam = float(rng.choice([0.0, 10.0, rng.uniform(0, 50), rng.uniform(0, 3000)]))
        c = int(rng.integers(0, 10_000))
        for _ in range(6):
            step = int(rng.choice([0, 0, 1, 2, int(rng.integers(0, 400))]))
            got = action_timing(lam, c, c + step, alpha, p)
            want = ref_timing(lam, c, c + step, alpha, p)
            assert got[1] == want[1], (lam, c, step, alpha, p)
            assert got[0] == pytest.approx(want[0], rel=1e-15, abs=0)
            lam, c = got[0], c + step


def test_action_timing_paper_defaults():
    assert action_timing(10.0, 0, 0) == (10.0, 39)
    lam, h = action_timing(10.0, 50, 150)
    assert lam == pytest.approx(19.0) and h == 150 + ref_timing(19.0, 0, 100)[1] - 100


def test_action_timing_rejects_bad_parameters():
    L = _lib.lib()
    lam, h = C.c_double(), C.c_int64()
    assert L.ps_action_timing(10.0, 0, 1, 0.0, 0.9, C.byref(lam), C.byref(h)) == _lib.PS_ERR_INVALID
    assert L.ps_action_timing(10.0, 0, 1, 0.1, 1.0, C.byref(lam), C.byref(h)) == _lib.PS_ERR_INVALID
    assert L.ps_action_timing(10.0, 0, 1, 0.1, 0.9, None, C.byref(h)) == _lib.PS_ERR_INVALID


def test_create_staged_rejects_bad_ranges_before_any_device_call():
    L = _lib.lib()
    h = C.c_void_p(1)
    P = lambda off: C.c_void_p(0x100000 + 4 * off)
    K, d = 1000, 16

    def cr(begin, slots, hs=2 * d, hacc=d):
        rb = (C.c_int64 * len(begin))(*begin)
        rs = (C.c_int64 * len(slots))(*slots)
        return L.ps_create_staged(C.byref(h), K, d, P(0), P(hacc), hs, P(10 ** 6), P(10 ** 6 + d), 2 * d,
                                  P(5 * 10 ** 6), len(begin), rb, rs, 0.1, 0.0, None)

    assert cr([1], [10]) == _lib.PS_ERR_INVALID              # first range must begin at 0
    assert cr([0, 500, 400], [1, 1, 1]) == _lib.PS_ERR_INVALID   # not ascending
    assert cr([0, 1000], [1, 1]) == _lib.PS_ERR_INVALID       # begins past num_keys
    assert cr([0, 500], [0, 5]) == _lib.PS_ERR_INVALID        # empty capacity
    assert cr([0, 500], [501, 5]) == _lib.PS_ERR_INVALID      # more slots than keys
    assert cr([0], [10], hs=d) == _lib.PS_ERR_INVALID         # home rows overlap
    assert cr([0], [10], hacc=d // 2) == _lib.PS_ERR_INVALID
    assert L.ps_create_staged(None, K, d, P(0), P(d), 2 * d, P(0), P(0), 2 * d, P(0), 1,
                              (C.c_int64 * 1)(0), (C.c_int64 * 1)(1), 0.1, 0.0, None) == _lib.PS_ERR_INVALID
    assert h.value is None


def test_staging_calls_on_plain_or_null_stores_are_rejected():
    L = _lib.lib()
    assert L.ps_intent(None, None, 0, 0, 1) == _lib.PS_ERR_INVALID
    assert L.ps_advance_clock(None, None) == _lib.PS_ERR_INVALID
    assert L.ps_stage_round(None, 0) == _lib.PS_ERR_INVALID
    assert L.ps_stage_flush(None, None) == _lib.PS_ERR_INVALID
    assert L.ps_stage_auto(None, 1) == _lib.PS_ERR_INVALID
    assert L.ps_status_string(_lib.PS_ERR_NOT_RESIDENT) == b"key not resident in the staged store"

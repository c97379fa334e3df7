"""Comparison helpers shared by the GPU parity tests."""
import sys

import numpy as np

RTOL, ATOL = 1e-5, 1e-6   # per fp32 element of W and G after a push or step


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def assert_close_tables(gpu: np.ndarray, ref: np.ndarray, what: str, rows_chunk: int = 1 << 20):
    """|gpu - ref| <= ATOL + RTOL |ref| for every element, checked in row chunks."""
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    worst = 0.0
    nbad = 0
    for lo in range(0, gpu.shape[0], rows_chunk):
        g = gpu[lo:lo + rows_chunk].astype(np.float64)
        r = ref[lo:lo + rows_chunk].astype(np.float64)
        err = np.abs(g - r) - (ATOL + RTOL * np.abs(r))
        nbad += int((err > 0).sum())
        worst = max(worst, float(err.max(initial=-1.0)))
    assert nbad == 0, f"{what}: {nbad} elements outside |d| <= {ATOL} + {RTOL}|ref| (worst excess {worst:.3g})"


def assert_bitwise(gpu: np.ndarray, ref: np.ndarray, what: str):
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    a = np.ascontiguousarray(gpu).view(np.uint8)
    b = np.ascontiguousarray(ref).view(np.uint8)
    if not np.array_equal(a, b):
        diff = np.flatnonzero(np.ascontiguousarray(gpu).ravel() != np.ascontiguousarray(ref).ravel())
        raise AssertionError(f"{what}: {diff.size} elements differ, first at flat index {diff[:5]}")


def mismatch_fraction(gpu: np.ndarray, ref: np.ndarray) -> float:
    return float(np.mean(np.ascontiguousarray(gpu).view(np.uint32) != np.ascontiguousarray(ref).view(np.uint32)))

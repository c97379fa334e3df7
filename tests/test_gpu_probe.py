"""The gather probe (instrumentation: the row reads of a gather-bound
kernel without its arithmetic) reads exactly the rows it is given: the
total of its fp64 sums equals the fp64 sum of those rows, keys outside the
table skipped, at row widths of every lane layout and ragged lengths."""
import numpy as np
import pytest
import torch

from paper_2206_00470_amd import Store
from paper_2206_00470_amd.store import interleaved_tables
from paper_2206_00470_amd.workloads import normal_table
from tests.helpers import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("K,d,n", [(1, 4, 1), (5000, 16, 4097), (5000, 100, 100_003), (3000, 3, 777),
                                   (3000, 300, 65_537), (2000, 512, 3001), (4000, 100, 0)])
def test_probe_reads_the_given_rows(K, d, n):
    say(f"probe K={K} d={d} n={n}")
    W = normal_table(K, d, 0.1, 11, 1)
    rng = np.random.default_rng(d + n)
    keys = rng.integers(0, K, n).astype(np.int32)
    if n > 10:
        keys[::7] = -1          # skipped
        keys[3::11] = K         # skipped
    Wt, Gt = interleaved_tables(torch.from_numpy(W).cuda()) if d % 4 == 0 else \
        (torch.from_numpy(W).cuda(), torch.zeros((K, d), dtype=torch.float32, device="cuda"))
    s = Store(Wt, Gt)
    sink = s.probe_gather(torch.from_numpy(keys).cuda())
    got = float(sink.sum().item())
    valid = keys[(keys >= 0) & (keys < K)]
    want = float(W[valid].astype(np.float64).sum())
    assert got == pytest.approx(want, rel=1e-10, abs=1e-9)

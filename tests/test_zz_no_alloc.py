"""The allocation-free push (ps_push_noalloc, workspace in the library's
static device scratch) against ps_push with a caller's workspace: the same
tables bit for bit after two pushes in a row, the second smaller (so stale
scratch contents from the first must not leak into it), both within the
oracle's tolerance; pushes too large for the scratch are refused on the
host with the state untouched."""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store, _lib
from paper_2206_00470_amd._lib import PSError
from paper_2206_00470_amd.workloads import normal_table, random_push
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# (num_keys, dim, first push size, Zipf exponent of its keys, second push size)
CASES = [(200_000, 100, 700_000, 1.1, 5_003), (50_000, 16, 1_400_000, 1.05, 777), (3_000, 512, 200_000, None, 64)]


@pytest.mark.parametrize("K,d,n1,zipf,n2", CASES)
def test_push_noalloc_equals_push_twice(K, d, n1, zipf, n2):
    W0 = normal_table(K, d, 0.1, 90, d)
    G0 = np.zeros_like(W0)
    WA, GA = dev(W0), dev(G0)
    WB, GB = dev(W0), dev(G0)
    A = Store(WA, GA, LR, EPS)
    B = Store(WB, GB, LR, EPS)
    Wr, Gr = W0.copy(), G0.copy()
    for i, (n, z) in enumerate([(n1, zipf), (n2, None)]):
        keys, grads = random_push(K, n, d, 91 + i, zipf_s=z)
        if i == 1:
            keys[[0, n // 2]] = [-5, K]      # invalid keys are skipped and flagged by both
        say(f"push {i}: K={K} d={d} n={n}")
        A.push(dev(keys), dev(grads))
        B.push_noalloc(dev(keys), dev(grads))
        assert A.error() == B.error() == (0 if i == 0 else _lib.PS_ERR_KEY_RANGE)
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after push {i}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after push {i}")
        oracle.push(Wr, Gr, keys, grads, LR, EPS)
        assert_close_tables(WB.cpu().numpy(), Wr, f"W after push {i} against the oracle")
        assert_close_tables(GB.cpu().numpy(), Gr, f"G after push {i} against the oracle")
    A.close()
    B.close()


def test_push_noalloc_refuses_pushes_beyond_the_scratch():
    K, d = 1000, 100
    W0 = normal_table(K, d, 0.1, 92, d)
    Wt, Gt = dev(W0), torch.zeros((K, d), dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, LR, EPS)
    n = 1
    while s.workspace_bytes(_lib.PS_OP_PUSH, n) <= _lib.PS_NOALLOC_SCRATCH_BYTES:
        n *= 2
    keys = torch.zeros(n, dtype=torch.int64, device="cuda")
    grads = torch.ones((n, d), dtype=torch.float32, device="cuda")
    with pytest.raises(PSError) as e:
        s.push_noalloc(keys, grads)
    assert e.value.status == _lib.PS_ERR_UNSUPPORTED
    assert "static scratch" in str(e.value)
    assert s.error() == 0
    assert_bitwise(Wt.cpu().numpy(), W0, "W untouched")
    assert not Gt.cpu().numpy().any()
    s.push_noalloc(keys[:0], grads[:0])     # empty: a no-op
    s.close()

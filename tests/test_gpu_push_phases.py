"""The push in two phases (ps_push_prepare: key work into a workspace;
ps_push_apply: the merge) against ps_push: bit for bit on one stream, and
bit for bit when the next push's key work runs on a second stream beside
this push's merge (two workspaces, ordered by events)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store, _lib
from paper_2206_00470_amd._lib import PSError
from paper_2206_00470_amd.store import interleaved_tables
from paper_2206_00470_amd.workloads import normal_table, random_push
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


CASES = [(1, 4, 1, None), (5000, 16, 4097, 1.1), (23_000, 100, 300_001, 1.1), (3000, 3, 2000, None),
         (40, 64, 70_001, 1.5), (700, 512, 999, None)]


@pytest.mark.parametrize("K,d,n,zipf", CASES)
def test_prepare_then_apply_is_push(K, d, n, zipf):
    W0 = normal_table(K, d, 0.1, 60, d)
    G0 = np.random.default_rng(61).uniform(0, 1, (K, d)).astype(np.float32)
    keys, grads = random_push(K, n, d, 62, zipf_s=zipf)
    keys[n // 3] = K + 5                     # an invalid key is skipped and flagged in both
    WA, GA, WB, GB = dev(W0), dev(G0), dev(W0), dev(G0)
    A, B = Store(WA, GA, LR, EPS), Store(WB, GB, LR, EPS)
    A.push(dev(keys), dev(grads))
    ws = B.push_workspace(n)
    B.push_prepare(dev(keys), ws)
    B.push_apply(n, dev(grads), ws)
    assert A.error() == B.error() == _lib.PS_ERR_KEY_RANGE
    assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), "W")
    assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), "G")
    Wr, Gr = W0.copy(), G0.copy()
    oracle.push(Wr, Gr, keys, grads, LR, EPS)
    assert_close_tables(WB.cpu().numpy(), Wr, "W against the oracle")
    assert_close_tables(GB.cpu().numpy(), Gr, "G against the oracle")


@pytest.mark.parametrize("K,d,n,zipf", [(50_000, 100, 200_003, 1.1), (2000, 16, 30_000, None)])
def test_overlapped_pushes_equal_sequential_pushes(K, d, n, zipf):
    """Six pushes; on the twin store the key work of push i+1 runs on a side
    stream while push i merges on the main stream."""
    W0 = normal_table(K, d, 0.1, 63, d)
    WA, GA = interleaved_tables(dev(W0))
    WB, GB = interleaved_tables(dev(W0))
    A, B = Store(WA, GA, LR, EPS), Store(WB, GB, LR, EPS)
    pushes = [tuple(dev(x) for x in random_push(K, n, d, 64 + i, zipf_s=zipf)) for i in range(6)]
    for k, g in pushes:
        A.push(k, g)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    ws = [B.push_workspace(n), B.push_workspace(n)]
    prepared = [torch.cuda.Event(), torch.cuda.Event()]
    applied = [torch.cuda.Event(), torch.cuda.Event()]
    side.wait_stream(main)
    B.push_prepare(pushes[0][0], ws[0], stream=side)
    prepared[0].record(side)
    for i, (_, g) in enumerate(pushes):
        main.wait_event(prepared[i % 2])
        B.push_apply(n, g, ws[i % 2], stream=main)
        applied[i % 2].record(main)
        if i + 1 < len(pushes):
            if i >= 1:
                side.wait_event(applied[(i + 1) % 2])   # the apply that last used that workspace
            B.push_prepare(pushes[i + 1][0], ws[(i + 1) % 2], stream=side)
            prepared[(i + 1) % 2].record(side)
    torch.cuda.synchronize()
    assert A.error() == 0 and B.error() == 0
    say(f"six pushes of {n} keys, overlapped")
    assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), "W")
    assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), "G")


def test_two_phase_push_argument_checks():
    K, d = 100, 8
    W, G = torch.zeros((K, d), device="cuda"), torch.zeros((K, d), device="cuda")
    s = Store(W, G, LR, EPS)
    keys = torch.arange(10, dtype=torch.int64, device="cuda")
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(PSError) as e:
        s.push_prepare(keys, small)
    assert e.value.status == _lib.PS_ERR_WORKSPACE
    ws = s.push_workspace(10)
    with pytest.raises(ValueError):
        s.push_apply(10, torch.zeros(9 * d, device="cuda"), ws)
    s.push_prepare(keys[:0], ws)               # empty: no-ops
    s.push_apply(0, torch.zeros(0, device="cuda"), ws)
    assert s.error() == 0
    assert not W.cpu().numpy().any()

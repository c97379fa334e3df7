"""Rows wider than 512 floats (the paper's widest models keep 1,000 floats
per parameter row, Table 3): pull and push serve them one column slice of
512 floats at a time.  Against the oracle, which handles the whole row:
pulls bit for bit, pushes within 1e-6 + 1e-5 |ref| (untouched rows bit for
bit), with hot keys whose segments are cut into chunks and folded; the
two-phase and allocation-free pushes bit for bit as ps_push; the first-touch
closed form exactly; the task steps refuse such rows."""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store, _lib
from paper_2206_00470_amd.store import interleaved_tables
from paper_2206_00470_amd.workloads import normal_table, random_push
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10
WIDE = [516, 600, 1000, 1024, 2000]


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def make(K, d, seed, interleaved, g_fill=True):
    W = normal_table(K, d, 0.1, seed, 1)
    G = np.random.default_rng(seed).uniform(0, 1, (K, d)).astype(np.float32) if g_fill else np.zeros((K, d), np.float32)
    if interleaved:
        Wt, Gt = interleaved_tables(dev(W), dev(G))
    else:
        Wt, Gt = dev(W), dev(G)
    return W, G, Wt, Gt, Store(Wt, Gt, LR, EPS)


@pytest.mark.parametrize("d", WIDE)
@pytest.mark.parametrize("interleaved", [False, True])
def test_wide_pull_is_bit_exact(d, interleaved):
    say(f"wide pull d={d} interleaved={interleaved}")
    K, n = 3000, 7001
    W, G, Wt, Gt, s = make(K, d, 3, interleaved)
    keys = np.random.default_rng(d).integers(0, K, n).astype(np.int64)
    keys[5] = K                     # out of range: a zero row and the error flag
    out = s.pull(dev(keys)).cpu().numpy()
    assert s.error() == _lib.PS_ERR_KEY_RANGE
    ref, bad = oracle.pull(W, keys)
    assert bad == 1
    assert_bitwise(out, ref, "pulled rows")


@pytest.mark.parametrize("d", WIDE)
@pytest.mark.parametrize("interleaved", [False, True])
def test_wide_push_matches_the_oracle(d, interleaved):
    say(f"wide push d={d} interleaved={interleaved}")
    K, n = 4000, 40_000
    W, G, Wt, Gt, s = make(K, d, 7, interleaved)
    keys, grads = random_push(K, n, d, 8, zipf_s=1.1)   # hot keys: chunks cut and folded
    keys[::997] = 0                                       # one key with > 2,048 occurrences
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Gr = W.copy(), G.copy()
    oracle.push(Wr, Gr, keys, grads, LR, EPS)
    Wg, Gg = Wt.cpu().numpy(), Gt.cpu().numpy()
    assert_close_tables(Wg, Wr, "W")
    assert_close_tables(Gg, Gr, "G")
    untouched = np.setdiff1d(np.arange(K), keys)
    assert_bitwise(Wg[untouched], W[untouched], "untouched W rows")
    assert_bitwise(Gg[untouched], G[untouched], "untouched G rows")


def test_wide_first_touch_closed_form():
    """Distinct keys with zero accumulators and |g| >= 2^-9: every element
    moves by exactly lr against the sign of its gradient, in every column
    slice."""
    K, d, n = 2000, 1000, 1500
    W, G, Wt, Gt, s = make(K, d, 9, False, g_fill=False)
    rng = np.random.default_rng(9)
    keys = rng.permutation(K)[:n].astype(np.int64)
    grads = (rng.uniform(0.01, 5, (n, d)) * rng.choice([-1, 1], (n, d))).astype(np.float32)
    s.push(dev(keys), dev(grads))
    expect = W.copy()
    expect[keys] = (W[keys] - np.float32(LR) * np.sign(grads)).astype(np.float32)
    assert_bitwise(Wt.cpu().numpy(), expect, "W after first touch")


@pytest.mark.parametrize("d", [600, 2000])
def test_wide_two_phase_and_allocation_free_pushes_equal_the_push(d):
    K, n = 3000, 20_000
    keys, grads = random_push(K, n, d, 12, zipf_s=1.05)
    runs = []
    for mode in ("push", "two_phase", "noalloc"):
        W, G, Wt, Gt, s = make(K, d, 11, True)
        k, g = dev(keys), dev(grads)
        if mode == "push":
            s.push(k, g)
        elif mode == "two_phase":
            ws = s.push_workspace(n)
            s.push_prepare(k, ws)
            s.push_apply(n, g, ws)
        else:
            need = s.workspace_bytes(_lib.PS_OP_PUSH, n, 1)
            assert need <= _lib.PS_NOALLOC_SCRATCH_BYTES, need
            s.push_noalloc(k, g)
        assert s.error() == 0
        runs.append((Wt.cpu().numpy(), Gt.cpu().numpy()))
    for name, (Wg, Gg) in zip(("two-phase", "allocation-free"), runs[1:]):
        assert_bitwise(Wg, runs[0][0], f"W {name} vs push")
        assert_bitwise(Gg, runs[0][1], f"G {name} vs push")


def test_wide_rows_are_refused_by_the_steps():
    K, d = 1000, 600
    W, G, Wt, Gt, s = make(K, d, 13, False)
    r = torch.zeros(8, dtype=torch.int32, device="cuda")
    v = torch.zeros(8, dtype=torch.float32, device="cuda")
    with pytest.raises(RuntimeError, match="at most 512"):
        s.step_mf(r, r, v, 500, 0.01)
    with pytest.raises(RuntimeError, match="at most 512"):
        s.push_async(torch.zeros(8, dtype=torch.int64, device="cuda"),
                     torch.zeros((8, d), dtype=torch.float32, device="cuda"))
    assert_bitwise(Wt.cpu().numpy(), W, "W untouched by the refused calls")

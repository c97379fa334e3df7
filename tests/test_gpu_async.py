"""GPU checks of the unmerged (asynchronous) updates, ps_push_async and
ps_step_mf_async, against the oracle's push_sequential: the order in which
occurrences of one key are applied is not fixed, so each element of W must
equal the result of SOME order (checked exactly for keys with at most three
occurrences, by enumerating their orders), lie within async_bounds for any
number of occurrences, and G must equal the order-free sum of squares."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store, _lib
from paper_2206_00470_amd.workloads import MF_10Mx1M, MFWorkload, random_push, small_variant
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10
RTOL, ATOL = 1e-5, 1e-6


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def orders_up_to_three(keys):
    """Six occurrence orders that, between them, apply the occurrences of
    every key with at most three occurrences in each of its possible orders."""
    groups = {}
    for i, k in enumerate(keys.tolist()):
        groups.setdefault(k, []).append(i)
    assert max(len(g) for g in groups.values()) <= 3
    out = []
    for p in range(6):
        order = []
        for g in groups.values():
            perms = list(itertools.permutations(g))
            order.extend(perms[p % len(perms)])
        out.append(np.array(order, np.int64))
    return out


def check_some_order(Wg, W0, G0, keys, grads, rowwise=False):
    """Every element of Wg equals, to the tolerance, its value after one of
    the enumerated orders."""
    best = np.full(Wg.shape, np.inf)
    for order in orders_up_to_three(keys):
        Wr, Gr = W0.copy(), G0.copy()
        oracle.push_sequential(Wr, Gr, keys, grads, LR, EPS, order=order, rowwise=rowwise)
        best = np.minimum(best, np.abs(Wg - Wr) - (ATOL + RTOL * np.abs(Wr)))
    bad = best > 0
    assert not bad.any(), f"{bad.sum()} elements match no order of their key's occurrences"


U32 = 2.0 ** -24   # unit roundoff of fp32


def counts_per_key(K, keys, shape):
    ok = (keys >= 0) & (keys < K)
    n = np.bincount(keys[ok], minlength=K).astype(np.float64)
    return n[:, None] if len(shape) == 2 else n


def check_bounds(Wg, W0, G0, keys, grads, rowwise=False, lr=LR, eps=EPS):
    """Wg within the any-order interval; the slack for fp32 rounding grows
    with the number n_k of the key's occurrences: each of its n_k updates
    rounds once in W and its step a few times (|W| along the way is at most
    |W0| plus the sum of the steps' largest magnitudes)."""
    lo, hi = oracle.async_bounds(W0, G0, keys, grads, lr, eps, rowwise=rowwise)
    lo_abs, _ = oracle.async_bounds(W0, G0, keys, np.abs(grads), lr, eps, rowwise=rowwise)
    reach = np.abs(W0) + (W0 - lo_abs)
    n = counts_per_key(W0.shape[0], keys, W0.shape)
    tol = ATOL + RTOL * np.abs(Wg) + 4.0 * n * U32 * reach
    out = (Wg < lo - tol) | (Wg > hi + tol)
    assert not out.any(), f"{out.sum()} elements outside the any-order bounds"


def check_accumulators(Gg, G0, keys, grads, rowwise=False):
    """G after any order: the initial value plus the sum of the squares
    (exact in fp64), up to the rounding of n_k fp32 additions."""
    K = G0.shape[0]
    ok = (keys >= 0) & (keys < K)
    g = grads[ok].astype(np.float64)
    exact = G0.astype(np.float64).copy()
    np.add.at(exact, keys[ok], (g * g).sum(axis=1) / g.shape[1] if rowwise else g * g)
    n = counts_per_key(K, keys, G0.shape)
    tol = ATOL + RTOL * np.abs(exact) + (n + 1.0) * U32 * np.abs(exact)
    bad = np.abs(Gg - exact) > tol
    assert not bad.any(), f"{bad.sum()} accumulators off the sum of squares"


def keys_with_at_most_three(K, n_distinct, seed):
    rng = np.random.default_rng(seed)
    base = rng.permutation(K)[:n_distinct]
    keys = np.concatenate([base, base[: n_distinct * 2 // 3], base[: n_distinct // 3]])
    return rng.permutation(keys).astype(np.int64)


@pytest.mark.parametrize("K,d", [(5000, 100), (3000, 16), (2000, 3), (800, 300), (600, 512)])
def test_push_async_some_order(K, d):
    say(f"unmerged push K={K} d={d}")
    rng = np.random.default_rng(20)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    G0 = rng.uniform(0, 1, (K, d)).astype(np.float32)
    keys = keys_with_at_most_three(K, K // 2, 21)
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    Wt, Gt = dev(W0), dev(G0)
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    assert s.error() == 0
    Wg, Gg = Wt.cpu().numpy(), Gt.cpu().numpy()
    check_some_order(Wg, W0, G0, keys, grads)
    check_bounds(Wg, W0, G0, keys, grads)
    check_accumulators(Gg, G0, keys, grads)
    untouched = np.setdiff1d(np.arange(K), keys)
    assert_bitwise(Wg[untouched], W0[untouched], "untouched rows")


def test_push_async_interleaved_rows():
    """W and G rows of a key side by side in one allocation (the benchmark's
    layout)."""
    from paper_2206_00470_amd.store import interleaved_tables
    K, d = 3000, 100
    rng = np.random.default_rng(31)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    G0 = rng.uniform(0, 1, (K, d)).astype(np.float32)
    keys = keys_with_at_most_three(K, 2000, 32)
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    Wt, Gt = interleaved_tables(dev(W0), dev(G0))
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    assert s.error() == 0
    Wg, Gg = np.ascontiguousarray(Wt.cpu().numpy()), np.ascontiguousarray(Gt.cpu().numpy())
    check_some_order(Wg, W0, G0, keys, grads)
    check_accumulators(Gg, G0, keys, grads)


def test_push_async_unaligned_gradient_rows():
    """Gradient rows starting 4 bytes past a 16-byte boundary are accepted
    (the unmerged push loads one float per lane)."""
    K, d, n = 1000, 100, 700
    rng = np.random.default_rng(33)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    keys = rng.permutation(K)[:n].astype(np.int64)
    grads = rng.standard_normal((n, d)).astype(np.float32)
    buf = torch.zeros(n * d + 1, dtype=torch.float32, device="cuda")
    buf[1:].copy_(dev(grads).reshape(-1))
    Wt, Gt = dev(W0), torch.zeros((K, d), dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), buf[1:])
    assert s.error() == 0
    Wr, Gr = W0.copy(), np.zeros((K, d), np.float32)
    oracle.push(Wr, Gr, keys, grads, LR, EPS)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")


def test_push_async_distinct_keys_equal_the_merged_push():
    K, d, n = 20_000, 100, 15_000
    rng = np.random.default_rng(22)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    keys = rng.permutation(K)[:n].astype(np.int64)
    grads = rng.standard_normal((n, d)).astype(np.float32)
    Wt, Gt = dev(W0), torch.zeros((K, d), dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    Wr, Gr = W0.copy(), np.zeros((K, d), np.float32)
    oracle.push(Wr, Gr, keys, grads, LR, EPS)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")
    assert_close_tables(Gt.cpu().numpy(), Gr, "G")


@pytest.mark.parametrize("zipf", [1.1, 1.5])
def test_push_async_hot_keys_within_bounds(zipf):
    """Zipf keys: the hottest keys take hundreds of occurrences in one launch."""
    K, d, n = 10_000, 64, 200_000
    keys, grads = random_push(K, n, d, 23, zipf_s=zipf)
    counts = np.bincount(keys, minlength=K)
    say(f"zipf {zipf}: most occurrences of one key {counts.max()}")
    W0 = (np.random.default_rng(24).standard_normal((K, d)) * 0.1).astype(np.float32)
    G0 = np.zeros((K, d), np.float32)
    Wt, Gt = dev(W0), dev(G0)
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    assert s.error() == 0
    check_bounds(Wt.cpu().numpy(), W0, G0, keys, grads)
    check_accumulators(Gt.cpu().numpy(), G0, keys, grads)


def test_push_async_identical_rows_are_order_free():
    """Equal gradient rows on a key: every order gives the same result, so
    the unmerged push must equal the sequential oracle."""
    K, d = 500, 32
    rng = np.random.default_rng(25)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    G0 = rng.uniform(0, 1, (K, d)).astype(np.float32)
    per_key = rng.standard_normal((K, d)).astype(np.float32)
    keys = rng.integers(0, K, 20_000).astype(np.int64)
    grads = per_key[keys]
    Wt, Gt = dev(W0), dev(G0)
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    Wr, Gr = W0.copy(), G0.copy()
    oracle.push_sequential(Wr, Gr, keys, grads, LR, EPS)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")
    assert_close_tables(Gt.cpu().numpy(), Gr, "G")


def test_push_async_rowwise():
    K, d = 4000, 100
    rng = np.random.default_rng(26)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    A0 = rng.uniform(0, 1, K).astype(np.float32)
    keys = keys_with_at_most_three(K, 3000, 27)
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    Wt, At = dev(W0), dev(A0)
    s = Store(Wt, At, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    assert s.error() == 0
    Wg = Wt.cpu().numpy()
    check_some_order(Wg, W0, A0, keys, grads, rowwise=True)
    check_bounds(Wg, W0, A0, keys, grads, rowwise=True)
    Ar = A0.copy()
    oracle.push_sequential(W0.copy(), Ar, keys, grads, LR, EPS, rowwise=True)
    assert_close_tables(At.cpu().numpy(), Ar, "row accumulators")


def test_push_async_invalid_keys_skipped_and_flagged():
    K, d = 100, 8
    rng = np.random.default_rng(28)
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    keys = np.array([3, -1, K, 7, 3 + K * 10, 50], np.int64)
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    Wt, Gt = dev(W0), torch.zeros((K, d), dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(dev(keys), dev(grads))
    assert s.error() == _lib.PS_ERR_KEY_RANGE
    Wr, Gr = W0.copy(), np.zeros((K, d), np.float32)
    assert oracle.push_sequential(Wr, Gr, keys, grads, LR, EPS) == 3
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")


def run_mf_async(cfg, steps):
    wl = MFWorkload(cfg)
    W = wl.init_table()
    Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    for step in steps:
        bt = wl.batch(step)
        say(f"unmerged {cfg.name} step {step}: B={bt.row.size}")
        W0, G0 = Wt.cpu().numpy(), Gt.cpu().numpy()
        loss = s.step_mf_async(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)
        assert s.error() == 0
        keys, grads, rloss, bad = oracle.grad_mf(W0, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam)
        assert bad == 0
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        Wg, Gg = Wt.cpu().numpy(), Gt.cpu().numpy()
        check_bounds(Wg, W0, G0, keys, grads, lr=cfg.opt.lr, eps=cfg.opt.eps)
        check_accumulators(Gg, G0, keys, grads)
    return s


def test_mf_async_small_steps():
    run_mf_async(small_variant(MF_10Mx1M), range(3))


def test_mf_async_paper_scale_sampled():
    """10M x 1M factors of rank 100, one batch of 2^20 entries: the loss in
    full, and the bounds and accumulators on 3,000 sampled touched keys
    (their rows and occurrences only)."""
    cfg = MF_10Mx1M
    wl = MFWorkload(cfg)
    say("generating the 11M x 100 table")
    W = wl.init_table()
    Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    bt = wl.batch(0)
    loss = s.step_mf_async(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)
    assert s.error() == 0
    say("oracle gradients")
    keys, grads, rloss, bad = oracle.grad_mf(W, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam)
    assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    rng = np.random.default_rng(29)
    uk = np.unique(keys)
    ck = keys[keys >= cfg.n_rows] - cfg.n_rows
    hot = np.bincount(ck, minlength=cfg.n_cols).argsort()[-50:] + cfg.n_rows   # the most frequent columns
    sample = np.unique(np.concatenate([rng.choice(uk, 3000, replace=False), hot]))
    sel = np.isin(keys, sample)
    local = np.searchsorted(sample, keys[sel])
    idx = torch.from_numpy(sample).cuda()
    Wg, Gg = Wt[idx].cpu().numpy(), Gt[idx].cpu().numpy()
    W0s, G0s = W[sample], np.zeros((sample.size, cfg.dim), np.float32)
    say(f"checking {sample.size} keys with {int(sel.sum())} occurrences")
    check_bounds(Wg, W0s, G0s, local, grads[sel], lr=cfg.opt.lr, eps=cfg.opt.eps)
    check_accumulators(Gg, G0s, local, grads[sel])


def test_mf_async_rowwise_store():
    """Row-wise AdaGrad under the unmerged MF step (accumulators in the
    padding of each value row)."""
    from paper_2206_00470_amd.store import padded_rowwise_table
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    W = wl.init_table()
    Wt, At = padded_rowwise_table(torch.from_numpy(W).cuda())
    s = Store(Wt, At, cfg.opt.lr, cfg.opt.eps)
    for step in range(2):
        bt = wl.batch(step)
        W0, A0 = np.ascontiguousarray(Wt.cpu().numpy()), np.ascontiguousarray(At.cpu().numpy())
        loss = s.step_mf_async(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)
        assert s.error() == 0
        keys, grads, rloss, _ = oracle.grad_mf(W0, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam)
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        check_bounds(np.ascontiguousarray(Wt.cpu().numpy()), W0, A0, keys, grads, rowwise=True, lr=cfg.opt.lr,
                     eps=cfg.opt.eps)
        check_accumulators(np.ascontiguousarray(At.cpu().numpy()), A0, keys, grads, rowwise=True)


def test_async_rejects_bf16_and_staged_stores():
    from paper_2206_00470_amd import StagedStore
    K, d = 100, 8
    Wb = torch.zeros((K, d), dtype=torch.bfloat16, device="cuda")
    s = Store(Wb, torch.zeros((K, d), dtype=torch.float32, device="cuda"), LR, EPS)
    keys, grads = dev(np.arange(4, dtype=np.int64)), torch.ones((4, d), dtype=torch.float32, device="cuda")
    with pytest.raises(_lib.PSError) as e:
        s.push_async(keys, grads)
    assert e.value.status == _lib.PS_ERR_UNSUPPORTED
    st = StagedStore(np.zeros((K, d), np.float32), [0], [50], LR, EPS)
    with pytest.raises(_lib.PSError) as e:
        st.push_async(keys, grads)
    assert e.value.status == _lib.PS_ERR_UNSUPPORTED


def test_async_empty_push_and_step_are_no_ops():
    K, d = 100, 16
    W0 = np.random.default_rng(30).standard_normal((K, d)).astype(np.float32)
    Wt, Gt = dev(W0), torch.zeros((K, d), dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, LR, EPS)
    s.push_async(torch.zeros(0, dtype=torch.int64, device="cuda"), torch.zeros((0, d), device="cuda"))
    e = torch.zeros(0, dtype=torch.int32, device="cuda")
    loss = s.step_mf_async(e, e, torch.zeros(0, dtype=torch.float32, device="cuda"), 60, 0.01)
    assert s.error() == 0 and float(loss.item()) == 0.0
    assert_bitwise(Wt.cpu().numpy(), W0, "W")

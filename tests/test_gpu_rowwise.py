"""GPU parity of the row-wise AdaGrad store (one accumulator per key) against
the CPU oracle's push_rowwise / step_rowwise, for the accumulators as a
separate vector and in the padding of each value row."""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store
from paper_2206_00470_amd.store import padded_rowwise_table
from paper_2206_00470_amd.workloads import (CTR_33M, KGE_COMPLEX, MF_10Mx1M, SGNS_1M, CTRWorkload, KGEWorkload,
                                            MFWorkload, SGNSWorkload, normal_table, random_push, small_variant)
from tests.helpers import assert_bitwise, assert_close_tables, mismatch_fraction, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10
LAYOUTS = ["vector", "padded"]


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def rowwise_store(W, A, layout, lr=LR, eps=EPS):
    """Device tables for a row-wise store; returns (store, W view, A view)."""
    if layout == "vector":
        Wt, At = dev(W), dev(A)
    else:
        Wt, At = padded_rowwise_table(dev(W), dev(A))
    return Store(Wt, At, lr, eps), Wt, At


# ------------------------------------------------------------------ push
PUSH_CASES = [
    # K, d, n, zipf (None = uniform), accumulators prefilled
    (1, 4, 1, None, False),
    (3, 16, 1000, None, False),          # long segments split into chunks (finalize path)
    (5000, 16, 4097, 1.1, True),
    (23_000, 100, 300_001, 1.1, True),   # hot keys far longer than a chunk (fold path)
    (3000, 3, 2000, None, True),         # dim not a multiple of 4
    (6000, 300, 20_000, 0.75, False),
    (1 << 16, 64, 212_992, 1.05, False),
    (500, 512, 3000, 1.0, True),
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("K,d,n,zipf,afill", PUSH_CASES)
def test_push_rowwise_parity(K, d, n, zipf, afill, layout):
    say(f"row-wise push K={K} d={d} n={n} zipf={zipf} layout={layout}")
    W = normal_table(K, d, 0.1, 30, 1)
    rng = np.random.default_rng(30)
    A = rng.uniform(0, 1, K).astype(np.float32) if afill else np.zeros(K, np.float32)
    keys, grads = random_push(K, n, d, 31, zipf_s=zipf)
    s, Wt, At = rowwise_store(W, A, layout)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Ar = W.copy(), A.copy()
    oracle.push_rowwise(Wr, Ar, keys, grads, LR, EPS)
    Wg, Ag = Wt.cpu().numpy(), At.cpu().numpy()
    assert_close_tables(Wg, Wr, "W")
    assert_close_tables(Ag, Ar, "accumulators")
    untouched = np.setdiff1d(np.arange(K), keys)
    assert_bitwise(Wg[untouched], W[untouched], "untouched W rows")
    assert_bitwise(Ag[untouched], A[untouched], "untouched accumulators")
    say(f"  W words differing from the oracle: {mismatch_fraction(Wg, Wr):.2e}")


@pytest.mark.parametrize("counts", [[8192, 16384, 3, 2], [1, 8191, 8193, 16383], [24576]])
def test_push_rowwise_long_segments(counts):
    say(f"row-wise push long segments {counts}")
    K, d = len(counts) + 3, 100
    W = normal_table(K, d, 0.1, 32, 1)
    A = np.random.default_rng(32).uniform(0, 1, K).astype(np.float32)
    rng = np.random.default_rng(33)
    keys = rng.permutation(np.repeat(np.arange(len(counts)), counts)).astype(np.int64)
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    s, Wt, At = rowwise_store(W, A, "padded")
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Ar = W.copy(), A.copy()
    oracle.push_rowwise(Wr, Ar, keys, grads, LR, EPS)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")
    assert_close_tables(At.cpu().numpy(), Ar, "accumulators")


@pytest.mark.parametrize("layout", LAYOUTS)
def test_push_rowwise_first_touch_is_exactly_lr(layout):
    """Equal magnitudes across each merged row, zero accumulators: each
    element steps by exactly lr against the sign of its gradient (the
    oracle's closed-form pin), on the short and the chunked paths."""
    K, d = 4000, 100
    rng = np.random.default_rng(34)
    W = normal_table(K, d, 0.1, 34, 1)
    keys = np.concatenate([rng.permutation(K - 1), np.full(3000, K - 1)]).astype(np.int64)
    # x of at most 8 significant bits: every merged magnitude y (x, or 3000x
    # for the hot key) has at most 20, so y*y and the fp64 sum of dim copies
    # are exact, the row mean is y*y and its square root y
    x = (rng.integers(1, 256, K) * 2.0 ** -6).astype(np.float32)
    sign = rng.choice([-1.0, 1.0], (keys.size, d)).astype(np.float32)
    # the hot key's occurrences carry one signed row, so its merged row is 3000*x*sign
    sign[K - 1:] = sign[K - 1]
    grads = (x[keys][:, None] * sign).astype(np.float32)
    s, Wt, At = rowwise_store(W, np.zeros(K, np.float32), layout)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    g_merged = np.zeros((K, d), np.float64)
    np.add.at(g_merged, keys, grads.astype(np.float64))
    g32 = g_merged.astype(np.float32)
    expect = (W - np.float32(LR) * np.sign(g32)).astype(np.float32)
    assert_bitwise(Wt.cpu().numpy(), expect, "W after first touch")
    assert_bitwise(At.cpu().numpy(), (np.abs(g32[:, 0]) * np.abs(g32[:, 0])).astype(np.float32), "accumulators")


def test_push_rowwise_zero_gradients_leave_state_unchanged():
    K, d = 3000, 64
    W = normal_table(K, d, 0.1, 35, 1)
    A = np.where(np.arange(K) % 3 == 0, 0, np.random.default_rng(35).uniform(0, 2, K)).astype(np.float32)
    s, Wt, At = rowwise_store(W, A, "padded")
    keys = np.random.default_rng(36).integers(0, K, 50_000)
    s.push(dev(keys), torch.zeros((keys.size, d), dtype=torch.float32, device="cuda"))
    assert s.error() == 0
    assert_bitwise(Wt.cpu().numpy(), W, "W after zero push")
    assert_bitwise(At.cpu().numpy(), A, "accumulators after zero push")


def test_push_rowwise_padding_beside_the_accumulator_is_untouched():
    """Padded layout: the pad columns other than the accumulator keep their bits."""
    K, d = 2000, 100
    W = normal_table(K, d, 0.1, 37, 1)
    T = torch.full((K, d + 4), 7.25, dtype=torch.float32, device="cuda")
    T[:, :d] = dev(W)
    T[:, d] = 0
    s = Store(T[:, :d], T[:, d], LR, EPS)
    keys, grads = random_push(K, 40_000, d, 38, zipf_s=1.1)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Tg = T.cpu().numpy()
    assert np.all(Tg[:, d + 1:] == np.float32(7.25))


# ------------------------------------------------------------------ task steps
def mf_args(cfg, bt):
    return (bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam)


def mf_gpu(s, cfg, bt):
    return s.step_mf(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)


def kge_args(cfg, bt):
    return (bt.head, bt.rel, bt.tail, bt.neg, cfg.n_head_neg, cfg.n_ent)


def kge_gpu(s, cfg, bt):
    return s.step_kge(dev(bt.head), dev(bt.rel), dev(bt.tail), dev(bt.neg), cfg.n_head_neg, cfg.n_ent)


def sgns_args(cfg, bt):
    return (bt.centre, bt.ctx, bt.neg, cfg.window, cfg.vocab)


def sgns_gpu(s, cfg, bt):
    return s.step_sgns(dev(bt.centre), dev(bt.ctx), dev(bt.neg), cfg.window, cfg.vocab)


def ctr_args(cfg, bt):
    return (bt.keys, bt.label)


def ctr_gpu(s, cfg, bt):
    return s.step_ctr(dev(bt.keys), dev(bt.label))


TASKS = {
    "mf": (MF_10Mx1M, MFWorkload, mf_gpu, mf_args),
    "kge": (KGE_COMPLEX, KGEWorkload, kge_gpu, kge_args),
    "sgns": (SGNS_1M, SGNSWorkload, sgns_gpu, sgns_args),
    "ctr": (CTR_33M, CTRWorkload, ctr_gpu, ctr_args),
}


def run_rowwise_steps(task, cfg, steps, layout):
    """Every step starts the oracle from the GPU's pre-step state."""
    _, WL, gpu, args = TASKS[task]
    wl = WL(cfg)
    W = wl.init_table()
    s, Wt, At = rowwise_store(W, np.zeros(W.shape[0], np.float32), layout, cfg.opt.lr, cfg.opt.eps)
    for step in steps:
        say(f"row-wise {cfg.name} step {step} ({layout})")
        bt = wl.batch(step)
        Wr, Ar = Wt.cpu().numpy(), At.cpu().numpy()
        loss = gpu(s, cfg, bt)
        assert s.error() == 0
        rloss, bad = oracle.step_rowwise(task, Wr, Ar, args(cfg, bt), cfg.opt.lr, cfg.opt.eps)
        assert bad == 0
        Wg, Ag = Wt.cpu().numpy(), At.cpu().numpy()
        assert_close_tables(Wg, Wr, f"W after step {step}")
        assert_close_tables(Ag, Ar, f"accumulators after step {step}")
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        say(f"  loss {rloss:.6g}; W words differing from the oracle: {mismatch_fraction(Wg, Wr):.2e}")


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("task", ["mf", "kge", "sgns", "ctr"])
def test_rowwise_small_steps(task, layout):
    run_rowwise_steps(task, small_variant(TASKS[task][0]), range(3), layout)


def test_rowwise_mf_paper_scale_one_step():
    """10M x 1M, rank 100, 1,048,576 entries, accumulators in the row padding
    (row stride 104): the bench's row-wise launch."""
    cfg = MF_10Mx1M
    wl = MFWorkload(cfg)
    say("generating the 11M x 100 table")
    W = wl.init_table()
    A = np.zeros(W.shape[0], np.float32)
    s, Wt, At = rowwise_store(W, A, "padded", cfg.opt.lr, cfg.opt.eps)
    bt = wl.batch(0)
    say("gpu step")
    loss = mf_gpu(s, cfg, bt)
    assert s.error() == 0
    say("oracle step")
    rloss, bad = oracle.step_rowwise("mf", W, A, mf_args(cfg, bt), cfg.opt.lr, cfg.opt.eps)
    say("compare")
    assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    assert_close_tables(Wt.cpu().numpy(), W, "W")
    assert_close_tables(At.cpu().numpy(), A, "accumulators")

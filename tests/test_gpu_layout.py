"""GPU parity with the row-interleaved table layout (W and G rows of a key side
by side in one [num_keys, 2*dim] allocation): every call must give what the
dense layout and the oracle give."""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store
from paper_2206_00470_amd.store import interleaved_tables
from paper_2206_00470_amd.workloads import (CTR_33M, KGE_COMPLEX, MF_10Mx1M, SGNS_1M, MFWorkload, normal_table,
                                            random_push, small_variant, workload)
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def interleaved_store(W, G, lr=LR, eps=EPS):
    Wt, Gt = interleaved_tables(dev(W), dev(G))
    assert Wt.stride(0) == 2 * W.shape[1]
    return Store(Wt, Gt, lr, eps), Wt, Gt


@pytest.mark.parametrize("K,d,n", [(1000, 100, 20_000), (777, 3, 5000), (4000, 256, 3000)])
def test_pull_interleaved(K, d, n):
    W = normal_table(K, d, 0.1, 1, 2)
    s, Wt, Gt = interleaved_store(W, np.ones_like(W))
    keys = np.random.default_rng(n).integers(0, K, n)
    out = s.pull(dev(keys))
    assert s.error() == 0
    assert_bitwise(out.cpu().numpy(), W[keys], "pull")


@pytest.mark.parametrize("K,d,n,zipf", [(23_000, 100, 300_001, 1.1), (3000, 3, 2000, None), (6000, 300, 20_000, 0.75),
                                        (1 << 16, 64, 212_992, 1.05)])
def test_push_interleaved(K, d, n, zipf):
    say(f"interleaved push K={K} d={d} n={n}")
    W = normal_table(K, d, 0.1, 3, 4)
    G = np.random.default_rng(5).uniform(0, 1, (K, d)).astype(np.float32)
    keys, grads = random_push(K, n, d, 6, zipf_s=zipf)
    s, Wt, Gt = interleaved_store(W, G)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Gr = W.copy(), G.copy()
    oracle.push(Wr, Gr, keys, grads, LR, EPS)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")
    assert_close_tables(Gt.cpu().numpy(), Gr, "G")


def _step(task, s, cfg, bt):
    if task == "mf":
        return s.step_mf(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)
    if task == "kge":
        return s.step_kge(dev(bt.head), dev(bt.rel), dev(bt.tail), dev(bt.neg), cfg.n_head_neg, cfg.n_ent)
    if task == "sgns":
        return s.step_sgns(dev(bt.centre), dev(bt.ctx), dev(bt.neg), cfg.window, cfg.vocab)
    return s.step_ctr(dev(bt.keys), dev(bt.label))


def _ref(task, W, G, cfg, bt):
    lr, eps = cfg.opt.lr, cfg.opt.eps
    if task == "mf":
        return oracle.step_mf(W, G, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam, lr, eps)
    if task == "kge":
        return oracle.step_kge(W, G, bt.head, bt.rel, bt.tail, bt.neg, cfg.n_head_neg, cfg.n_ent, lr, eps)
    if task == "sgns":
        return oracle.step_sgns(W, G, bt.centre, bt.ctx, bt.neg, cfg.window, cfg.vocab, lr, eps)
    return oracle.step_ctr(W, G, bt.keys, bt.label, lr, eps)


@pytest.mark.parametrize("task,cfg", [("mf", MF_10Mx1M), ("kge", KGE_COMPLEX), ("sgns", SGNS_1M), ("ctr", CTR_33M)])
def test_steps_interleaved_match_oracle_and_dense(task, cfg):
    cfg = small_variant(cfg)
    wl = workload(cfg)
    W = wl.init_table()
    G = np.zeros_like(W)
    s, Wt, Gt = interleaved_store(W, G, cfg.opt.lr, cfg.opt.eps)
    Wd, Gd = dev(W), dev(G)
    sd = Store(Wd, Gd, cfg.opt.lr, cfg.opt.eps)
    Wr, Gr = W.copy(), G.copy()
    for step in range(2):
        bt = wl.batch(step)
        loss = _step(task, s, cfg, bt)
        lossd = _step(task, sd, cfg, bt)
        rloss, bad = _ref(task, Wr, Gr, cfg, bt)
        assert s.error() == 0 and sd.error() == 0 and bad == 0
        assert_bitwise(Wt.cpu().numpy(), Wd.cpu().numpy(), "W interleaved vs dense")
        assert_bitwise(Gt.cpu().numpy(), Gd.cpu().numpy(), "G interleaved vs dense")
        assert float(loss.item()) == float(lossd.item())
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W vs oracle")
    assert_close_tables(Gt.cpu().numpy(), Gr, "G vs oracle")


def test_mf_paper_scale_interleaved():
    """The bench's configuration: 10M x 1M, rank 100, interleaved tables."""
    cfg = MF_10Mx1M
    wl = MFWorkload(cfg)
    say("generating the 11M x 100 table")
    W = wl.init_table()
    G = np.zeros_like(W)
    s, Wt, Gt = interleaved_store(W, G, cfg.opt.lr, cfg.opt.eps)
    for step in range(2):
        bt = wl.batch(step)
        say(f"gpu step {step}")
        loss = _step("mf", s, cfg, bt)
        assert s.error() == 0
        say(f"oracle step {step}")
        rloss, bad = _ref("mf", W, G, cfg, bt)
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    say("compare")
    assert_close_tables(Wt.cpu().numpy(), W, "W")
    assert_close_tables(Gt.cpu().numpy(), G, "G")

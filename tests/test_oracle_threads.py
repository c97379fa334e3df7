"""The oracle's steps spread over host threads (used to time the oracle on
all of a host's cores) leave W and G bit for bit as the one-thread steps."""
from dataclasses import replace

import numpy as np
import pytest

import oracle
from paper_2206_00470_amd.workloads import (CTR_33M, KGE_COMPLEX, MF_10Mx1M, SGNS_1M, CTRWorkload, KGEWorkload,
                                            MFWorkload, SGNSWorkload, small_variant)

CASES = {
    "mf": (MF_10Mx1M, MFWorkload, lambda c, b: (b.row, b.col, b.val, c.n_rows, c.lam), oracle.step_mf),
    "kge": (KGE_COMPLEX, KGEWorkload, lambda c, b: (b.head, b.rel, b.tail, b.neg, c.n_head_neg, c.n_ent),
            oracle.step_kge),
    "sgns": (SGNS_1M, SGNSWorkload, lambda c, b: (b.centre, b.ctx, b.neg, c.window, c.vocab), oracle.step_sgns),
    "ctr": (CTR_33M, CTRWorkload, lambda c, b: (b.keys, b.label), oracle.step_ctr),
}


@pytest.mark.parametrize("threads", [1, 3, 8])
@pytest.mark.parametrize("task", list(CASES))
def test_threaded_step_equals_the_one_thread_step(task, threads):
    base, WL, args, step = CASES[task]
    cfg = small_variant(base)
    if task == "mf":
        cfg = replace(cfg, row_zipf_s=1.1)          # hot row keys: long merges split across ranges
    wl = WL(cfg)
    W = wl.init_table()
    G = np.random.default_rng(5).uniform(0, 1, W.shape).astype(np.float32)
    W1, G1, W2, G2 = W.copy(), G.copy(), W.copy(), G.copy()
    for s in range(2):
        bt = wl.batch(s)
        if task == "ctr" and s == 1:
            bt.keys[3, 2] = -7                      # a skipped sample
        l1, b1 = step(W1, G1, *args(cfg, bt), cfg.opt.lr, cfg.opt.eps)
        l2, b2 = oracle.step_threads(task, W2, G2, args(cfg, bt), cfg.opt.lr, cfg.opt.eps, threads)
        assert b1 == b2
        assert l2 == pytest.approx(l1, rel=1e-10)     # another order of additions
        assert np.array_equal(W1.view(np.uint32), W2.view(np.uint32))
        assert np.array_equal(G1.view(np.uint32), G2.view(np.uint32))

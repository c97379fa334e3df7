"""GPU tests of the staged store: home tables in pinned host memory, slots
in HBM, intent signalling and adaptive action timing.

Each step is checked against the oracle step from the same pre-step state
(the home tables after a flush), and after every round and clock advance
the set of resident keys must equal that of the plain reference planner
(oracle/staging.py) fed the same intents, rounds and advances."""
import numpy as np
import pytest
import torch

import oracle
from oracle.staging import StagingOracle
from paper_2206_00470_amd import StagedStore, _lib
from paper_2206_00470_amd.workloads import (CTR_33M, KGE_COMPLEX, MF_10Mx1M, SGNS_1M, CTRWorkload, KGEWorkload,
                                            MFWorkload, SGNSWorkload, small_variant)
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# ------------------------------------------------------------------ per task
def mf_keys(cfg, bt):
    return np.concatenate([bt.row.astype(np.int64), cfg.n_rows + bt.col.astype(np.int64)])


def mf_gpu(s, cfg, bt):
    return s.step_mf(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)


def mf_ref(W, G, cfg, bt):
    return oracle.step_mf(W, G, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam, cfg.opt.lr, cfg.opt.eps)


def kge_keys(cfg, bt):
    return np.concatenate([bt.head, bt.tail, bt.neg.ravel(), cfg.n_ent + bt.rel.astype(np.int64)]).astype(np.int64)


def kge_gpu(s, cfg, bt):
    return s.step_kge(dev(bt.head), dev(bt.rel), dev(bt.tail), dev(bt.neg), cfg.n_head_neg, cfg.n_ent)


def kge_ref(W, G, cfg, bt):
    return oracle.step_kge(W, G, bt.head, bt.rel, bt.tail, bt.neg, cfg.n_head_neg, cfg.n_ent, cfg.opt.lr, cfg.opt.eps)


def sgns_keys(cfg, bt):
    out = np.concatenate([bt.ctx.ravel(), bt.neg.ravel()]).astype(np.int64)
    return np.concatenate([bt.centre.astype(np.int64), cfg.vocab + out[out >= 0]])


def sgns_gpu(s, cfg, bt):
    return s.step_sgns(dev(bt.centre), dev(bt.ctx), dev(bt.neg), cfg.window, cfg.vocab)


def sgns_ref(W, G, cfg, bt):
    return oracle.step_sgns(W, G, bt.centre, bt.ctx, bt.neg, cfg.window, cfg.vocab, cfg.opt.lr, cfg.opt.eps)


def ctr_keys(cfg, bt):
    return bt.keys.ravel().astype(np.int64)


def ctr_gpu(s, cfg, bt):
    return s.step_ctr(dev(bt.keys), dev(bt.label))


def ctr_ref(W, G, cfg, bt):
    return oracle.step_ctr(W, G, bt.keys, bt.label, cfg.opt.lr, cfg.opt.eps)


def mf_ranges(cfg):
    return [0, cfg.n_rows], [16_000, cfg.n_cols]        # rows: 16,000 slots of 20,000 keys


def kge_ranges(cfg):
    return [0, cfg.n_ent], [cfg.n_ent, cfg.n_rel]


def sgns_ranges(cfg):
    return [0, cfg.vocab], [cfg.vocab, cfg.vocab]


def ctr_ranges(cfg):
    return [0], [16_384]                                 # 16,384 slots of 65,536 keys


TASKS = {
    "mf": (MF_10Mx1M, MFWorkload, mf_keys, mf_gpu, mf_ref, mf_ranges),
    "kge": (KGE_COMPLEX, KGEWorkload, kge_keys, kge_gpu, kge_ref, kge_ranges),
    "sgns": (SGNS_1M, SGNSWorkload, sgns_keys, sgns_gpu, sgns_ref, sgns_ranges),
    "ctr": (CTR_33M, CTRWorkload, ctr_keys, ctr_gpu, ctr_ref, ctr_ranges),
}


def check_same_resident(s, o, what):
    got = s.resident()
    want = np.array(sorted(o.resident()), np.int64)
    assert np.array_equal(got, want), f"{what}: {got.size} resident keys, the reference has {want.size}"


def run_staged(task, steps, lookahead, rounds_per_step, timing=None, seed=0):
    """Explicit rounds (rounds_per_step[i] before the advance to clock i) and
    intents `lookahead` batches ahead; every step is compared with the oracle
    step from the same flushed state, every planner state with the reference."""
    base, WL, keys_of, gpu, ref, ranges_of = TASKS[task]
    cfg = small_variant(base)
    wl = WL(cfg)
    W0 = wl.init_table()
    begin, slots = ranges_of(cfg)
    s = StagedStore(W0, begin, slots, cfg.opt.lr, cfg.opt.eps)
    o = StagingOracle(W0.shape[0], begin, slots)
    if timing:
        s.set_action_timing(*timing)
        o.alpha, o.p, o.lam = timing
    batches = {i: wl.batch(i - 1) for i in range(1, steps + lookahead + 1)}
    for i in range(1, lookahead + 1):
        k = keys_of(cfg, batches[i])
        s.intent(k, i, i + 1)
        o.intent(k, i, i + 1)
    for i in range(1, steps + 1):
        for r in range(rounds_per_step[i - 1]):
            s.round()
            o.round()
            check_same_resident(s, o, f"{task} round {r} before clock {i}")
        s.advance_clock()
        o.advance_clock()
        check_same_resident(s, o, f"{task} clock {i}")
        st = s.stats()
        assert (st["clock"], st["forced"], st["staged"], st["evicted"]) == \
            (i, o.forced, o.staged_total, o.evicted_total)
        s.flush()
        Wh, Gh = s.home_tables()
        Wr, Gr = Wh.copy(), Gh.copy()
        bt = batches[i]
        loss = gpu(s, cfg, bt)
        assert s.error() == 0
        rloss, bad = ref(Wr, Gr, cfg, bt)
        assert bad == 0
        s.flush()
        Wh, Gh = s.home_tables()
        assert_close_tables(Wh, Wr, f"{task} W after step {i}")
        assert_close_tables(Gh, Gr, f"{task} G after step {i}")
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        say(f"{task} step {i}: resident {st['resident']}, staged {st['staged']}, evicted {st['evicted']}, "
            f"forced {st['forced']}, estimate {st['lambda']:.3f}")
        k = keys_of(cfg, batches[i + lookahead]) if i + lookahead in batches else None
        if k is not None:
            s.intent(k, i + lookahead, i + lookahead + 1)
            o.intent(k, i + lookahead, i + lookahead + 1)
    return s, o


@pytest.mark.parametrize("task", ["mf", "kge", "sgns", "ctr"])
def test_staged_steps_match_oracle_and_reference_planner(task):
    run_staged(task, steps=4, lookahead=1, rounds_per_step=[1, 1, 1, 1])


def test_staged_irregular_rounds_and_deferred_action():
    """Rounds at irregular times (none before some advances: forced actions;
    two before others) with a small rate estimate and quantile, so that
    intents signalled three batches ahead wait for later rounds."""
    rng = np.random.default_rng(60)
    rounds = [int(x) for x in rng.choice([0, 1, 2], 7)]
    rounds[0] = 1
    run_staged("mf", steps=7, lookahead=3, rounds_per_step=rounds, timing=(0.3, 0.6, 0.2))


def test_staged_capacity_stalls_like_the_reference():
    """CTR with 4,096 slots: the keys of two batches do not fit, so the first
    round stops at the full range; at clock 2 the first batch's keys expire
    and the forced action stages the rest of the second batch, whose step
    then matches the oracle."""
    cfg = small_variant(CTR_33M)
    wl = CTRWorkload(cfg)
    W0 = wl.init_table()
    s = StagedStore(W0, [0], [4096], cfg.opt.lr, cfg.opt.eps)
    o = StagingOracle(W0.shape[0], [0], [4096])
    b1, b2 = wl.batch(0), wl.batch(1)
    for i, bt in ((1, b1), (2, b2)):
        s.intent(ctr_keys(cfg, bt), i, i + 1)
        o.intent(ctr_keys(cfg, bt), i, i + 1)
    s.round()
    o.round()
    check_same_resident(s, o, "after the first round")
    st = s.stats()
    assert st["resident"] == len(o.resident()) == 4096
    assert st["stalled"] > 0 and o.pending
    for i, bt in ((1, b1), (2, b2)):
        s.advance_clock()
        o.advance_clock()
        check_same_resident(s, o, f"clock {i}")
        s.flush()
        Wh, Gh = s.home_tables()
        Wr, Gr = Wh.copy(), Gh.copy()
        ctr_gpu(s, cfg, bt)
        assert s.error() == 0
        ctr_ref(Wr, Gr, cfg, bt)
        s.flush()
        Wh, Gh = s.home_tables()
        assert_close_tables(Wh, Wr, f"W after step {i}")
        assert_close_tables(Gh, Gr, f"G after step {i}")
    assert s.stats()["forced"] == o.forced == 1


def test_staged_access_without_intent_is_flagged_not_resident():
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    W0 = wl.init_table()
    begin, slots = mf_ranges(cfg)
    s = StagedStore(W0, begin, slots, cfg.opt.lr, cfg.opt.eps)
    bt = wl.batch(0)
    s.advance_clock()
    mf_gpu(s, cfg, bt)                 # no intent at all: every entry is skipped
    assert s.error() == _lib.PS_ERR_NOT_RESIDENT
    s.flush()
    Wh, _ = s.home_tables()
    assert_bitwise(Wh, W0, "home table after a step with nothing resident")
    out = s.pull(dev(np.arange(10, dtype=np.int64)))
    assert s.error() == _lib.PS_ERR_NOT_RESIDENT
    assert not out.cpu().numpy().any()


def test_staged_push_and_pull():
    """ps_push and ps_pull on resident keys equal the oracle's push and the
    home rows after a flush."""
    rng = np.random.default_rng(61)
    K, d = 5000, 64
    W0 = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    s = StagedStore(W0, [0, 2500], [1500, 1500], 0.1, 1e-10)
    # 1,200 distinct keys in each range (1,500 slots each), drawn with repeats
    pool = np.concatenate([rng.choice(2500, 1200, replace=False), 2500 + rng.choice(2500, 1200, replace=False)])
    keys = pool[rng.integers(0, pool.size, 6000)].astype(np.int64)
    s.intent(keys, 1, 2)
    s.round()
    s.advance_clock()
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Gr = W0.copy(), np.zeros_like(W0)
    oracle.push(Wr, Gr, keys, grads, 0.1, 1e-10)
    s.flush()
    Wh, Gh = s.home_tables()
    assert_close_tables(Wh, Wr, "W after a staged push")
    assert_close_tables(Gh, Gr, "G after a staged push")
    u = np.unique(keys)
    out = s.pull(dev(u)).cpu().numpy()
    assert s.error() == 0
    assert_bitwise(out, Wh[u], "pulled rows against the flushed home rows")


def test_staged_auto_rounds_match_oracle_trajectory():
    """Rounds on the library's thread, intents two batches ahead: after six
    steps the flushed home tables equal six oracle steps from the start."""
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    W0 = wl.init_table()
    begin, slots = mf_ranges(cfg)
    s = StagedStore(W0, begin, slots, cfg.opt.lr, cfg.opt.eps)
    batches = [wl.batch(i) for i in range(8)]
    for i in (1, 2):
        s.intent(mf_keys(cfg, batches[i - 1]), i, i + 1)
    s.auto(True)
    Wr, Gr = W0.copy(), np.zeros_like(W0)
    for i in range(1, 7):
        s.advance_clock()
        mf_gpu(s, cfg, batches[i - 1])
        if i + 2 <= 8:
            s.intent(mf_keys(cfg, batches[i + 1]), i + 2, i + 3)
        mf_ref(Wr, Gr, cfg, batches[i - 1])
    torch.cuda.synchronize()
    s.auto(False)
    assert s.error() == 0
    s.flush()
    st = s.stats()
    say(f"auto rounds: {st}")
    assert st["rounds"] > 0
    Wh, Gh = s.home_tables()
    assert_close_tables(Wh, Wr, "W after six auto-staged steps")
    assert_close_tables(Gh, Gr, "G after six auto-staged steps")

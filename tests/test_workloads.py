"""The synthetic input recipe (CPU): word2vec-style subsampling and dynamic
windows for skip-gram, and the column visiting order for MF."""
import numpy as np
import pytest

from paper_2206_00470_amd.workloads import (MF_10Mx1M, MF_10Mx1M_COLORDER, SGNS_1M, SGNS_1M_W2V, MFWorkload,
                                            SGNSWorkload, small_variant)


def test_subsampling_keeps_each_rank_at_the_rule_rate():
    """Keep probability min(1, sqrt(t / f(w))): checked per frequency rank on
    the 100,000 positions of the reduced stream (binomial 5 sigma)."""
    cfg = small_variant(SGNS_1M_W2V)
    wl = SGNSWorkload(cfg)
    pos = np.arange(cfg.n_tokens, dtype=np.int64)
    from paper_2206_00470_amd.workloads import _hash_uniform
    r = wl.zipf.ranks(_hash_uniform(pos.astype(np.uint64) ^ wl._key))
    kept = wl.kept(pos)
    for rank in range(8):
        m = r == rank
        p = min(1.0, np.sqrt(cfg.subsample / wl.zipf.pmf[rank]))
        n = int(m.sum())
        assert abs(kept[m].mean() - p) <= 5 * np.sqrt(p * (1 - p) / n) + 1e-12, (rank, kept[m].mean(), p)
    rare = wl.zipf.pmf[r] <= cfg.subsample   # f <= t: always kept
    assert kept[rare].all() and not wl.kept(np.array([-1, cfg.n_tokens])).any()


def brute_context(wl, step):
    """The batch's centres and contexts by a plain scan of the kept stream."""
    cfg = wl.cfg
    lo = step * cfg.batch
    hi = min(cfg.n_tokens, lo + cfg.batch)
    pos = np.arange(max(0, lo - 500), min(cfg.n_tokens, hi + 500))
    kp = list(pos[wl.kept(pos)])
    out = []
    for i, p in enumerate(kp):
        if lo <= p < hi:
            left = [kp[i - d] if i - d >= 0 else -1 for d in range(cfg.window, 0, -1)]
            right = [kp[i + d] if i + d < len(kp) else -1 for d in range(1, cfg.window + 1)]
            out.append((p, left + right))
    return out


@pytest.mark.parametrize("step", [0, 5])
def test_w2v_contexts_are_the_nearest_kept_tokens_within_the_drawn_window(step):
    cfg = small_variant(SGNS_1M_W2V)
    wl = SGNSWorkload(cfg)
    bt = wl.batch(step)
    ref = brute_context(wl, step)
    assert bt.centre.size == len(ref)
    assert np.array_equal(bt.centre, wl.tokens(np.array([p for p, _ in ref])))
    offs = wl.offsets()
    sizes = []
    for j, (p, cpos) in enumerate(ref):
        present = bt.ctx[j] >= 0
        b = int(np.abs(offs[present]).max()) if present.any() else 0
        sizes.append(b)
        # slots within the drawn window b hold the nearest kept tokens; the rest are absent
        for k, d in enumerate(offs):
            want = wl.tokens(np.array([cpos[k]]))[0] if (abs(d) <= b and cpos[k] >= 0) else -1
            assert bt.ctx[j, k] == want
        assert (bt.neg[j][~present] == -1).all() and (bt.neg[j][present] >= 0).all()
    counts = np.bincount(sizes, minlength=cfg.window + 1)[1:]
    assert counts.min() > 0 and counts.sum() == len(ref)


def test_w2v_off_is_the_plain_generator():
    wl = SGNSWorkload(small_variant(SGNS_1M))
    bt = wl.batch(2)
    assert bt.centre.size == small_variant(SGNS_1M).batch and (bt.ctx >= 0).all()


def test_dynamic_window_sizes_are_uniform_at_full_scale():
    wl = SGNSWorkload(SGNS_1M_W2V)
    bt = wl.batch(0)
    present = (bt.ctx >= 0).sum(axis=1)          # 2b per centre away from the stream ends
    frac = np.bincount(present // 2, minlength=6)[1:] / present.size
    assert np.allclose(frac, 0.2, atol=0.01)
    assert 0.90 < bt.centre.size / SGNS_1M_W2V.batch < 0.95   # about 7% of tokens subsampled


def test_column_order_epoch_visits_each_column_once_with_its_count():
    cfg = small_variant(MF_10Mx1M_COLORDER)
    wl = MFWorkload(cfg)
    cols = np.concatenate([wl.batch(s).col for s in range(cfg.steps_per_epoch)])
    assert cols.size == cfg.nnz
    # contiguous runs in the visiting order
    change = np.flatnonzero(np.diff(cols) != 0) + 1
    runs = np.split(cols, change)
    order = [r[0] for r in runs]
    assert len(set(order)) == len(order)
    place = np.empty(cfg.n_cols, np.int64)
    place[wl.col_order] = np.arange(cfg.n_cols)
    assert np.all(np.diff(place[np.array(order)]) > 0)      # runs follow the visiting order
    # each column's count is its Zipf share of nnz, rounded
    cnt = np.bincount(cols, minlength=cfg.n_cols)
    share = cfg.nnz * wl.zipf.pmf
    assert np.all(np.abs(cnt[wl.zipf.perm] - share) < 1.0)
    assert cnt.sum() == cfg.nnz


def test_column_order_batches_are_deterministic_and_full():
    wl = MFWorkload(MF_10Mx1M_COLORDER)
    a, b = wl.batch(7), wl.batch(7)
    assert np.array_equal(a.row, b.row) and np.array_equal(a.col, b.col) and np.array_equal(a.val, b.val)
    assert a.row.size == MF_10Mx1M.batch
    assert a.row.min() >= 0 and a.row.max() < MF_10Mx1M.n_rows

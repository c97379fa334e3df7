"""GPU parity of the MF step when row keys repeat many times in one batch
(users with many ratings, Appendix C "Matrix factorization").

A row key with more than 32 occurrences is cut into chunks whose partial
sums the merge stores and a finalize pass adds; past 64 x 32 occurrences
whole runs of chunk partials are folded first.  Every store layout and
update variant runs those paths here against the oracle: W and G (or the
row-wise accumulators) after every step within 1e-6 + 1e-5 |ref|, the loss
within 1e-9 relative, untouched rows bit for bit.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store
from paper_2206_00470_amd.store import interleaved_bf16_tables, interleaved_tables, padded_rowwise_table
from paper_2206_00470_amd.workloads import MF_10Mx1M, MFWorkload, small_variant
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu

# 33: one cut; 64, 65: a cut at the CHUNK boundary and just past it; 2,049:
# 64 chunks plus one; 70,001: many whole fold runs of 64 x 32 occurrences
HOT_COUNTS = [33, 64, 65, 2049, 70_001]
N_PLAIN = 5003


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bf16_words(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class Layout:
    """A store of one layout over the initial table W, with host views of its
    state and the oracle step that matches its update."""

    def __init__(self, kind, W, cfg):
        self.kind, self.cfg = kind, cfg
        K, d = W.shape
        if kind == "dense":
            self.Wt, self.Gt = dev(W), dev(np.zeros_like(W))
        elif kind == "interleaved":
            self.Wt, self.Gt = interleaved_tables(dev(W))
        elif kind == "rowwise_vector":
            self.Wt, self.Gt = dev(W), torch.zeros(K, dtype=torch.float32, device="cuda")
        elif kind == "rowwise_padded":
            self.Wt, self.Gt = padded_rowwise_table(dev(W))
        elif kind == "bf16_dense":
            Wb = oracle.f32_to_bf16(W)
            self.Wt = torch.from_numpy(Wb.view(np.int16)).cuda().view(torch.bfloat16)
            self.Gt = torch.zeros((K, d), dtype=torch.float32, device="cuda")
        elif kind == "bf16_interleaved":
            self.Wt, self.Gt = interleaved_bf16_tables(dev(oracle.bf16_to_f32(oracle.f32_to_bf16(W))))
        else:
            raise ValueError(kind)
        self.s = Store(self.Wt, self.Gt, cfg.opt.lr, cfg.opt.eps)

    def state(self):
        W = bf16_words(self.Wt) if self.kind.startswith("bf16") else self.Wt.cpu().numpy()
        return W, self.Gt.cpu().numpy()

    def oracle_step(self, W, G, bt):
        c = self.cfg
        args = (bt.row, bt.col, bt.val, c.n_rows, c.lam)
        if self.kind.startswith("rowwise"):
            return oracle.step_rowwise("mf", W, G, args, c.opt.lr, c.opt.eps)
        if self.kind.startswith("bf16"):
            return oracle.step_mf_bf16(W, G, *args, c.opt.lr, c.opt.eps)
        return oracle.step_mf(W, G, *args, c.opt.lr, c.opt.eps)

    def widened(self, W):
        return oracle.bf16_to_f32(W) if self.kind.startswith("bf16") else W

    def gpu_step(self, bt, two_phase):
        c = self.cfg
        r, co, v = dev(bt.row), dev(bt.col), dev(bt.val)
        if not two_phase:
            return self.s.step_mf(r, co, v, c.n_rows, c.lam)
        ws = self.s.mf_workspace(bt.row.size)
        self.s.step_mf_prepare(r, co, v, c.n_rows, ws)
        return self.s.step_mf_apply(bt.row.size, c.lam, ws)


def check_steps(kind, cfg, batches, two_phase=False):
    wl = MFWorkload(cfg)
    lay = Layout(kind, wl.init_table(), cfg)
    for i, bt in enumerate(batches):
        counts = np.bincount(bt.row)
        say(f"{kind}{' two-phase' if two_phase else ''} {cfg.name} batch {i}: {bt.row.size} entries, "
            f"hottest row key {counts.max()} times")
        Wr, Gr = lay.state()
        W0 = Wr.copy()
        loss = lay.gpu_step(bt, two_phase)
        assert lay.s.error() == 0
        rloss, bad = lay.oracle_step(Wr, Gr, bt)
        assert bad == 0
        Wg, Gg = lay.state()
        assert_close_tables(lay.widened(Wg), lay.widened(Wr), f"W after batch {i}")
        if Gg.ndim == 1:
            assert_close_tables(Gg[:, None], Gr[:, None], f"accumulators after batch {i}")
        else:
            assert_close_tables(Gg, Gr, f"G after batch {i}")
        touched = np.zeros(cfg.num_keys, bool)
        touched[bt.row] = True
        touched[cfg.n_rows + bt.col] = True
        assert_bitwise(Wg[~touched], W0[~touched], "untouched rows")
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)


KINDS = ["dense", "interleaved", "rowwise_vector", "rowwise_padded", "bf16_dense", "bf16_interleaved"]


@pytest.mark.parametrize("kind", KINDS)
def test_mf_hot_row_keys(kind):
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    check_steps(kind, cfg, [wl.hot_row_batch(HOT_COUNTS, N_PLAIN, step) for step in range(2)])


@pytest.mark.parametrize("kind", ["dense", "rowwise_padded", "bf16_interleaved"])
def test_mf_hot_row_keys_two_phase(kind):
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    check_steps(kind, cfg, [wl.hot_row_batch(HOT_COUNTS, N_PLAIN, step) for step in range(2)], two_phase=True)


@pytest.mark.parametrize("kind", ["dense", "interleaved", "rowwise_padded", "bf16_interleaved"])
def test_mf_zipf_rows(kind):
    """Rows Zipf 1.1 (heavy users) over 20,000 rows, 50,000 entries per batch:
    the hottest rows hold several thousand entries."""
    cfg = replace(small_variant(MF_10Mx1M), name="mf_small_zipf_rows", row_zipf_s=1.1, batch=50_000,
                  nnz=150_000)
    wl = MFWorkload(cfg)
    check_steps(kind, cfg, [wl.batch(step) for step in range(3)])


def test_mf_hot_row_keys_paper_scale():
    """The 10M x 1M table on the bench's interleaved layout, one batch of
    1,048,576 entries in which six row keys repeat 33 ... 130,000 times."""
    cfg = MF_10Mx1M
    wl = MFWorkload(cfg)
    counts = HOT_COUNTS + [130_000]
    bt = wl.hot_row_batch(counts, cfg.batch - int(np.sum(counts)))
    say("generating the 11M x 100 table")
    W = wl.init_table()
    Wt, Gt = interleaved_tables(dev(W))
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    say("gpu step")
    loss = s.step_mf(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)
    assert s.error() == 0
    G = np.zeros_like(W)
    say("oracle step")
    rloss, bad = oracle.step_mf(W, G, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam, cfg.opt.lr, cfg.opt.eps)
    assert bad == 0
    say("compare")
    assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    assert_close_tables(Wt.cpu().numpy(), W, "W")
    assert_close_tables(Gt.cpu().numpy(), G, "G")

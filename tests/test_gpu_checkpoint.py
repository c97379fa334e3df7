"""Checkpoint and resume: a run that stops after step k, saves its tables
(values, accumulators, and the Wide & Deep dense buffers) to a file,
reloads them into fresh device memory under a new store and continues,
ends bit for bit where the uninterrupted run ends.  The store keeps no
training state besides the tables it borrows."""
from dataclasses import replace

import numpy as np
import pytest
import torch

from paper_2206_00470_amd import StagedStore, Store
from paper_2206_00470_amd.store import interleaved_bf16_tables, interleaved_tables, padded_rowwise_table
from paper_2206_00470_amd.workloads import (CTR_33M, CTR_33M_WD, KGE_COMPLEX, MF_10Mx1M, SGNS_1M, CTRWorkload,
                                            KGEWorkload, MFWorkload, SGNSWorkload, small_variant)
from tests.helpers import assert_bitwise, say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def mf_step(s, cfg, bt, extra):
    return s.step_mf(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)


def kge_step(s, cfg, bt, extra):
    return s.step_kge(dev(bt.head), dev(bt.rel), dev(bt.tail), dev(bt.neg), cfg.n_head_neg, cfg.n_ent)


def sgns_step(s, cfg, bt, extra):
    return s.step_sgns(dev(bt.centre), dev(bt.ctx), dev(bt.neg), cfg.window, cfg.vocab)


def ctr_step(s, cfg, bt, extra):
    return s.step_ctr(dev(bt.keys), dev(bt.label))


def wd_step(s, cfg, bt, extra):
    D, A = extra
    return s.step_ctr_wd(dev(bt.keys), dev(bt.label), D, A, cfg.emb_dim, cfg.deep)


CASES = {
    "mf_dense": (small_variant(MF_10Mx1M), MFWorkload, mf_step, "dense"),
    "mf_interleaved": (small_variant(MF_10Mx1M), MFWorkload, mf_step, "interleaved"),
    "mf_rowwise": (small_variant(MF_10Mx1M), MFWorkload, mf_step, "rowwise"),
    "mf_bf16": (small_variant(MF_10Mx1M), MFWorkload, mf_step, "bf16"),
    "kge": (small_variant(KGE_COMPLEX), KGEWorkload, kge_step, "interleaved"),
    "sgns": (small_variant(SGNS_1M), SGNSWorkload, sgns_step, "interleaved"),
    "ctr": (small_variant(CTR_33M), CTRWorkload, ctr_step, "interleaved"),
    "ctr_widedeep": (replace(small_variant(CTR_33M_WD), deep=(64, 32)), CTRWorkload, wd_step, "dense"),
}


def make(layout, W, G=None):
    """Device tables of a layout from host arrays; returns (W, G) tensors."""
    if layout == "dense":
        return dev(W), dev(np.zeros_like(W) if G is None else G)
    if layout == "interleaved":
        return interleaved_tables(dev(W), None if G is None else dev(G))
    if layout == "rowwise":
        return padded_rowwise_table(dev(W), None if G is None else dev(G))
    if layout == "bf16":
        Wb = W if W.dtype == np.uint16 else None
        if Wb is None:
            return interleaved_bf16_tables(dev(W), None if G is None else dev(G))
        Wt, Gt = interleaved_bf16_tables(torch.zeros(W.shape, device="cuda"), None if G is None else dev(G))
        Wt.view(torch.int16).copy_(torch.from_numpy(Wb.view(np.int16)).cuda())
        return Wt, Gt
    raise ValueError(layout)


def host(layout, Wt, Gt):
    W = Wt.contiguous().view(torch.int16).cpu().numpy().view(np.uint16) if layout == "bf16" else Wt.cpu().numpy()
    return W, Gt.cpu().numpy()


@pytest.mark.parametrize("case", list(CASES))
def test_checkpoint_resume_is_bit_exact(case, tmp_path):
    cfg, WL, step, layout = CASES[case]
    wl = WL(cfg)
    W0 = wl.init_table()
    dense0 = wl.init_dense() if case == "ctr_widedeep" else None
    extra = lambda: (dev(dense0), torch.zeros(dense0.shape, dtype=torch.float32, device="cuda")) if dense0 is not None else None
    k, total = 2, 5
    # the uninterrupted run
    Wa, Ga = make(layout, W0)
    xa = extra()
    a = Store(Wa, Ga, cfg.opt.lr, cfg.opt.eps)
    for i in range(total):
        step(a, cfg, wl.batch(i), xa)
    assert a.error() == 0
    # the interrupted run: k steps, save, drop everything, reload, continue
    Wb, Gb = make(layout, W0)
    xb = extra()
    b = Store(Wb, Gb, cfg.opt.lr, cfg.opt.eps)
    for i in range(k):
        step(b, cfg, wl.batch(i), xb)
    assert b.error() == 0
    Wh, Gh = host(layout, Wb, Gb)
    ck = {"W": Wh, "G": Gh}
    if xb is not None:
        ck["dense"], ck["dense_acc"] = xb[0].cpu().numpy(), xb[1].cpu().numpy()
    path = tmp_path / "ck.npz"
    np.savez(path, **ck)
    b.close()
    del b, Wb, Gb, xb
    torch.cuda.synchronize()
    say(f"{case}: checkpoint after step {k} ({path.stat().st_size / 1e6:.1f} MB), resuming")
    ld = np.load(path)
    Wc, Gc = make(layout, ld["W"], ld["G"])
    xc = (dev(ld["dense"]), dev(ld["dense_acc"])) if "dense" in ld else None
    c = Store(Wc, Gc, cfg.opt.lr, cfg.opt.eps)
    for i in range(k, total):
        step(c, cfg, wl.batch(i), xc)
    assert c.error() == 0
    Wf, Gf = host(layout, Wc, Gc)
    Wr, Gr = host(layout, Wa, Ga)
    assert_bitwise(Wf, Wr, "W after resuming")
    assert_bitwise(Gf, Gr, "G after resuming")
    if xc is not None:
        assert_bitwise(xc[0].cpu().numpy(), xa[0].cpu().numpy(), "dense parameters after resuming")
        assert_bitwise(xc[1].cpu().numpy(), xa[1].cpu().numpy(), "dense accumulators after resuming")


def test_staged_checkpoint_resume_is_bit_exact(tmp_path):
    """A staged store (home tables in pinned host memory): flush, save the
    home tables, rebuild a staged store from them with fresh intents, and
    continue; the flushed home tables end bit for bit as the uninterrupted
    run's."""
    cfg = small_variant(CTR_33M)
    wl = CTRWorkload(cfg)
    W0 = wl.init_table()
    keys = [np.unique(wl.batch(i).keys) for i in range(6)]

    def run(store, first, count):
        for c in range(first + 1, first + 3):
            store.intent(keys[c - 1], c, c + 1)
        for i in range(first, first + count):
            store.advance_clock()
            ctr_step(store, cfg, wl.batch(i), None)
            if i + 3 <= len(keys):
                store.intent(keys[i + 2], i + 3, i + 4)
            store.round(wait=True)
        store.flush()
        assert store.error() == 0
        return store.home_tables()

    full = run(StagedStore(W0, [0], [16_384], cfg.opt.lr, cfg.opt.eps), 0, 5)
    first = StagedStore(W0, [0], [16_384], cfg.opt.lr, cfg.opt.eps)
    Wh, Gh = (np.array(t, copy=True) for t in run(first, 0, 2))
    first.close()
    np.savez(tmp_path / "home.npz", W=Wh, G=Gh)
    ld = np.load(tmp_path / "home.npz")
    again = StagedStore(ld["W"], [0], [16_384], cfg.opt.lr, cfg.opt.eps, G0=ld["G"])
    # the clock restarts at 0 in the new store: batches 2.. are its clocks 1..
    def run_from(store, first, count):
        for c in range(1, 3):
            store.intent(keys[first + c - 1], c, c + 1)
        for j in range(count):
            store.advance_clock()
            ctr_step(store, cfg, wl.batch(first + j), None)
            if first + j + 3 <= len(keys):
                store.intent(keys[first + j + 2], j + 3, j + 4)
            store.round(wait=True)
        store.flush()
        assert store.error() == 0
        return store.home_tables()
    resumed = run_from(again, 2, 3)
    assert_bitwise(np.array(resumed[0]), np.array(full[0]), "home values after resuming")
    assert_bitwise(np.array(resumed[1]), np.array(full[1]), "home accumulators after resuming")

"""GPU parity of the Wide & Deep CTR step (fp64 MLP on the matrix cores,
sparse push of the embedding and wide-weight rows, dense AdaGrad) against
oracle/widedeep.py, every step from the same pre-step state."""
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle.widedeep import step_ctr_wd
from paper_2206_00470_amd import Store
from paper_2206_00470_amd.workloads import CTR_33M_WD, CTRWorkload, small_variant
from tests.helpers import assert_bitwise, assert_close_tables, mismatch_fraction, say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_wd(cfg, steps, W=None, dense=None):
    wl = CTRWorkload(cfg)
    W = wl.init_table() if W is None else W
    dense = wl.init_dense() if dense is None else dense
    Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
    Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    for step in steps:
        say(f"{cfg.name} step {step}: B={cfg.batch} F={cfg.n_fields} E={cfg.emb_dim} hidden={cfg.deep}")
        bt = wl.batch(step)
        Wr, Gr, Dr, Ar = Wt.cpu().numpy(), Gt.cpu().numpy(), Dt.cpu().numpy(), At.cpu().numpy()
        loss = s.step_ctr_wd(dev(bt.keys), dev(bt.label), Dt, At, cfg.emb_dim, cfg.deep)
        assert s.error() == 0
        rloss, bad = step_ctr_wd(Wr, Gr, Dr, Ar, bt.keys, bt.label, cfg.emb_dim, cfg.deep, cfg.opt.lr, cfg.opt.eps)
        assert bad == 0
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        Wg, Gg, Dg, Ag = Wt.cpu().numpy(), Gt.cpu().numpy(), Dt.cpu().numpy(), At.cpu().numpy()
        assert_close_tables(Wg, Wr, f"W after step {step}")
        assert_close_tables(Gg, Gr, f"G after step {step}")
        assert_close_tables(Dg, Dr, f"dense parameters after step {step}")
        assert_close_tables(Ag, Ar, f"dense accumulators after step {step}")
        assert_bitwise(Wg[:, cfg.emb_dim + 1:], W[:, cfg.emb_dim + 1:], "row padding")
        say(f"  loss {rloss:.6g}; dense words differing from the oracle: {mismatch_fraction(Dg, Dr):.2e}")
    return s, Wt, Dt


SMALL = small_variant(CTR_33M_WD)
# ragged everywhere: 97 samples, 5 fields of 12, hidden 37 and 20 (no dimension a multiple of a tile)
ODD = replace(SMALL, name="widedeep_odd", table_rows=500, dim=16, emb_dim=12, n_fields=5, deep=(37, 20), batch=97,
              vocab_max=500)


@pytest.mark.parametrize("cfg", [ODD, replace(ODD, deep=()), replace(ODD, deep=(70,)), replace(ODD, dim=15, emb_dim=13)],
                         ids=["two_hidden", "no_hidden", "one_hidden", "odd_row"])
def test_wd_small_shapes(cfg):
    run_wd(cfg, range(3))


def test_wd_paper_mlp_small_batch():
    """Three hidden layers of 1024 over 26 fields of 64; 301 samples."""
    run_wd(SMALL, range(2))


def test_wd_invalid_samples_are_skipped_and_flagged():
    cfg = ODD
    wl = CTRWorkload(cfg)
    W, dense = wl.init_table(), wl.init_dense()
    bt = wl.batch(0)
    bt.keys[3, 2] = cfg.num_keys
    bt.keys[40, 0] = -1
    Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
    Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    loss = s.step_ctr_wd(dev(bt.keys), dev(bt.label), Dt, At, cfg.emb_dim, cfg.deep)
    assert s.error() == -2
    Wr, Gr, Dr, Ar = W.copy(), np.zeros_like(W), dense.copy(), np.zeros_like(dense)
    rloss, bad = step_ctr_wd(Wr, Gr, Dr, Ar, bt.keys, bt.label, cfg.emb_dim, cfg.deep, cfg.opt.lr, cfg.opt.eps)
    assert bad == 2
    assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")
    assert_close_tables(Dt.cpu().numpy(), Dr, "dense parameters")


def test_wd_deterministic():
    cfg = SMALL
    wl = CTRWorkload(cfg)
    W, dense = wl.init_table(), wl.init_dense()
    out = []
    for _ in range(2):
        Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
        Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
        s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
        bt = wl.batch(0)
        l = s.step_ctr_wd(dev(bt.keys), dev(bt.label), Dt, At, cfg.emb_dim, cfg.deep)
        out.append((Wt.cpu().numpy(), Dt.cpu().numpy(), At.cpu().numpy(), float(l.item())))
    assert_bitwise(out[0][0], out[1][0], "W")
    assert_bitwise(out[0][1], out[1][1], "dense")
    assert_bitwise(out[0][2], out[1][2], "dense accumulators")
    assert out[0][3] == out[1][3]


def test_wd_paper_scale_one_step():
    """2^25 rows of 68, 8,192 samples of 26 fields, hidden 1024 x 3: the bench's launch."""
    cfg = CTR_33M_WD
    wl = CTRWorkload(cfg)
    say("generating the 2^25 x 68 table")
    W, dense = wl.init_table(), wl.init_dense()
    Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
    Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    bt = wl.batch(0)
    say("gpu step")
    loss = s.step_ctr_wd(dev(bt.keys), dev(bt.label), Dt, At, cfg.emb_dim, cfg.deep)
    assert s.error() == 0
    say("oracle step")
    G, A = np.zeros_like(W), np.zeros_like(dense)
    rloss, bad = step_ctr_wd(W, G, dense, A, bt.keys, bt.label, cfg.emb_dim, cfg.deep, cfg.opt.lr, cfg.opt.eps)
    say("compare")
    assert bad == 0
    assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    assert_close_tables(Wt.cpu().numpy(), W, "W")
    assert_close_tables(Gt.cpu().numpy(), G, "G")
    assert_close_tables(Dt.cpu().numpy(), dense, "dense parameters")
    assert_close_tables(At.cpu().numpy(), A, "dense accumulators")


def test_wd_on_a_staged_store():
    """Home table in pinned host memory, slots for the batch's keys: the
    same step as on an in-HBM store (the keys are translated to slots)."""
    from paper_2206_00470_amd import StagedStore
    cfg = ODD
    wl = CTRWorkload(cfg)
    W, dense = wl.init_table(), wl.init_dense()
    s = StagedStore(W, [0], [400], cfg.opt.lr, cfg.opt.eps)
    Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
    Dr, Ar = dense.copy(), np.zeros_like(dense)
    Wr, Gr = W.copy(), np.zeros_like(W)
    for step in range(3):
        bt = wl.batch(step)
        s.intent(bt.keys.ravel(), step + 1, step + 2)
        s.round()
        s.advance_clock()
        loss = s.step_ctr_wd(dev(bt.keys), dev(bt.label), Dt, At, cfg.emb_dim, cfg.deep)
        assert s.error() == 0
        rloss, _ = step_ctr_wd(Wr, Gr, Dr, Ar, bt.keys, bt.label, cfg.emb_dim, cfg.deep, cfg.opt.lr, cfg.opt.eps)
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
    s.flush()
    Wh, Gh = s.home_tables()
    assert_close_tables(Wh, Wr, "home W after three staged steps")
    assert_close_tables(Gh, Gr, "home G after three staged steps")
    assert_close_tables(Dt.cpu().numpy(), Dr, "dense parameters")


def test_wd_on_a_rowwise_store():
    """Row-wise AdaGrad for the table rows (one accumulator per key), per
    element for the dense buffer."""
    import oracle
    from oracle.widedeep import grad_ctr_wd
    cfg = ODD
    wl = CTRWorkload(cfg)
    W, dense = wl.init_table(), wl.init_dense()
    Wt, At_rows = dev(W), torch.zeros(W.shape[0], dtype=torch.float32, device="cuda")
    Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, At_rows, cfg.opt.lr, cfg.opt.eps)
    bt = wl.batch(0)
    s.step_ctr_wd(dev(bt.keys), dev(bt.label), Dt, At, cfg.emb_dim, cfg.deep)
    assert s.error() == 0
    okeys, grads, dflat, _, _ = grad_ctr_wd(W, dense, bt.keys, bt.label, cfg.emb_dim, cfg.deep)
    Wr, Ar = W.copy(), np.zeros(W.shape[0], np.float32)
    oracle.push_rowwise(Wr, Ar, okeys, grads, cfg.opt.lr, cfg.opt.eps)
    Dr, _ = oracle.adagrad_row(dense.copy(), np.zeros_like(dense), dflat.astype(np.float32), cfg.opt.lr, cfg.opt.eps)
    assert_close_tables(Wt.cpu().numpy(), Wr, "W")
    assert_close_tables(At_rows.cpu().numpy(), Ar, "row accumulators")
    assert_close_tables(Dt.cpu().numpy(), Dr, "dense parameters")


def test_wd_empty_batch_is_a_no_op():
    cfg = ODD
    wl = CTRWorkload(cfg)
    W, dense = wl.init_table(), wl.init_dense()
    Wt, Gt = dev(W), torch.zeros(W.shape, dtype=torch.float32, device="cuda")
    Dt, At = dev(dense), torch.zeros(dense.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    loss = s.step_ctr_wd(torch.zeros((0, cfg.n_fields), dtype=torch.int64, device="cuda"),
                         torch.zeros(0, dtype=torch.float32, device="cuda"), Dt, At, cfg.emb_dim, cfg.deep)
    assert s.error() == 0 and float(loss.item()) == 0.0
    assert_bitwise(Wt.cpu().numpy(), W, "W")
    assert_bitwise(Dt.cpu().numpy(), dense, "dense")

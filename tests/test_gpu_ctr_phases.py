"""The CTR step in two phases (ps_step_ctr_prepare: sample validity, key
sort and segments into a workspace; ps_step_ctr_apply: gradients, merge,
update and loss) against ps_step_ctr: bit for bit on one stream, bit for bit
when the next batch's key work runs on a second stream beside this batch's
update (two workspaces ordered by events), and bit for bit when that
pipelined loop is captured in a HIP graph and replayed; the one-stream form
is also checked against the oracle."""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import StagedStore, Store, _lib
from paper_2206_00470_amd._lib import PSError
from paper_2206_00470_amd.store import interleaved_tables, padded_rowwise_table
from paper_2206_00470_amd.workloads import CTR_33M, CTRWorkload, small_variant
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def twin_stores(W0, layout):
    """Two stores on equal copies of W0: dense fp32, interleaved or row-wise."""
    out = []
    for _ in range(2):
        if layout == "interleaved":
            W, G = interleaved_tables(dev(W0))
        elif layout == "rowwise":
            W, G = padded_rowwise_table(dev(W0))
        else:
            W, G = dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda")
        out.append((W, G))
    return out


def new_pipe():
    """The side stream and the events of ctr_pipeline (made outside any capture)."""
    return torch.cuda.Stream(), [torch.cuda.Event(), torch.cuda.Event()], [torch.cuda.Event(), torch.cuda.Event()]


def ctr_pipeline(s, batches, ws, loss_out, pipe):
    """ps_step_ctr_prepare of batch i+1 on a side stream beside
    ps_step_ctr_apply of batch i on the current stream; batches are
    (keys, label) device pairs; the loss of step i goes to loss_out[i]."""
    main = torch.cuda.current_stream()
    side, prepared, applied = pipe
    F = batches[0][0].numel() // batches[0][1].numel()
    side.wait_stream(main)
    s.step_ctr_prepare(batches[0][0], F, ws[0], stream=side)
    prepared[0].record(side)
    for i, (k, y) in enumerate(batches):
        main.wait_event(prepared[i % 2])
        s.step_ctr_apply(k, y, ws[i % 2], loss=loss_out[i], stream=main)
        applied[i % 2].record(main)
        if i + 1 < len(batches):
            if i >= 1:
                side.wait_event(applied[(i + 1) % 2])   # the apply that last used that workspace
            s.step_ctr_prepare(batches[i + 1][0], F, ws[(i + 1) % 2], stream=side)
            prepared[(i + 1) % 2].record(side)


SHAPES = [(64, 26, "dense"), (7, 26, "dense"), (100, 17, "interleaved"), (16, 33, "rowwise"), (12, 65, "dense"),
          (256, 1, "dense")]


@pytest.mark.parametrize("dim,F,layout", SHAPES)
def test_prepare_then_apply_is_step_ctr(dim, F, layout):
    cfg = replace(small_variant(CTR_33M), dim=dim, n_fields=F)
    wl = CTRWorkload(cfg)
    W0 = wl.init_table()
    (WA, GA), (WB, GB) = twin_stores(W0, layout)
    A, B = Store(WA, GA, cfg.opt.lr, cfg.opt.eps), Store(WB, GB, cfg.opt.lr, cfg.opt.eps)
    ws = B.ctr_workspace(cfg.batch, F)
    for step in range(3):
        bt = wl.batch(step)
        keys = bt.keys.copy()
        if step == 1:
            keys[5, F // 2] = cfg.num_keys + 7          # sample 5 is skipped and flagged by both
        Wr, Gr = WA.cpu().numpy(), GA.cpu().numpy()
        la = A.step_ctr(dev(keys), dev(bt.label))
        kd, yd = dev(keys), dev(bt.label)
        B.step_ctr_prepare(kd, F, ws)
        lb = B.step_ctr_apply(kd, yd, ws)
        expect = _lib.PS_ERR_KEY_RANGE if step == 1 else 0
        assert A.error() == expect and B.error() == expect
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after step {step}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after step {step}")
        assert lb.item() == la.item()
        if layout == "dense":
            rloss, bad = oracle.step_ctr(Wr, Gr, keys, bt.label, cfg.opt.lr, cfg.opt.eps)
            assert bad == (1 if step == 1 else 0)
            assert_close_tables(WB.cpu().numpy(), Wr, f"W against the oracle, step {step}")
            assert_close_tables(GB.cpu().numpy(), Gr, f"G against the oracle, step {step}")
            assert lb.item() == pytest.approx(rloss, rel=1e-9)
        say(f"dim {dim} F {F} {layout} step {step}: loss {lb.item():.6g}")


@pytest.mark.parametrize("full", [False, True], ids=["small", "paper_scale"])
def test_overlapped_ctr_steps_equal_sequential_steps(full):
    """Five steps (three at full size: 2^25 keys of 64 floats, 8,192 samples
    of 26 fields, hot keys with segments long enough to be cut and folded)."""
    cfg = CTR_33M if full else small_variant(CTR_33M)
    wl = CTRWorkload(cfg)
    W0 = wl.init_table()
    (WA, GA), (WB, GB) = twin_stores(W0, "dense")
    del W0
    A, B = Store(WA, GA, cfg.opt.lr, cfg.opt.eps), Store(WB, GB, cfg.opt.lr, cfg.opt.eps)
    steps = 3 if full else 5
    batches = [(dev(bt.keys), dev(bt.label)) for bt in (wl.batch(i) for i in range(steps))]
    la = [A.step_ctr(k, y).clone() for k, y in batches]
    F = cfg.n_fields
    ws = [B.ctr_workspace(cfg.batch, F), B.ctr_workspace(cfg.batch, F)]
    lb = [torch.empty(1, dtype=torch.float64, device="cuda") for _ in batches]
    ctr_pipeline(B, batches, ws, lb, new_pipe())
    torch.cuda.synchronize()
    assert A.error() == 0 and B.error() == 0
    say(f"{cfg.name}: {steps} steps overlapped")
    assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), "W")
    assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), "G")
    for i in range(steps):
        assert lb[i].item() == la[i].item(), i


def test_overlapped_ctr_steps_graph_replays_match_eager():
    """The pipelined loop over three resident batches captured once; each
    replay follows eager work (three ps_step_ctr calls on the twin store, a
    synchronisation) and must leave both stores equal bit for bit."""
    cfg = small_variant(CTR_33M)
    wl = CTRWorkload(cfg)
    W0 = wl.init_table()
    (WA, GA), (WB, GB) = twin_stores(W0, "dense")
    A, B = Store(WA, GA, cfg.opt.lr, cfg.opt.eps), Store(WB, GB, cfg.opt.lr, cfg.opt.eps)
    batches = [(dev(bt.keys), dev(bt.label)) for bt in (wl.batch(i) for i in range(3))]
    ws = [B.ctr_workspace(cfg.batch, cfg.n_fields), B.ctr_workspace(cfg.batch, cfg.n_fields)]
    lb = [torch.empty(1, dtype=torch.float64, device="cuda") for _ in batches]
    # one eager pass on both (also sizes every workspace before the capture)
    pipe = new_pipe()
    for k, y in batches:
        A.step_ctr(k, y)
    ctr_pipeline(B, batches, ws, lb, pipe)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ctr_pipeline(B, batches, ws, lb, pipe)
    for r in range(3):
        la = [A.step_ctr(k, y).clone() for k, y in batches]
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert A.error() == 0 and B.error() == 0
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after replay {r}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after replay {r}")
        for i in range(3):
            assert lb[i].item() == la[i].item(), (r, i)
        say(f"replay {r}: equal")


def test_two_phase_ctr_argument_checks():
    K, d, Bn, F = 100, 8, 10, 3
    W, G = torch.zeros((K, d), device="cuda"), torch.zeros((K, d), device="cuda")
    s = Store(W, G, 0.1, 1e-10)
    keys = torch.arange(Bn * F, dtype=torch.int64, device="cuda")
    label = torch.ones(Bn, dtype=torch.float32, device="cuda")
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(PSError) as e:
        s.step_ctr_prepare(keys, F, small)
    assert e.value.status == _lib.PS_ERR_WORKSPACE
    with pytest.raises(PSError) as e:
        s.step_ctr_apply(keys, label, small)
    assert e.value.status == _lib.PS_ERR_WORKSPACE
    ws = s.ctr_workspace(Bn, F)
    with pytest.raises(PSError) as e:
        s.step_ctr_prepare(keys, 0, ws)
    assert e.value.status == _lib.PS_ERR_INVALID
    s.step_ctr_prepare(keys[:0], F, ws)                  # empty: no-ops, the loss is zeroed
    loss = torch.full((1,), 5.0, dtype=torch.float64, device="cuda")
    s.step_ctr_apply(keys[:0], label[:0], ws, loss=loss)
    assert loss.item() == 0.0
    assert s.error() == 0
    assert not W.cpu().numpy().any()
    staged = StagedStore(np.zeros((K, d), dtype=np.float32), [0], [16], 0.1, 1e-10)
    try:
        with pytest.raises(PSError) as e:
            staged.step_ctr_prepare(keys, F, ws)
        assert e.value.status == _lib.PS_ERR_UNSUPPORTED
        with pytest.raises(PSError) as e:
            staged.step_ctr_apply(keys, label, ws)
        assert e.value.status == _lib.PS_ERR_UNSUPPORTED
    finally:
        staged.close()

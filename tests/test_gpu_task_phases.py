"""The ComplEx and skip-gram steps in two phases (prepare: unit validity,
key sort and segments into a workspace; apply: gradients, merges, update and
loss) against the one-call steps: bit for bit on one stream, bit for bit when
the next batch's key work runs on a second stream beside this batch's update
(two workspaces ordered by events), and bit for bit when that pipelined loop
is captured in a HIP graph and replayed; the one-stream form is also checked
against the oracle."""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import StagedStore, Store, _lib
from paper_2206_00470_amd._lib import PSError
from paper_2206_00470_amd.store import interleaved_tables
from paper_2206_00470_amd.workloads import (KGE_COMPLEX, SGNS_1M, SGNS_1M_W2V, KGEWorkload, SGNSWorkload,
                                            small_variant)
from tests.helpers import assert_bitwise, assert_close_tables, say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


class KGE:
    WL = KGEWorkload

    @staticmethod
    def to_dev(bt):
        return [dev(bt.head), dev(bt.rel), dev(bt.tail), dev(bt.neg)]

    @staticmethod
    def one_call(s, cfg, x, loss=None):
        return s.step_kge(*x, cfg.n_head_neg, cfg.n_ent, loss=loss)

    @staticmethod
    def workspace(s, cfg, x):
        return s.kge_workspace(x[0].numel(), x[3].numel() // x[0].numel())

    @staticmethod
    def prepare(s, cfg, x, ws, stream=None):
        s.step_kge_prepare(*x, cfg.n_ent, ws, stream=stream)

    @staticmethod
    def apply(s, cfg, x, ws, loss=None, stream=None):
        return s.step_kge_apply(*x, cfg.n_head_neg, cfg.n_ent, ws, loss=loss, stream=stream)

    @staticmethod
    def oracle(W, G, cfg, bt):
        return oracle.step_kge(W, G, bt.head, bt.rel, bt.tail, bt.neg, cfg.n_head_neg, cfg.n_ent, cfg.opt.lr,
                               cfg.opt.eps)

    @staticmethod
    def spoil(bt, cfg):
        bt.rel[3] = -1                           # triple 3 is skipped and flagged


class SGNS:
    WL = SGNSWorkload

    @staticmethod
    def to_dev(bt):
        return [dev(bt.centre), dev(bt.ctx), dev(bt.neg)]

    @staticmethod
    def one_call(s, cfg, x, loss=None):
        return s.step_sgns(*x, cfg.window, cfg.vocab, loss=loss)

    @staticmethod
    def workspace(s, cfg, x):
        return s.sgns_workspace(x[0].numel(), cfg.window, cfg.n_neg)

    @staticmethod
    def prepare(s, cfg, x, ws, stream=None):
        s.step_sgns_prepare(*x, cfg.window, cfg.vocab, ws, stream=stream)

    @staticmethod
    def apply(s, cfg, x, ws, loss=None, stream=None):
        return s.step_sgns_apply(*x, cfg.window, cfg.vocab, ws, loss=loss, stream=stream)

    @staticmethod
    def oracle(W, G, cfg, bt):
        return oracle.step_sgns(W, G, bt.centre, bt.ctx, bt.neg, cfg.window, cfg.vocab, cfg.opt.lr, cfg.opt.eps)

    @staticmethod
    def spoil(bt, cfg):
        bt.centre[4] = cfg.vocab + 1             # a centre id in the output table: skipped and flagged


def stores(cfg, W0, interleaved):
    out = []
    for _ in range(2):
        W, G = interleaved_tables(dev(W0)) if interleaved else (dev(W0), torch.zeros(W0.shape, device="cuda"))
        out.append((W, G, Store(W, G, cfg.opt.lr, cfg.opt.eps)))
    return out


def pipeline(T, s, cfg, batches, ws, losses, pipe):
    """prepare of batch i+1 on a side stream beside apply of batch i on the current stream."""
    main = torch.cuda.current_stream()
    side, prepared, applied = pipe
    side.wait_stream(main)
    T.prepare(s, cfg, batches[0], ws[0], stream=side)
    prepared[0].record(side)
    for i, x in enumerate(batches):
        main.wait_event(prepared[i % 2])
        T.apply(s, cfg, x, ws[i % 2], loss=losses[i], stream=main)
        applied[i % 2].record(main)
        if i + 1 < len(batches):
            if i >= 1:
                side.wait_event(applied[(i + 1) % 2])   # the apply that last used that workspace
            T.prepare(s, cfg, batches[i + 1], ws[(i + 1) % 2], stream=side)
            prepared[(i + 1) % 2].record(side)


def new_pipe():
    return torch.cuda.Stream(), [torch.cuda.Event(), torch.cuda.Event()], [torch.cuda.Event(), torch.cuda.Event()]


ONE_STREAM = [("kge", KGE, small_variant(KGE_COMPLEX), False),
              ("kge_cdim3_interleaved", KGE, replace(small_variant(KGE_COMPLEX), cdim=3, n_neg=7, n_head_neg=3,
                                                     batch=61), True),
              ("kge_no_negatives", KGE, replace(small_variant(KGE_COMPLEX), n_neg=0, n_head_neg=0), False),
              ("sgns", SGNS, small_variant(SGNS_1M), False),
              ("sgns_w2v_interleaved", SGNS, small_variant(SGNS_1M_W2V), True),
              ("sgns_dim3", SGNS, replace(small_variant(SGNS_1M), dim=3, batch=130), False)]


@pytest.mark.parametrize("name,T,cfg,interleaved", ONE_STREAM, ids=[c[0] for c in ONE_STREAM])
def test_prepare_then_apply_is_one_call(name, T, cfg, interleaved):
    wl = T.WL(cfg)
    W0 = wl.init_table()
    (WA, GA, A), (WB, GB, B) = stores(cfg, W0, interleaved)
    for step in range(3):
        bt = wl.batch(step)
        if step == 1:
            T.spoil(bt, cfg)
        Wr, Gr = WA.cpu().numpy(), GA.cpu().numpy()
        x = T.to_dev(bt)
        la = T.one_call(A, cfg, x)
        ws = T.workspace(B, cfg, x)                # word2vec batches differ in size
        T.prepare(B, cfg, x, ws)
        lb = T.apply(B, cfg, x, ws)
        expect = _lib.PS_ERR_KEY_RANGE if step == 1 else 0
        assert A.error() == expect and B.error() == expect
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after step {step}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after step {step}")
        assert lb.item() == la.item()
        if not interleaved:
            rloss, bad = T.oracle(Wr, Gr, cfg, bt)
            assert bad == (1 if step == 1 else 0)
            assert_close_tables(WB.cpu().numpy(), Wr, f"W against the oracle, step {step}")
            assert_close_tables(GB.cpu().numpy(), Gr, f"G against the oracle, step {step}")
            assert lb.item() == pytest.approx(rloss, rel=1e-9)
        say(f"{name} step {step}: loss {lb.item():.6g}")


OVERLAPPED = [("kge_small", KGE, small_variant(KGE_COMPLEX), 5), ("kge_paper_scale", KGE, KGE_COMPLEX, 3),
              ("sgns_small", SGNS, small_variant(SGNS_1M), 5), ("sgns_paper_scale", SGNS, SGNS_1M, 2)]


@pytest.mark.parametrize("name,T,cfg,steps", OVERLAPPED, ids=[c[0] for c in OVERLAPPED])
def test_overlapped_steps_equal_one_call_steps(name, T, cfg, steps):
    wl = T.WL(cfg)
    W0 = wl.init_table()
    (WA, GA, A), (WB, GB, B) = stores(cfg, W0, False)
    del W0
    batches = [T.to_dev(wl.batch(i)) for i in range(steps)]
    la = [T.one_call(A, cfg, x).clone() for x in batches]
    n = max(x[0].numel() for x in batches)
    big = max(batches, key=lambda x: x[0].numel())
    assert all(x[0].numel() == n for x in batches)
    ws = [T.workspace(B, cfg, big), T.workspace(B, cfg, big)]
    lb = [torch.empty(1, dtype=torch.float64, device="cuda") for _ in batches]
    pipeline(T, B, cfg, batches, ws, lb, new_pipe())
    torch.cuda.synchronize()
    assert A.error() == 0 and B.error() == 0
    say(f"{name}: {steps} steps overlapped")
    assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), "W")
    assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), "G")
    for i in range(steps):
        assert lb[i].item() == la[i].item(), i


@pytest.mark.parametrize("name,T,cfg", [("kge", KGE, small_variant(KGE_COMPLEX)),
                                        ("sgns", SGNS, small_variant(SGNS_1M))], ids=["kge", "sgns"])
def test_overlapped_steps_graph_replays_match_eager(name, T, cfg):
    """The pipelined loop over three resident batches captured once; each
    replay follows eager one-call steps on the twin store and a
    synchronisation, and must leave both stores equal bit for bit."""
    wl = T.WL(cfg)
    W0 = wl.init_table()
    (WA, GA, A), (WB, GB, B) = stores(cfg, W0, False)
    batches = [T.to_dev(wl.batch(i)) for i in range(3)]
    ws = [T.workspace(B, cfg, batches[0]), T.workspace(B, cfg, batches[0])]
    lb = [torch.empty(1, dtype=torch.float64, device="cuda") for _ in batches]
    pipe = new_pipe()
    for x in batches:
        T.one_call(A, cfg, x)
    pipeline(T, B, cfg, batches, ws, lb, pipe)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pipeline(T, B, cfg, batches, ws, lb, pipe)
    for r in range(3):
        la = [T.one_call(A, cfg, x).clone() for x in batches]
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert A.error() == 0 and B.error() == 0
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after replay {r}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after replay {r}")
        for i in range(3):
            assert lb[i].item() == la[i].item(), (r, i)
        say(f"{name} replay {r}: equal")


def test_two_phase_argument_checks():
    K, d = 200, 8
    W, G = torch.zeros((K, d), device="cuda"), torch.zeros((K, d), device="cuda")
    s = Store(W, G, 0.1, 1e-10)
    i32 = lambda *v: torch.tensor(v, dtype=torch.int32, device="cuda")
    head, rel, tail, neg = i32(1, 2), i32(0, 1), i32(3, 4), i32(5, 6, 7, 8)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(PSError) as e:
        s.step_kge_prepare(head, rel, tail, neg, 100, small)
    assert e.value.status == _lib.PS_ERR_WORKSPACE
    ws = s.kge_workspace(2, 2)
    with pytest.raises(PSError) as e:
        s.step_kge_apply(head, rel, tail, neg, 3, 100, ws)          # n_head_neg > n_neg
    assert e.value.status == _lib.PS_ERR_INVALID
    with pytest.raises(PSError) as e:
        s.step_kge_prepare(head, rel, tail, neg, -1, ws)
    assert e.value.status == _lib.PS_ERR_INVALID
    centre, ctx, negs = i32(1, 2), i32(3, -1, 4, 5), i32(*range(10, 18))
    with pytest.raises(PSError) as e:
        s.step_sgns_prepare(centre, ctx, negs, 1, 100, small)
    assert e.value.status == _lib.PS_ERR_WORKSPACE
    wss = s.sgns_workspace(2, 1, 2)
    with pytest.raises(PSError) as e:
        s.step_sgns_apply(centre, ctx, negs, 1, 0, wss)               # no output table
    assert e.value.status == _lib.PS_ERR_INVALID
    loss = torch.full((1,), 5.0, dtype=torch.float64, device="cuda")
    s.step_kge_prepare(head[:0], rel[:0], tail[:0], neg[:0], 100, ws)   # empty: no-ops, the loss is zeroed
    s.step_kge_apply(head[:0], rel[:0], tail[:0], neg[:0], 0, 100, ws, loss=loss)
    assert loss.item() == 0.0
    loss.fill_(5.0)
    s.step_sgns_prepare(centre[:0], ctx[:0], negs[:0], 1, 100, wss)
    s.step_sgns_apply(centre[:0], ctx[:0], negs[:0], 1, 100, wss, loss=loss)
    assert loss.item() == 0.0
    assert s.error() == 0
    assert not W.cpu().numpy().any()
    staged = StagedStore(np.zeros((K, d), dtype=np.float32), [0, 100], [16, 16], 0.1, 1e-10)
    try:
        for call in (lambda: staged.step_kge_prepare(head, rel, tail, neg, 100, ws),
                     lambda: staged.step_kge_apply(head, rel, tail, neg, 1, 100, ws),
                     lambda: staged.step_sgns_prepare(centre, ctx, negs, 1, 100, wss),
                     lambda: staged.step_sgns_apply(centre, ctx, negs, 1, 100, wss)):
            with pytest.raises(PSError) as e:
                call()
            assert e.value.status == _lib.PS_ERR_UNSUPPORTED
    finally:
        staged.close()


def test_every_unit_invalid_leaves_tables_and_zero_loss():
    """A batch in which every unit holds an id out of range: no key reaches
    a segment, so the one-call and the two-phase steps both leave W and G
    bit-identical, report a zero loss and raise the sticky error (ComplEx,
    skip-gram and CTR; the oracle skips every unit too)."""
    from paper_2206_00470_amd.workloads import CTR_33M, CTRWorkload
    cases = []
    cfg = small_variant(KGE_COMPLEX)
    bt = KGEWorkload(cfg).batch(0)
    bt.rel[:] = -1
    cases.append((KGE, cfg, bt))
    cfg = small_variant(SGNS_1M)
    bt = SGNSWorkload(cfg).batch(0)
    bt.centre[:] = cfg.vocab                       # an output-table id as centre: invalid
    cases.append((SGNS, cfg, bt))
    for T, cfg, bt in cases:
        W0 = T.WL(cfg).init_table()
        (WA, GA, A), (WB, GB, B) = stores(cfg, W0, False)
        x = T.to_dev(bt)
        la = T.one_call(A, cfg, x)
        ws = T.workspace(B, cfg, x)
        T.prepare(B, cfg, x, ws)
        lb = T.apply(B, cfg, x, ws)
        assert A.error() == _lib.PS_ERR_KEY_RANGE and B.error() == _lib.PS_ERR_KEY_RANGE
        assert la.item() == 0.0 and lb.item() == 0.0
        for t in (WA, WB):
            assert_bitwise(t.cpu().numpy(), W0, "W")
        assert not GA.cpu().numpy().any() and not GB.cpu().numpy().any()
        rloss, bad = T.oracle(W0.copy(), np.zeros_like(W0), cfg, bt)
        assert bad == bt.centre.size if T is SGNS else bad == bt.head.size
        assert rloss == 0.0
    cfg = small_variant(CTR_33M)
    bt = CTRWorkload(cfg).batch(0)
    bt.keys[:, 0] = -1
    W0 = CTRWorkload(cfg).init_table()
    (WA, GA, A), (WB, GB, B) = stores(cfg, W0, False)
    k, y = dev(bt.keys), dev(bt.label)
    la = A.step_ctr(k, y)
    ws = B.ctr_workspace(cfg.batch, cfg.n_fields)
    B.step_ctr_prepare(k, cfg.n_fields, ws)
    lb = B.step_ctr_apply(k, y, ws)
    assert A.error() == _lib.PS_ERR_KEY_RANGE and B.error() == _lib.PS_ERR_KEY_RANGE
    assert la.item() == 0.0 and lb.item() == 0.0
    for t in (WA, WB):
        assert_bitwise(t.cpu().numpy(), W0, "W")
    assert not GA.cpu().numpy().any() and not GB.cpu().numpy().any()
    rloss, bad = oracle.step_ctr(W0.copy(), np.zeros_like(W0), bt.keys, bt.label, cfg.opt.lr, cfg.opt.eps)
    assert bad == cfg.batch and rloss == 0.0

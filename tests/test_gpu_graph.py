"""Steps captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

The step entry points enqueue kernels only (no allocation, no host
synchronisation, no memset nodes), so a caller can capture one and replay
it.  Each replay here follows eager work of the program (copying the next
batch into the captured input buffers, an eager step on a twin store, a
device synchronisation) and must match that eager step bit for bit: both
run the same deterministic kernels on the same state.
"""
import numpy as np
import pytest
import torch

from paper_2206_00470_amd import Store
from paper_2206_00470_amd.workloads import (CTR_33M, KGE_COMPLEX, MF_10Mx1M, MF_TINY, SGNS_1M, CTRWorkload,
                                            KGEWorkload, MFWorkload, SGNSWorkload, small_variant)
from tests.helpers import assert_bitwise, say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def mf_call(cfg):
    return lambda s, b, loss: s.step_mf(b["row"], b["col"], b["val"], cfg.n_rows, cfg.lam, loss=loss)


def kge_call(cfg):
    return lambda s, b, loss: s.step_kge(b["head"], b["rel"], b["tail"], b["neg"], cfg.n_head_neg, cfg.n_ent,
                                         loss=loss)


def sgns_call(cfg):
    return lambda s, b, loss: s.step_sgns(b["centre"], b["ctx"], b["neg"], cfg.window, cfg.vocab, loss=loss)


def ctr_call(cfg):
    return lambda s, b, loss: s.step_ctr(b["keys"], b["label"], loss=loss)


CASES = {
    "mf_tiny": (MF_TINY, MFWorkload, mf_call),
    "mf_small": (small_variant(MF_10Mx1M), MFWorkload, mf_call),
    "kge_small": (small_variant(KGE_COMPLEX), KGEWorkload, kge_call),
    "sgns_small": (small_variant(SGNS_1M), SGNSWorkload, sgns_call),
    "ctr_small": (small_variant(CTR_33M), CTRWorkload, ctr_call),
}


@pytest.mark.parametrize("name", list(CASES))
def test_step_graph_replays_match_eager(name):
    cfg, WL, make_call = CASES[name]
    call = make_call(cfg)
    wl = WL(cfg)
    W0 = wl.init_table()
    WA, GA = dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda")
    WB, GB = dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda")
    eager = Store(WA, GA, cfg.opt.lr, cfg.opt.eps)
    graphed = Store(WB, GB, cfg.opt.lr, cfg.opt.eps)
    lossA = torch.zeros(1, dtype=torch.float64, device="cuda")
    lossB = torch.zeros(1, dtype=torch.float64, device="cuda")

    def batch(step):
        return {k: dev(v) for k, v in wl.batch(step).__dict__.items()}

    # one eager step on both stores sizes their workspaces before the capture
    warm = batch(0)
    call(eager, warm, lossA)
    call(graphed, warm, lossB)
    static = batch(1)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(graphed, static, lossB)
    torch.cuda.synchronize()
    for step in range(1, 5):
        say(f"{name}: replay for step {step}")
        b = batch(step)
        assert all(b[k].shape == static[k].shape for k in b), "batches of one shape"
        for k in b:
            static[k].copy_(b[k])
        call(eager, b, lossA)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert graphed.error() == 0 and eager.error() == 0
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after replay {step}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after replay {step}")
        assert lossB.item() == lossA.item()


def graph_vs_eager(make_store, call, batch, snapshot, name):
    """Capture call(store_B, static batch) once; before each replay copy the
    next batch in, run the same step eagerly on store_A, and compare."""
    A, B = make_store(), make_store()
    lossA = torch.zeros(1, dtype=torch.float64, device="cuda")
    lossB = torch.zeros(1, dtype=torch.float64, device="cuda")
    warm = batch(0)
    call(A, warm, lossA)
    call(B, warm, lossB)
    static = batch(1)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(B, static, lossB)
    torch.cuda.synchronize()
    for step in range(1, 5):
        say(f"{name}: replay for step {step}")
        b = batch(step)
        for k in b:
            static[k].copy_(b[k])
        call(A, b, lossA)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert A[0].error() == 0 and B[0].error() == 0
        for i, (x, y) in enumerate(zip(snapshot(A), snapshot(B))):
            assert_bitwise(y, x, f"{name} state {i} after replay {step}")
        assert lossB.item() == lossA.item()


def test_widedeep_graph_replays_match_eager():
    from dataclasses import replace
    from paper_2206_00470_amd.workloads import CTR_33M_WD
    cfg = replace(small_variant(CTR_33M_WD), deep=(96, 40), emb_dim=12, dim=16, n_fields=7)
    wl = CTRWorkload(cfg)
    W0, D0 = wl.init_table(), wl.init_dense()

    def make():
        s = Store(dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda"), cfg.opt.lr, cfg.opt.eps)
        return (s, dev(D0), torch.zeros(D0.shape, dtype=torch.float32, device="cuda"))

    def call(st, b, loss):
        s, D, Acc = st
        s.step_ctr_wd(b["keys"], b["label"], D, Acc, cfg.emb_dim, cfg.deep, loss=loss)

    graph_vs_eager(make, call, lambda i: {k: dev(v) for k, v in wl.batch(i).__dict__.items()},
                   lambda st: (st[0].W.cpu().numpy(), st[0].G.cpu().numpy(), st[1].cpu().numpy(), st[2].cpu().numpy()),
                   "wide & deep")


@pytest.mark.parametrize("kind", ["rowwise", "bf16"])
def test_mf_variant_graph_replays_match_eager(kind):
    from paper_2206_00470_amd.store import interleaved_bf16_tables, padded_rowwise_table
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    W0 = torch.from_numpy(wl.init_table()).cuda()

    def make():
        if kind == "rowwise":
            W, A = padded_rowwise_table(W0)
        else:
            W, A = interleaved_bf16_tables(W0)
        return (Store(W, A, cfg.opt.lr, cfg.opt.eps),)

    def call(st, b, loss):
        st[0].step_mf(b["row"], b["col"], b["val"], cfg.n_rows, cfg.lam, loss=loss)

    def snap(st):
        W = st[0].W
        w = W.float().cpu().numpy() if W.dtype == torch.bfloat16 else W.cpu().numpy()
        return (w, st[0].G.cpu().numpy())

    graph_vs_eager(make, call, lambda i: {k: dev(v) for k, v in wl.batch(i).__dict__.items()}, snap, f"mf {kind}")


def test_mf_async_graph_replays_within_bounds():
    """The unmerged MF step captured once and replayed on new batches: each
    replay's result equals some order's result, so it is checked against the
    any-order bounds and the sum of squares from the state before it."""
    from tests.test_gpu_async import check_accumulators, check_bounds
    import oracle
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    W0 = wl.init_table()
    s = Store(dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda"), cfg.opt.lr, cfg.opt.eps)
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    b0 = {k: dev(v) for k, v in wl.batch(0).__dict__.items()}
    s.step_mf_async(b0["row"], b0["col"], b0["val"], cfg.n_rows, cfg.lam, loss=loss)
    static = {k: dev(v) for k, v in wl.batch(1).__dict__.items()}
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        s.step_mf_async(static["row"], static["col"], static["val"], cfg.n_rows, cfg.lam, loss=loss)
    torch.cuda.synchronize()
    for step in range(1, 5):
        say(f"unmerged mf: replay for step {step}")
        bt = wl.batch(step)
        for k, v in bt.__dict__.items():
            static[k].copy_(dev(v))
        Wb, Gb = s.W.cpu().numpy(), s.G.cpu().numpy()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert s.error() == 0
        keys, grads, rloss, _ = oracle.grad_mf(Wb, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam)
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        check_bounds(s.W.cpu().numpy(), Wb, Gb, keys, grads, lr=cfg.opt.lr, eps=cfg.opt.eps)
        check_accumulators(s.G.cpu().numpy(), Gb, keys, grads)


@pytest.mark.parametrize("cfg", [MF_TINY, small_variant(MF_10Mx1M)], ids=["mf_tiny", "mf_small"])
def test_mf_two_phase_pipeline_graph_replays_match_eager(cfg):
    """The MF two-phase loop over three resident batches (prepare of batch
    i+1 on a side stream after the row-key merge of batch i, ordered by the
    library's rows_done event and per-workspace events) captured once; each
    replay follows three eager ps_step_mf calls on the twin store and must
    leave both stores equal bit for bit."""
    wl = MFWorkload(cfg)
    W0 = wl.init_table()
    WA, GA = dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda")
    WB, GB = dev(W0), torch.zeros(W0.shape, dtype=torch.float32, device="cuda")
    A, B = Store(WA, GA, cfg.opt.lr, cfg.opt.eps), Store(WB, GB, cfg.opt.lr, cfg.opt.eps)
    batches = []
    for i in range(3):
        bt = wl.batch(i)
        batches.append((dev(bt.row), dev(bt.col), dev(bt.val)))
    nB = batches[0][0].numel()
    assert all(b[0].numel() == nB for b in batches)
    side = torch.cuda.Stream()
    ws = [B.mf_workspace(nB), B.mf_workspace(nB)]
    prepared = [torch.cuda.Event(), torch.cuda.Event()]
    applied = [torch.cuda.Event(), torch.cuda.Event()]
    rows_done = torch.cuda.Event()
    rows_done.record()
    losses = [torch.zeros(1, dtype=torch.float64, device="cuda") for _ in batches]

    def pipeline():
        main = torch.cuda.current_stream()      # the capture stream inside torch.cuda.graph
        side.wait_stream(main)
        B.step_mf_prepare(*batches[0], cfg.n_rows, ws[0], stream=side)
        prepared[0].record(side)
        for i in range(len(batches)):
            main.wait_event(prepared[i % 2])
            B.step_mf_apply(nB, cfg.lam, ws[i % 2], loss=losses[i], stream=main, rows_done=rows_done)
            applied[i % 2].record(main)
            if i + 1 < len(batches):
                if i >= 1:
                    side.wait_event(applied[(i + 1) % 2])
                side.wait_event(rows_done)
                B.step_mf_prepare(*batches[i + 1], cfg.n_rows, ws[(i + 1) % 2], stream=side)
                prepared[(i + 1) % 2].record(side)

    for r, c, v in batches:
        A.step_mf(r, c, v, cfg.n_rows, cfg.lam)
    pipeline()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pipeline()
    for rep in range(3):
        lossA = [A.step_mf(r, c, v, cfg.n_rows, cfg.lam).clone() for r, c, v in batches]
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert A.error() == 0 and B.error() == 0
        assert_bitwise(WB.cpu().numpy(), WA.cpu().numpy(), f"W after replay {rep}")
        assert_bitwise(GB.cpu().numpy(), GA.cpu().numpy(), f"G after replay {rep}")
        assert [l.item() for l in losses] == [l.item() for l in lossA]
        say(f"{cfg.name}: replay {rep} equal")

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

"""GPU parity of stores with bf16 values (fp32 accumulators) against the
oracle's push_bf16 / step_mf_bf16: pull bit-exact, push and MF steps to
the tolerance on the widened values, other steps rejected."""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00470_amd import Store, _lib
from paper_2206_00470_amd.workloads import CTR_33M, MF_10Mx1M, CTRWorkload, MFWorkload, random_push, small_variant
from tests.helpers import assert_bitwise, assert_close_tables, mismatch_fraction, say

pytestmark = pytest.mark.gpu

LR, EPS = 0.1, 1e-10


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bf16_dev(Wb):
    return torch.from_numpy(np.ascontiguousarray(Wb).view(np.int16)).cuda().view(torch.bfloat16)


def bf16_host(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_table(K, d, seed):
    rng = np.random.default_rng(seed)
    return oracle.f32_to_bf16((rng.standard_normal((K, d)) * 0.1).astype(np.float32))


@pytest.mark.parametrize("K,d,n", [(1, 4, 1), (5000, 16, 4097), (3000, 3, 777), (700, 512, 999)])
def test_pull_bf16_is_the_widened_rows(K, d, n):
    Wb = bf16_table(K, d, 80)
    s = Store(bf16_dev(Wb), torch.zeros((K, d), dtype=torch.float32, device="cuda"), LR, EPS)
    keys = np.random.default_rng(81).integers(0, K, n)
    out = s.pull(dev(keys)).cpu().numpy()
    assert s.error() == 0
    assert_bitwise(out, oracle.bf16_to_f32(Wb[keys]), "pulled rows")


PUSH_CASES = [(3, 16, 1000, None), (5000, 16, 4097, 1.1), (23_000, 100, 300_001, 1.1), (3000, 3, 2000, None),
              (6000, 300, 20_000, 0.75), (500, 512, 3000, 1.0)]


@pytest.mark.parametrize("K,d,n,zipf", PUSH_CASES)
def test_push_bf16_parity(K, d, n, zipf):
    say(f"bf16 push K={K} d={d} n={n}")
    Wb = bf16_table(K, d, 82)
    G0 = np.random.default_rng(83).uniform(0, 1, (K, d)).astype(np.float32)
    keys, grads = random_push(K, n, d, 84, zipf_s=zipf)
    Wt, Gt = bf16_dev(Wb), dev(G0)
    s = Store(Wt, Gt, LR, EPS)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Gr = Wb.copy(), G0.copy()
    oracle.push_bf16(Wr, Gr, keys, grads, LR, EPS)
    Wg = bf16_host(Wt)
    assert_close_tables(oracle.bf16_to_f32(Wg), oracle.bf16_to_f32(Wr), "widened W")
    assert_close_tables(Gt.cpu().numpy(), Gr, "G")
    untouched = np.setdiff1d(np.arange(K), keys)
    assert_bitwise(Wg[untouched], Wb[untouched], "untouched rows")
    say(f"  W words differing from the oracle: {np.mean(Wg != Wr):.2e}")


def run_mf_bf16(cfg, steps):
    wl = MFWorkload(cfg)
    say(f"{cfg.name}: generating the {cfg.num_keys} x {cfg.dim} table")
    Wb = oracle.f32_to_bf16(wl.init_table())
    Wt, Gt = bf16_dev(Wb), torch.zeros(Wb.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    for step in steps:
        say(f"bf16 {cfg.name} step {step}")
        bt = wl.batch(step)
        Wr, Gr = bf16_host(Wt), Gt.cpu().numpy()
        loss = s.step_mf(dev(bt.row), dev(bt.col), dev(bt.val), cfg.n_rows, cfg.lam)
        assert s.error() == 0
        rloss, bad = oracle.step_mf_bf16(Wr, Gr, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam, cfg.opt.lr, cfg.opt.eps)
        assert bad == 0
        assert float(loss.item()) == pytest.approx(rloss, rel=1e-9)
        Wg = bf16_host(Wt)
        assert_close_tables(oracle.bf16_to_f32(Wg), oracle.bf16_to_f32(Wr), f"widened W after step {step}")
        assert_close_tables(Gt.cpu().numpy(), Gr, f"G after step {step}")
        say(f"  loss {rloss:.6g}; W words differing: {np.mean(Wg != Wr):.2e}")
    return s, Wt, Gt


def test_mf_bf16_small_steps():
    run_mf_bf16(small_variant(MF_10Mx1M), range(3))


def test_mf_bf16_two_phase_equals_one_call():
    cfg = small_variant(MF_10Mx1M)
    wl = MFWorkload(cfg)
    Wb = oracle.f32_to_bf16(wl.init_table())
    bt = wl.batch(0)
    outs = []
    for two_phase in (False, True):
        Wt, Gt = bf16_dev(Wb), torch.zeros(Wb.shape, dtype=torch.float32, device="cuda")
        s = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
        args = (dev(bt.row), dev(bt.col), dev(bt.val))
        if two_phase:
            ws = s.mf_workspace(bt.row.size)
            s.step_mf_prepare(*args, cfg.n_rows, ws)
            loss = s.step_mf_apply(bt.row.size, cfg.lam, ws)
        else:
            loss = s.step_mf(*args, cfg.n_rows, cfg.lam)
        assert s.error() == 0
        outs.append((bf16_host(Wt), Gt.cpu().numpy(), float(loss.item())))
    assert_bitwise(outs[0][0], outs[1][0], "W")
    assert_bitwise(outs[0][1], outs[1][1], "G")
    assert outs[0][2] == outs[1][2]


def test_mf_bf16_paper_scale_one_step():
    cfg = MF_10Mx1M
    run_mf_bf16(cfg, [0])


def test_other_steps_reject_bf16_values():
    cfg = small_variant(CTR_33M)
    wl = CTRWorkload(cfg)
    Wb = oracle.f32_to_bf16(wl.init_table())
    s = Store(bf16_dev(Wb), torch.zeros(Wb.shape, dtype=torch.float32, device="cuda"), LR, EPS)
    bt = wl.batch(0)
    with pytest.raises(_lib.PSError) as e:
        s.step_ctr(dev(bt.keys), dev(bt.label))
    assert e.value.status == _lib.PS_ERR_UNSUPPORTED
    assert_bitwise(bf16_host(s.W), Wb, "table untouched")


@pytest.mark.parametrize("d", [100, 3])
def test_push_bf16_interleaved_rows(d):
    """Values and accumulators of a key side by side in one allocation."""
    from paper_2206_00470_amd.store import interleaved_bf16_tables
    K, n = 4000, 50_000
    Wb = bf16_table(K, d, 85)
    keys, grads = random_push(K, n, d, 86, zipf_s=1.1)
    Wt, Gt = interleaved_bf16_tables(torch.from_numpy(oracle.bf16_to_f32(Wb)).cuda())
    assert Wt.stride(0) * 2 == Gt.stride(0) * 4
    s = Store(Wt, Gt, LR, EPS)
    s.push(dev(keys), dev(grads))
    assert s.error() == 0
    Wr, Gr = Wb.copy(), np.zeros((K, d), np.float32)
    oracle.push_bf16(Wr, Gr, keys, grads, LR, EPS)
    assert_close_tables(oracle.bf16_to_f32(bf16_host(Wt.contiguous())), oracle.bf16_to_f32(Wr), "widened W")
    assert_close_tables(Gt.cpu().numpy(), Gr, "G")


def test_bf16_empty_push_and_step_are_no_ops():
    cfg = small_variant(MF_10Mx1M)
    Wb = bf16_table(cfg.num_keys, cfg.dim, 87)
    Wt, Gt = bf16_dev(Wb), torch.zeros(Wb.shape, dtype=torch.float32, device="cuda")
    s = Store(Wt, Gt, LR, EPS)
    s.push(torch.zeros(0, dtype=torch.int64, device="cuda"), torch.zeros((0, cfg.dim), dtype=torch.float32,
                                                                          device="cuda"))
    e = torch.zeros(0, dtype=torch.int32, device="cuda")
    loss = s.step_mf(e, e, torch.zeros(0, dtype=torch.float32, device="cuda"), cfg.n_rows, cfg.lam)
    assert s.error() == 0 and float(loss.item()) == 0.0
    assert_bitwise(bf16_host(Wt), Wb, "W")

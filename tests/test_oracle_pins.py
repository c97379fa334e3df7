"""Pins of the CPU oracle against things other than itself.

Each test checks the oracle against a library routine, a closed form, an
invariant, finite differences or brute force, chosen so that a plausible
mistake (a dropped term, a wrong sign or index, a transposed operand, a
broken tie-break) fails at least one of them.  No GPU is involved.
"""
import math

import numpy as np
import pytest
import torch

import oracle

LR, EPS = 0.1, 1e-10


def grid_table(rng, rows, dim, scale=64):
    """Values k/scale: exactly representable, so w +- 2^-12 is exact too."""
    return (rng.integers(-scale, scale + 1, (rows, dim)) / scale).astype(np.float32)


def per_key_sum(num_keys, keys, grads):
    """Brute-force per-key fp64 sum of gradient rows (np.add.at)."""
    out = np.zeros((num_keys, grads.shape[1]), np.float64)
    ok = keys >= 0
    np.add.at(out, keys[ok], grads[ok].astype(np.float64))
    return out


def fd_grad(loss_fn, W, h=2.0 ** -12):
    """Central finite differences of loss_fn over every element of W."""
    g = np.zeros(W.shape, np.float64)
    for idx in np.ndindex(*W.shape):
        w0 = W[idx]
        W[idx] = w0 + np.float32(h)
        lp = loss_fn(W)
        W[idx] = w0 - np.float32(h)
        lm = loss_fn(W)
        W[idx] = w0
        g[idx] = (lp - lm) / (2 * h)
    return g


# ---------------------------------------------------------------- pull
def test_pull_is_numpy_fancy_indexing():
    rng = np.random.default_rng(1)
    W = rng.standard_normal((50, 7)).astype(np.float32)
    keys = rng.integers(0, 50, 300)
    out, bad = oracle.pull(W, keys)
    assert bad == 0
    assert np.array_equal(out.view(np.uint32), W[keys].view(np.uint32))


def test_pull_invalid_keys_give_zero_rows_and_are_counted():
    W = np.arange(12, dtype=np.float32).reshape(4, 3) + 1
    keys = np.array([0, -1, 3, 4, 2, 1 << 40])
    out, bad = oracle.pull(W, keys)
    assert bad == 3
    assert np.array_equal(out[[0, 2, 4]], W[[0, 3, 2]])
    assert not out[[1, 3, 5]].any()


# ---------------------------------------------------------------- dedup
@pytest.mark.parametrize("n,num_keys", [(0, 5), (1, 5), (1000, 37), (5000, 100_000)])
def test_dedup_is_numpy_stable_argsort_and_unique(n, num_keys):
    rng = np.random.default_rng(n)
    keys = rng.integers(-3, num_keys + 3, n)
    uniq, perm, offs, bad = oracle.dedup(num_keys, keys)
    valid = (keys >= 0) & (keys < num_keys)
    mapped = np.where(valid, keys, num_keys)
    assert bad == int((~valid).sum())
    assert np.array_equal(perm, np.argsort(mapped, kind="stable"))
    u, first, counts = np.unique(keys[valid], return_index=True, return_counts=True)
    assert np.array_equal(uniq, u)
    assert np.array_equal(np.diff(offs), counts)
    assert offs[0] == 0 and offs[-1] == valid.sum()


def test_dedup_bruteforce_tiny():
    keys = [5, 2, 5, 7, 2, 2, 9, 0, 5, 12, -4, 2]
    num_keys = 10
    uniq, perm, offs, bad = oracle.dedup(num_keys, np.array(keys))
    # brute force: for each distinct valid key ascending, its occurrences ascending
    exp_perm, exp_uniq, exp_offs = [], [], [0]
    for k in range(num_keys):
        occ = [i for i, x in enumerate(keys) if x == k]
        if occ:
            exp_uniq.append(k)
            exp_perm += occ
            exp_offs.append(len(exp_perm))
    exp_perm += [i for i, x in enumerate(keys) if not 0 <= x < num_keys]
    assert bad == 2
    assert list(uniq) == exp_uniq and list(perm) == exp_perm and list(offs) == exp_offs


# ---------------------------------------------------------------- AdaGrad and push
def test_adagrad_first_touch_closed_form():
    """G = 0: sqrt(fl(g*g)) == |g| exactly and eps vanishes for |g| >= 2^-9,
    so the step is exactly -lr*sign(g) whatever the magnitude of g."""
    rng = np.random.default_rng(2)
    g = (rng.uniform(2.0 ** -9, 50.0, 4096) * rng.choice([-1, 1], 4096)).astype(np.float32)
    w0 = rng.standard_normal(4096).astype(np.float32)
    w, acc = oracle.adagrad_row(w0.copy(), np.zeros(4096, np.float32), g, LR, EPS)
    assert np.array_equal(w, (w0 - np.float32(LR) * np.sign(g).astype(np.float32)).astype(np.float32))
    assert np.array_equal(acc, (g * g).astype(np.float32))


def test_adagrad_repeated_pushes_closed_form():
    """k pushes of the same g: G_k = k g^2, so W_k = W_0 - lr sign(g) sum_j j^-1/2."""
    g = np.array([0.75, -3.0, 1e-2, -1e3], np.float32)
    w = np.zeros(4, np.float32)
    acc = np.zeros(4, np.float32)
    for _ in range(25):
        w, acc = oracle.adagrad_row(w, acc, g, LR, EPS)
    expect = -LR * np.sign(g) * sum(j ** -0.5 for j in range(1, 26))
    np.testing.assert_allclose(w, expect, rtol=2e-6)
    np.testing.assert_allclose(acc, 25 * g.astype(np.float64) ** 2, rtol=2e-6)


def test_adagrad_matches_torch_optim_dense():
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal(257).astype(np.float32)
    p = torch.nn.Parameter(torch.from_numpy(w0.copy()))
    opt = torch.optim.Adagrad([p], lr=LR, eps=EPS, initial_accumulator_value=0.0)
    w, acc = w0.copy(), np.zeros_like(w0)
    for _ in range(6):
        g = rng.standard_normal(257).astype(np.float32)
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        w, acc = oracle.adagrad_row(w, acc, g, LR, EPS)
    # torch divides (lr*g)/s where the oracle rounds g/s first: <= 1-2 ulp apart
    np.testing.assert_allclose(w, p.detach().numpy(), rtol=3e-7, atol=1e-7)
    # torch may fuse G + g*g into one FMA: 1 ulp
    np.testing.assert_allclose(acc, opt.state[p]["sum"].numpy(), rtol=3e-7)


def test_push_matches_torch_sparse_embedding_adagrad():
    """Sparse nn.Embedding gradients are coalesced (duplicate rows summed)
    before torch's AdaGrad: the same merge-then-update the push defines."""
    rng = np.random.default_rng(4)
    K, d, n = 40, 6, 500
    W0 = rng.standard_normal((K, d)).astype(np.float32)
    emb = torch.nn.Embedding(K, d, sparse=True)
    emb.weight.data = torch.from_numpy(W0.copy())
    opt = torch.optim.Adagrad(emb.parameters(), lr=LR, eps=EPS)
    W, G = W0.copy(), np.zeros_like(W0)
    for _ in range(3):
        keys = rng.integers(0, K, n)
        grads = rng.standard_normal((n, d)).astype(np.float32)
        opt.zero_grad()
        out = emb(torch.from_numpy(keys))
        out.backward(torch.from_numpy(grads))
        opt.step()
        oracle.push(W, G, keys, grads, LR, EPS)
    # torch sums duplicates in fp32, the oracle in fp64: compare to tolerance
    np.testing.assert_allclose(W, emb.weight.detach().numpy(), rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(G, opt.state[emb.weight]["sum"].to_dense().numpy(), rtol=1e-4, atol=1e-6)


def test_push_brute_force_merge():
    """Each touched row equals one AdaGrad step (torch) on the fp64 sum of its
    occurrences rounded once to fp32; untouched rows are bit-unchanged."""
    rng = np.random.default_rng(5)
    K, d, n = 30, 5, 200
    W0 = rng.standard_normal((K, d)).astype(np.float32)
    G0 = rng.uniform(0, 2, (K, d)).astype(np.float32)
    keys = rng.integers(-2, K + 2, n)
    grads = rng.standard_normal((n, d)).astype(np.float32)
    W, G = W0.copy(), G0.copy()
    bad = oracle.push(W, G, keys, grads, LR, EPS)
    assert bad == int(((keys < 0) | (keys >= K)).sum())
    valid = (keys >= 0) & (keys < K)
    for k in range(K):
        rows = [grads[i].astype(np.float64) for i in range(n) if keys[i] == k]
        if not rows:
            assert np.array_equal(W[k], W0[k]) and np.array_equal(G[k], G0[k])
            continue
        g = np.float32(0) + np.sum(rows, axis=0).astype(np.float32)
        p = torch.nn.Parameter(torch.from_numpy(W0[k].copy()))
        opt = torch.optim.Adagrad([p], lr=LR, eps=EPS)
        opt.state[p]["sum"] = torch.from_numpy(G0[k].copy())
        opt.state[p]["step"] = torch.tensor(0.0)
        p.grad = torch.from_numpy(g)
        opt.step()
        np.testing.assert_allclose(W[k], p.detach().numpy(), rtol=3e-7, atol=1e-7)
        np.testing.assert_allclose(G[k], G0[k] + g * g, rtol=1e-7)
    assert valid.any()


def test_push_exact_cancellation_leaves_row_unchanged():
    rng = np.random.default_rng(6)
    W0 = rng.standard_normal((3, 8)).astype(np.float32)
    G0 = rng.uniform(0, 1, (3, 8)).astype(np.float32)
    x = rng.standard_normal(8).astype(np.float32)
    W, G = W0.copy(), G0.copy()
    oracle.push(W, G, np.array([1, 1]), np.stack([x, -x]), LR, EPS)
    assert np.array_equal(W.view(np.uint32), W0.view(np.uint32))
    assert np.array_equal(G.view(np.uint32), G0.view(np.uint32))


def test_zero_push_then_pull_returns_same_rows():
    rng = np.random.default_rng(7)
    W0 = rng.standard_normal((20, 9)).astype(np.float32)
    G0 = np.where(rng.random((20, 9)) < 0.5, 0, rng.uniform(0, 3, (20, 9))).astype(np.float32)
    W, G = W0.copy(), G0.copy()
    keys = rng.integers(0, 20, 60)
    oracle.push(W, G, keys, np.zeros((60, 9), np.float32), LR, EPS)
    out, _ = oracle.pull(W, np.arange(20))
    assert np.array_equal(out.view(np.uint32), W0.view(np.uint32))
    assert np.array_equal(G.view(np.uint32), G0.view(np.uint32))


def test_push_small_sum_uses_fp64_not_fp32():
    """1 + 2^-30 - 1 is 2^-30 in fp64 but 0 in fp32: the merge must keep it,
    which decides the sign of the first AdaGrad step."""
    W, G = np.zeros((1, 1), np.float32), np.zeros((1, 1), np.float32)
    grads = np.array([[1.0], [2.0 ** -30], [-1.0]], np.float32)
    oracle.push(W, G, np.array([0, 0, 0]), grads, LR, EPS)
    assert G[0, 0] == np.float32(2.0 ** -60)
    assert W[0, 0] < 0


# ---------------------------------------------------------------- row-wise AdaGrad (update variant)
def test_rowwise_first_touch_constant_magnitude_closed_form():
    """Every |g_c| = x with x of at most 12 significant bits: x*x fits fp32 and
    the fp64 partial sums k*x*x are exact, so the row mean of g^2 is x*x, its
    square root is x, each step is exactly -lr*sign(g_c) and the accumulator
    is x*x.  A dropped 1/dim, a sum in place of the mean or the old
    accumulator in the denominator all fail here."""
    rng = np.random.default_rng(40)
    for dim in (1, 3, 64, 100, 129):
        x = np.float32(rng.integers(1, 4096) * 2.0 ** int(rng.integers(-16, -5)))
        g = (x * rng.choice([-1, 1], dim)).astype(np.float32)
        w0 = rng.standard_normal(dim).astype(np.float32)
        w, a = oracle.adagrad_rowwise(w0.copy(), np.float32(0), g, LR, EPS)
        assert a == np.float32(x * x)
        assert np.array_equal(w, (w0 - np.float32(LR) * np.sign(g).astype(np.float32)).astype(np.float32))


def test_rowwise_dim1_is_elementwise_adagrad():
    """With one element per row the two forms coincide bit for bit; the
    element-wise form is pinned to torch.optim.Adagrad above."""
    rng = np.random.default_rng(41)
    w, a = np.float32(0.3), np.float32(0)
    we, ae = np.array([0.3], np.float32), np.zeros(1, np.float32)
    for _ in range(20):
        g = rng.standard_normal(1).astype(np.float32)
        wv, a = oracle.adagrad_rowwise(np.array([w], np.float32), a, g, LR, EPS)
        w = wv[0]
        we, ae = oracle.adagrad_row(we, ae, g, LR, EPS)
        assert w == we[0] and a == ae[0]


def test_rowwise_repeated_pushes_closed_form():
    """k pushes of the same row g: a_k = k*mean(g^2), so
    W_k = W_0 - lr * g/rms(g) * sum_{j<=k} j^-1/2, and every step is parallel to g."""
    rng = np.random.default_rng(42)
    g = rng.standard_normal(37).astype(np.float32)
    ms = float(np.mean(g.astype(np.float64) ** 2))
    w, a = np.zeros(37, np.float32), np.float32(0)
    for _ in range(25):
        w, a = oracle.adagrad_rowwise(w, a, g, LR, EPS)
    expect = -LR * g.astype(np.float64) / math.sqrt(ms) * sum(j ** -0.5 for j in range(1, 26))
    np.testing.assert_allclose(w, expect, rtol=3e-6)
    np.testing.assert_allclose(a, 25 * ms, rtol=3e-6)


def test_rowwise_matches_torch_on_a_row_mean_accumulator():
    """torch reference built from separate pieces: the accumulator is the running
    sum of g.pow(2).mean(); the update divides by its square root plus eps."""
    rng = np.random.default_rng(43)
    d = 50
    w0 = rng.standard_normal(d).astype(np.float32)
    wt, at = torch.from_numpy(w0.copy()).double(), torch.zeros((), dtype=torch.float64)
    w, a = w0.copy(), np.float32(0)
    for _ in range(8):
        g = (rng.standard_normal(d) * rng.uniform(0.01, 10)).astype(np.float32)
        gt = torch.from_numpy(g).double()
        at = at + gt.pow(2).mean()
        wt = wt - LR * gt / (at.sqrt() + EPS)
        w, a = oracle.adagrad_rowwise(w, a, g, LR, EPS)
    np.testing.assert_allclose(w, wt.numpy(), rtol=2e-6, atol=1e-6)
    np.testing.assert_allclose(a, at.item(), rtol=2e-6)


def test_push_rowwise_brute_force_merge():
    """Each touched key gets one row-wise step on the fp64 sum of its occurrences
    rounded once to fp32; untouched rows and accumulators are bit-unchanged."""
    rng = np.random.default_rng(44)
    K, d, n = 30, 7, 250
    W0 = rng.standard_normal((K, d)).astype(np.float32)
    A0 = rng.uniform(0, 2, K).astype(np.float32)
    keys = rng.integers(-2, K + 2, n)
    grads = rng.standard_normal((n, d)).astype(np.float32)
    W, A = W0.copy(), A0.copy()
    bad = oracle.push_rowwise(W, A, keys, grads, LR, EPS)
    assert bad == int(((keys < 0) | (keys >= K)).sum())
    for k in range(K):
        rows = [grads[i].astype(np.float64) for i in range(n) if keys[i] == k]
        if not rows:
            assert np.array_equal(W[k], W0[k]) and A[k] == A0[k]
            continue
        g = np.sum(rows, axis=0).astype(np.float32)
        acc = np.float64(A0[k]) + np.mean(g.astype(np.float64) ** 2)
        np.testing.assert_allclose(A[k], acc, rtol=2e-7)
        np.testing.assert_allclose(W[k], W0[k] - LR * g / (np.sqrt(acc) + EPS), rtol=1e-6, atol=1e-7)


def test_push_rowwise_zero_push_and_cancellation_leave_state_unchanged():
    rng = np.random.default_rng(45)
    W0 = rng.standard_normal((6, 9)).astype(np.float32)
    A0 = np.where(rng.random(6) < 0.5, 0, rng.uniform(0, 3, 6)).astype(np.float32)
    W, A = W0.copy(), A0.copy()
    oracle.push_rowwise(W, A, rng.integers(0, 6, 20), np.zeros((20, 9), np.float32), LR, EPS)
    x = rng.standard_normal(9).astype(np.float32)
    oracle.push_rowwise(W, A, np.array([2, 4, 2]), np.stack([x, np.zeros(9, np.float32), -x]), LR, EPS)
    assert np.array_equal(W.view(np.uint32), W0.view(np.uint32))
    assert np.array_equal(A.view(np.uint32), A0.view(np.uint32))


def test_step_rowwise_on_one_column_table_is_the_elementwise_step():
    """A task step with the row-wise update on a one-column table is the
    element-wise step bit for bit (the merge and gradients are shared)."""
    W, row, col, val, R = mf_setup(46)
    W = np.ascontiguousarray(W[:, :1])
    G = np.zeros_like(W)
    Wr, Ar = W.copy(), np.zeros(W.shape[0], np.float32)
    for _ in range(3):
        loss, _ = oracle.step_mf(W, G, row, col, val, R, 1e-2, LR, EPS)
        loss_r, _ = oracle.step_rowwise("mf", Wr, Ar, (row, col, val, R, 1e-2), LR, EPS)
        assert loss == loss_r
        assert np.array_equal(W, Wr) and np.array_equal(G[:, 0], Ar)


# ---------------------------------------------------------------- MF
def mf_setup(seed=8):
    rng = np.random.default_rng(seed)
    R, Ccols, d, B = 5, 4, 3, 12
    W = grid_table(rng, R + Ccols, d)
    row = rng.integers(0, R, B).astype(np.int32)
    col = rng.integers(0, Ccols, B).astype(np.int32)
    val = (rng.integers(-32, 33, B) / 16).astype(np.float32)
    return W, row, col, val, R


def test_mf_gradients_match_finite_differences():
    W, row, col, val, R = mf_setup()
    keys, grads, loss, bad = oracle.grad_mf(W, row, col, val, R, 1e-2)
    assert bad == 0 and keys.size == 2 * row.size
    fd = fd_grad(lambda T: oracle.grad_mf(T, row, col, val, R, 1e-2)[2], W)
    np.testing.assert_allclose(per_key_sum(W.shape[0], keys, grads), fd, rtol=1e-5, atol=1e-6)


def test_mf_single_entry_rank1_closed_form():
    W = np.array([[0.5], [-1.25]], np.float32)
    keys, grads, loss, _ = oracle.grad_mf(W, np.array([0]), np.array([0]), np.array([2.0]), 1, 0.25)
    # e = 2 - (0.5)(-1.25) = 2.625 ; loss = e^2/2 + 0.25/2 (0.25 + 1.5625)
    assert loss == pytest.approx(0.5 * 2.625 ** 2 + 0.125 * (0.25 + 1.5625), rel=1e-15)
    assert list(keys) == [0, 1]
    assert grads[0, 0] == np.float32(0.25 * 0.5 - 2.625 * -1.25)
    assert grads[1, 0] == np.float32(0.25 * -1.25 - 2.625 * 0.5)


def test_mf_gradients_match_torch_autograd_float64():
    W, row, col, val, R = mf_setup(9)
    keys, grads, loss, _ = oracle.grad_mf(W, row, col, val, R, 1e-2)
    T = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    U, M = T[torch.from_numpy(row.astype(np.int64))], T[R + torch.from_numpy(col.astype(np.int64))]
    e = torch.from_numpy(val.astype(np.float64)) - (U * M).sum(1)
    lam = float(np.float32(1e-2))      # the oracle takes lambda as a float
    L = 0.5 * (e ** 2).sum() + 0.5 * lam * ((U ** 2).sum() + (M ** 2).sum())
    L.backward()
    assert loss == pytest.approx(L.item(), rel=1e-12)
    np.testing.assert_allclose(per_key_sum(W.shape[0], keys, grads), T.grad.numpy(), rtol=1e-6, atol=1e-7)


def test_mf_invalid_entry_is_skipped():
    W, row, col, val, R = mf_setup()
    row[3] = 99
    keys, grads, loss, bad = oracle.grad_mf(W, row, col, val, R, 1e-2)
    assert bad == 1 and keys[6] == -1 and keys[7] == -1 and not grads[6:8].any()


def test_mf_row_id_must_index_the_row_factors():
    W, row, col, val, R = mf_setup()
    row[2] = R            # a column-factor key used as a row id
    keys, grads, loss, bad = oracle.grad_mf(W, row, col, val, R, 1e-2)
    assert bad == 1 and keys[4] == -1 and keys[5] == -1


def test_mf_step_is_grad_then_push():
    W, row, col, val, R = mf_setup(10)
    G = np.zeros_like(W)
    W1, G1 = W.copy(), G.copy()
    loss, _ = oracle.step_mf(W1, G1, row, col, val, R, 1e-2, LR, EPS)
    keys, grads, loss2, _ = oracle.grad_mf(W, row, col, val, R, 1e-2)
    oracle.push(W, G, keys, grads, LR, EPS)
    assert loss == loss2
    assert np.array_equal(W, W1) and np.array_equal(G, G1)


# ---------------------------------------------------------------- KGE (ComplEx)
def test_complex_score_is_real_part_of_trilinear_complex_product():
    rng = np.random.default_rng(11)
    for cdim in (1, 4, 128):
        s, r, o = (rng.standard_normal(2 * cdim).astype(np.float32) for _ in range(3))
        c = lambda x: x[:cdim].astype(np.float64) + 1j * x[cdim:].astype(np.float64)
        expect = np.real(np.sum(c(s) * c(r) * np.conj(c(o))))
        assert oracle.complex_score(s, r, o) == pytest.approx(expect, rel=1e-12, abs=1e-12)


def test_complex_reduces_to_distmult_and_has_the_right_symmetries():
    rng = np.random.default_rng(12)
    cd = 16
    s, r, o = (rng.standard_normal(2 * cd).astype(np.float32) for _ in range(3))
    z = np.zeros(cd, np.float32)
    # imaginary parts zero: DistMult
    sr, rr, orr = (np.concatenate([x[:cd], z]) for x in (s, r, o))
    dm = float(np.sum(sr[:cd].astype(np.float64) * rr[:cd] * orr[:cd]))
    assert oracle.complex_score(sr, rr, orr) == pytest.approx(dm, rel=1e-12)
    # purely imaginary relation: antisymmetric in (s, o)
    ri = np.concatenate([z, r[cd:]])
    assert oracle.complex_score(o, ri, s) == pytest.approx(-oracle.complex_score(s, ri, o), rel=1e-12)
    # purely real relation: symmetric in (s, o)
    rre = np.concatenate([r[:cd], z])
    assert oracle.complex_score(o, rre, s) == pytest.approx(oracle.complex_score(s, rre, o), rel=1e-12)


def kge_setup(seed=13):
    rng = np.random.default_rng(seed)
    E, Rn, cd, B, nneg = 7, 2, 2, 3, 4
    W = grid_table(rng, E + Rn, 2 * cd, scale=16)
    head = rng.integers(0, E, B).astype(np.int32)
    tail = rng.integers(0, E, B).astype(np.int32)
    rel = rng.integers(0, Rn, B).astype(np.int32)
    neg = rng.integers(0, E, (B, nneg)).astype(np.int32)
    return W, head, rel, tail, neg, E


def test_kge_gradients_match_finite_differences():
    W, head, rel, tail, neg, E = kge_setup()
    keys, grads, loss, bad = oracle.grad_kge(W, head, rel, tail, neg, 2, E)
    assert bad == 0 and keys.size == head.size * 7
    fd = fd_grad(lambda T: oracle.grad_kge(T, head, rel, tail, neg, 2, E)[2], W)
    np.testing.assert_allclose(per_key_sum(W.shape[0], keys, grads), fd, rtol=1e-5, atol=1e-6)


def test_kge_loss_and_gradients_match_torch_complex_autograd():
    W, head, rel, tail, neg, E = kge_setup(14)
    keys, grads, loss, _ = oracle.grad_kge(W, head, rel, tail, neg, 2, E)
    T = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    cd = W.shape[1] // 2
    Z = torch.complex(T[:, :cd], T[:, cd:])
    L = 0
    for t in range(head.size):
        s, r, o = Z[head[t]], Z[E + rel[t]], Z[tail[t]]
        L = L + torch.nn.functional.softplus(-torch.real((s * r * o.conj()).sum()))
        for j in range(neg.shape[1]):
            x = Z[neg[t, j]]
            phi = torch.real((x * r * o.conj()).sum()) if j < 2 else torch.real((s * r * x.conj()).sum())
            L = L + torch.nn.functional.softplus(phi)
    L.backward()
    assert loss == pytest.approx(L.item(), rel=1e-12)
    np.testing.assert_allclose(per_key_sum(W.shape[0], keys, grads), T.grad.numpy(), rtol=1e-6, atol=1e-7)


def test_kge_occurrence_layout():
    W, head, rel, tail, neg, E = kge_setup(15)
    keys, grads, loss, _ = oracle.grad_kge(W, head, rel, tail, neg, 2, E)
    per = 3 + neg.shape[1]
    for t in range(head.size):
        assert list(keys[t * per: (t + 1) * per]) == [head[t], E + rel[t], tail[t], *neg[t]]


# ---------------------------------------------------------------- SGNS
def sgns_setup(seed=16, zero_out=False):
    rng = np.random.default_rng(seed)
    V, d, B, w, K = 9, 3, 4, 2, 3
    W = grid_table(rng, 2 * V, d, scale=16)
    if zero_out:
        W[V:] = 0
    centre = rng.integers(0, V, B).astype(np.int32)
    ctx = rng.integers(0, V, (B, 2 * w)).astype(np.int32)
    ctx[0, 0] = -1          # a window slot outside the stream
    neg = rng.integers(0, V, (B, 2 * w, K)).astype(np.int32)
    neg[0, 0] = -1
    return W, centre, ctx, neg, w, V


def test_sgns_gradients_match_finite_differences():
    W, centre, ctx, neg, w, V = sgns_setup()
    keys, grads, loss, bad = oracle.grad_sgns(W, centre, ctx, neg, w, V)
    assert bad == 0
    fd = fd_grad(lambda T: oracle.grad_sgns(T, centre, ctx, neg, w, V)[2], W)
    np.testing.assert_allclose(per_key_sum(W.shape[0], keys, grads), fd, rtol=1e-5, atol=1e-6)


def test_sgns_zero_output_table_closed_form():
    """word2vec starts the output vectors at 0: every score is 0, sigmoid(0)
    = 1/2 exactly, the input-vector gradient is exactly 0 and each output
    occurrence gets -v/2 (context) or +v/2 (negative)."""
    W, centre, ctx, neg, w, V = sgns_setup(17, zero_out=True)
    G = np.zeros_like(W)
    W0 = W.copy()
    loss, bad = oracle.step_sgns(W, G, centre, ctx, neg, w, V, LR, EPS)
    pairs = int((ctx >= 0).sum())
    K = neg.shape[2]
    assert loss == pytest.approx(pairs * (1 + K) * math.log(2.0), rel=1e-14)
    assert np.array_equal(W[:V], W0[:V]) and not G[:V].any()
    gsum = np.zeros((V, W.shape[1]))
    for b in range(centre.size):
        for q in range(ctx.shape[1]):
            if ctx[b, q] < 0:
                continue
            gsum[ctx[b, q]] -= 0.5 * W0[centre[b]]
            for k in range(K):
                gsum[neg[b, q, k]] += 0.5 * W0[centre[b]]
    np.testing.assert_allclose(G[V:], (gsum.astype(np.float32)) ** 2, rtol=1e-6, atol=1e-12)
    # first touch (G = 0): sqrt(g*g) = |g| exactly, so each output element
    # moves by exactly lr against the sign of its summed gradient; the grid
    # values make every nonzero sum at least 1/32 in magnitude
    g32 = gsum.astype(np.float32)
    assert np.all((g32 == 0) | (np.abs(g32) >= 1.0 / 32))
    expect = (W0[V:] - np.float32(LR) * np.sign(g32)).astype(np.float32)
    assert np.array_equal(W[V:].view(np.uint32), expect.view(np.uint32))


def test_sgns_loss_and_gradients_match_torch_autograd():
    """The skip-gram negative-sampling loss of word2vec: for each present
    (centre, context) pair, -log sigmoid(<u_ctx, v>) - sum_k log sigmoid(-<u_neg_k, v>),
    with v the centre's input vector and u output vectors; torch float64
    autograd gives its gradient with respect to both tables."""
    W, centre, ctx, neg, w, V = sgns_setup(22)
    keys, grads, loss, bad = oracle.grad_sgns(W, centre, ctx, neg, w, V)
    assert bad == 0
    T = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    L = torch.zeros((), dtype=torch.float64)
    for b in range(centre.size):
        v = T[centre[b]]
        for q in range(ctx.shape[1]):
            if ctx[b, q] < 0:
                continue
            L = L - torch.nn.functional.logsigmoid(torch.dot(T[V + ctx[b, q]], v))
            for k in range(neg.shape[2]):
                L = L - torch.nn.functional.logsigmoid(-torch.dot(T[V + neg[b, q, k]], v))
    L.backward()
    assert loss == pytest.approx(L.item(), rel=1e-12)
    np.testing.assert_allclose(per_key_sum(W.shape[0], keys, grads), T.grad.numpy(), rtol=1e-6, atol=1e-7)
    # each context occurrence's gradient row points against the centre vector
    # (it raises <u_ctx, v>), each negative's along it
    per = 1 + 2 * w * (1 + neg.shape[2])
    K = neg.shape[2]
    for b in range(centre.size):
        v = W[centre[b]].astype(np.float64)
        for q in range(ctx.shape[1]):
            if ctx[b, q] < 0:
                continue
            o = b * per + 1 + q * (1 + K)
            assert np.dot(grads[o].astype(np.float64), v) < 0
            for k in range(K):
                assert np.dot(grads[o + 1 + k].astype(np.float64), v) > 0


def test_sgns_centre_must_index_the_input_table():
    W, centre, ctx, neg, w, V = sgns_setup(21)
    centre[1] = V + 2            # an output-table row used as a centre word
    keys, grads, loss, bad = oracle.grad_sgns(W, centre, ctx, neg, w, V)
    per = 1 + 2 * w * (1 + neg.shape[2])
    assert bad == 1 and np.all(keys[per:2 * per] == -1) and not grads[per:2 * per].any()


def test_sgns_occurrence_layout_and_absent_slots():
    W, centre, ctx, neg, w, V = sgns_setup(18)
    keys, grads, loss, _ = oracle.grad_sgns(W, centre, ctx, neg, w, V)
    per = 1 + 2 * w * (1 + neg.shape[2])
    assert keys[0] == centre[0]
    assert np.all(keys[1:1 + 1 + neg.shape[2]] == -1)          # slot 0 of centre 0 is absent
    assert keys[per + 1] == V + ctx[1, 0] and keys[per + 2] == V + neg[1, 0, 0]


# ---------------------------------------------------------------- CTR
def ctr_setup(seed=19):
    rng = np.random.default_rng(seed)
    K, d, B, F = 11, 3, 4, 5
    W = grid_table(rng, K, d, scale=16)
    keys = rng.integers(0, K, (B, F))
    keys[0, 1] = keys[0, 3]        # the same row twice in one sample
    label = rng.integers(0, 2, B).astype(np.float32)
    return W, keys, label


def test_ctr_interaction_is_half_square_norm_identity():
    """loss(y=0) - loss(y=1) = z; z = (|S|^2 - sum_f |e_f|^2) / 2."""
    W, keys, _ = ctr_setup()
    for b in range(keys.shape[0]):
        kb = keys[b:b + 1]
        l0 = oracle.grad_ctr(W, kb, np.array([0.0]))[2]
        l1 = oracle.grad_ctr(W, kb, np.array([1.0]))[2]
        E = W[kb[0]].astype(np.float64)
        z = 0.5 * (np.sum(E.sum(0) ** 2) - np.sum(E ** 2))
        assert l0 - l1 == pytest.approx(z, rel=1e-12, abs=1e-14)


def test_ctr_gradients_match_finite_differences():
    W, keys, label = ctr_setup(20)
    okeys, grads, loss, bad = oracle.grad_ctr(W, keys, label)
    assert bad == 0 and np.array_equal(okeys, keys.ravel())
    fd = fd_grad(lambda T: oracle.grad_ctr(T, keys, label)[2], W)
    np.testing.assert_allclose(per_key_sum(W.shape[0], okeys, grads), fd, rtol=1e-5, atol=1e-6)


def test_ctr_single_nonzero_field_closed_form():
    """Only one non-zero embedding: z = 0, a = 1/2 - y exactly; that field's
    gradient is 0 and every other field gets a * e."""
    W = np.zeros((6, 4), np.float32)
    W[2] = [0.5, -1.0, 2.0, 0.25]
    keys = np.array([[0, 2, 1, 5]])
    for y in (0.0, 1.0):
        okeys, grads, loss, _ = oracle.grad_ctr(W, keys, np.array([y]))
        assert loss == pytest.approx(math.log(2.0), rel=1e-15)
        assert not grads[1].any()
        for f in (0, 2, 3):
            assert np.array_equal(grads[f], ((0.5 - y) * W[2]).astype(np.float32))


# ---------------------------------------------------------------- Table 3 arithmetic
def test_table3_bytes_per_value_fits_fp32_value_plus_fp32_accumulator():
    """KGE and WV sizes in Table 3 imply 8 bytes per parameter value: one fp32
    value and one fp32 AdaGrad accumulator, the store's row layout."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "table3_model_sizes.txt")
    rows = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            t, k, v, s = line.split()
            rows[t] = (float(k), float(v), float(s))
    for task in ("kge", "wv"):
        _, values, gb = rows[task]
        assert gb * 2 ** 30 / values == pytest.approx(8.0, rel=0.02)


# ---------------------------------------------------------------- bf16 values (update variant)
def bf16_nearest_brute(x):
    """The nearest bf16 value by comparing the two candidates around x in
    fp64; ties go to the word with an even last bit."""
    u = np.float32(x).view(np.uint32)
    lo = np.uint16(u >> np.uint32(16))
    hi = np.uint16(lo + 1)
    vlo = float(oracle.bf16_to_f32(np.array([lo]))[0])
    vhi = float(oracle.bf16_to_f32(np.array([hi]))[0])
    dlo, dhi = abs(float(x) - vlo), abs(vhi - float(x))
    if dlo < dhi or (dlo == dhi and lo % 2 == 0):
        return lo
    return hi


def test_bf16_rounding_is_nearest_ties_to_even_and_matches_torch():
    rng = np.random.default_rng(70)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([0.0, -0.0, 1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -9, -2.5, 3e38, 1e-40, -1e-41],
                                 np.float32)]).astype(np.float32)
    got = oracle.f32_to_bf16(x)
    want_torch = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want_torch)
    f = oracle.lib().orc_f32_to_bf16           # the scalar routine the array form applies
    for v in x[:3000]:
        if np.isfinite(v) and abs(v) < 3.3e38:
            assert f(float(v)) == bf16_nearest_brute(v), v


def test_bf16_widening_is_exact_and_rounds_back_to_itself():
    words = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    f = oracle.bf16_to_f32(words)
    finite = np.isfinite(f)
    assert np.array_equal(oracle.f32_to_bf16(f[finite]), words[finite])
    assert np.isnan(f[~finite & (words & 0x7f != 0) & ((words & 0x7f80) == 0x7f80)]).all()


def test_push_bf16_is_the_fp32_push_on_widened_values_then_one_rounding():
    rng = np.random.default_rng(71)
    K, d, n = 40, 12, 600
    Wb = oracle.f32_to_bf16(rng.standard_normal((K, d)).astype(np.float32) * 0.1)
    G0 = rng.uniform(0, 1, (K, d)).astype(np.float32)
    keys = rng.integers(-1, K + 1, n)
    grads = rng.standard_normal((n, d)).astype(np.float32)
    W1, G1 = Wb.copy(), G0.copy()
    bad = oracle.push_bf16(W1, G1, keys, grads, LR, EPS)
    W2, G2 = oracle.bf16_to_f32(Wb), G0.copy()
    assert oracle.push(W2, G2, keys, grads, LR, EPS) == bad
    assert np.array_equal(W1, oracle.f32_to_bf16(W2))
    assert np.array_equal(G1, G2)


def test_push_bf16_zero_gradients_keep_every_bit():
    rng = np.random.default_rng(72)
    Wb = oracle.f32_to_bf16(rng.standard_normal((30, 8)).astype(np.float32))
    G0 = rng.uniform(0, 1, (30, 8)).astype(np.float32)
    W1, G1 = Wb.copy(), G0.copy()
    oracle.push_bf16(W1, G1, rng.integers(0, 30, 90), np.zeros((90, 8), np.float32), LR, EPS)
    assert np.array_equal(W1, Wb) and np.array_equal(G1.view(np.uint32), G0.view(np.uint32))

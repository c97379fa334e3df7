"""Pins of the oracle's unmerged push (the asynchronous update semantics of
the paper's experiments, Section 5.1): each occurrence is its own AdaGrad
step, in an order that is not fixed.  Checked against closed forms, the
merged push where they must agree, brute force over every order of tiny
inputs, and invariants."""
import itertools

import numpy as np
import pytest

import oracle

LR, EPS = 0.1, 1e-8


def tables(K, d, seed):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    G = rng.uniform(0.0, 1.0, (K, d)).astype(np.float32)
    return W, G


def test_one_occurrence_per_key_is_the_merged_push():
    K, d = 50, 7
    W, G = tables(K, d, 1)
    keys = np.random.default_rng(2).permutation(K)[:30]
    grads = np.random.default_rng(3).standard_normal((30, d)).astype(np.float32)
    Wa, Ga, Wm, Gm = W.copy(), G.copy(), W.copy(), G.copy()
    oracle.push_sequential(Wa, Ga, keys, grads, LR, EPS)
    oracle.push(Wm, Gm, keys, grads, LR, EPS)
    assert np.array_equal(Wa, Wm) and np.array_equal(Ga, Gm)


@pytest.mark.parametrize("k", [2, 3, 7])
def test_identical_occurrences_closed_form(k):
    """k equal rows g on one key: a_i = a0 + i g^2 and
    w_k = w0 - lr * sum_{i=1..k} g / (sqrt(a0 + i g^2) + eps)."""
    d = 5
    W, G = tables(1, d, 4)
    g = np.array([0.3, -1.25, 0.5, 2.0, -0.0625], np.float32)
    keys = np.zeros(k, np.int64)
    grads = np.tile(g, (k, 1))
    Wa, Ga = W.copy(), G.copy()
    oracle.push_sequential(Wa, Ga, keys, grads, LR, EPS)
    a0, w0, g64 = G[0].astype(np.float64), W[0].astype(np.float64), g.astype(np.float64)
    a = a0 + k * g64 * g64
    w = w0 - LR * sum(g64 / (np.sqrt(a0 + i * g64 * g64) + EPS) for i in range(1, k + 1))
    np.testing.assert_allclose(Ga[0], a, rtol=1e-6)
    np.testing.assert_allclose(Wa[0], w, rtol=1e-5, atol=1e-7)
    # the merged push takes one step with the summed gradient instead
    Wm, Gm = W.copy(), G.copy()
    oracle.push(Wm, Gm, keys, grads, LR, EPS)
    assert not np.allclose(Gm[0], Ga[0])


def test_rowwise_identical_occurrences_closed_form():
    d, k = 6, 4
    W = (np.random.default_rng(5).standard_normal((1, d)) * 0.1).astype(np.float32)
    Gr = np.array([0.25], np.float32)
    g = np.array([0.5, -1.0, 0.25, 0.75, -0.5, 1.5], np.float32)
    Wa, Ga = W.copy(), Gr.copy()
    oracle.push_sequential(Wa, Ga, np.zeros(k, np.int64), np.tile(g, (k, 1)), LR, EPS, rowwise=True)
    t = float((g.astype(np.float64) ** 2).sum() / d)
    np.testing.assert_allclose(Ga[0], 0.25 + k * t, rtol=1e-6)
    w = W[0] - LR * sum(g / (np.sqrt(0.25 + i * t) + EPS) for i in range(1, k + 1))
    np.testing.assert_allclose(Wa[0], w, rtol=1e-5, atol=1e-7)


def test_order_matters_and_the_order_argument_is_followed():
    d = 4
    W, G = tables(1, d, 6)
    grads = np.array([[1.0, -2.0, 0.5, 3.0], [-0.25, 0.75, 2.0, -1.0]], np.float32)
    keys = np.zeros(2, np.int64)
    outs = []
    for order in ([0, 1], [1, 0]):
        Wa, Ga = W.copy(), G.copy()
        oracle.push_sequential(Wa, Ga, keys, grads, LR, EPS, order=order)
        outs.append(Wa)
    assert not np.allclose(outs[0], outs[1], rtol=1e-6, atol=0)
    # order [1, 0] is index order of the swapped occurrences
    Wb, Gb = W.copy(), G.copy()
    oracle.push_sequential(Wb, Gb, keys, grads[::-1], LR, EPS)
    assert np.array_equal(Wb, outs[1])


@pytest.mark.parametrize("rowwise", [False, True])
def test_bounds_hold_every_order_brute_force(rowwise):
    """Every permutation of the occurrences of a tiny push ends inside
    async_bounds (up to fp32 rounding); a key with one occurrence has a
    point interval."""
    K, d = 3, 3
    rng = np.random.default_rng(7)
    W = (rng.standard_normal((K, d)) * 0.1).astype(np.float32)
    G = rng.uniform(0.0, 0.5, K if rowwise else (K, d)).astype(np.float32)
    keys = np.array([0, 1, 0, 2, 0, 1], np.int64)
    grads = rng.standard_normal((keys.size, d)).astype(np.float32)
    lo, hi = oracle.async_bounds(W, G, keys, grads, LR, EPS, rowwise=rowwise)
    results = []
    for perm in itertools.permutations(range(keys.size)):
        Wa, Ga = W.copy(), G.copy()
        oracle.push_sequential(Wa, Ga, keys, grads, LR, EPS, order=np.array(perm), rowwise=rowwise)
        tol = 1e-6 + 1e-6 * np.abs(Wa)
        assert np.all(Wa >= lo - tol) and np.all(Wa <= hi + tol)
        results.append(Wa)
    R = np.stack(results)
    # key 2 has one occurrence: a point interval, reached by every order
    np.testing.assert_allclose(lo[2], hi[2], rtol=0, atol=0)
    assert np.all(R[:, 2] == R[0, 2])
    # untouched rows stay put; touched rows move
    assert not np.allclose(R[0, 0], W[0])


def test_accumulator_is_order_free_and_zero_gradients_change_nothing():
    K, d = 20, 4
    W, G = tables(K, d, 9)
    rng = np.random.default_rng(10)
    keys = rng.integers(0, K, 200)
    grads = rng.standard_normal((200, d)).astype(np.float32)
    Wa, Ga = W.copy(), G.copy()
    oracle.push_sequential(Wa, Ga, keys, grads, LR, EPS, order=rng.permutation(200))
    exp = G.astype(np.float64)
    np.add.at(exp, keys, grads.astype(np.float64) ** 2)
    np.testing.assert_allclose(Ga, exp, rtol=1e-5)
    Wz, Gz = W.copy(), G.copy()
    oracle.push_sequential(Wz, Gz, keys, np.zeros_like(grads), LR, EPS)
    assert np.array_equal(Wz, W) and np.array_equal(Gz, G)


def test_invalid_keys_are_skipped_and_counted():
    K, d = 10, 3
    W, G = tables(K, d, 11)
    keys = np.array([1, -1, K, 4, 1], np.int64)
    grads = np.random.default_rng(12).standard_normal((5, d)).astype(np.float32)
    Wa, Ga = W.copy(), G.copy()
    bad = oracle.push_sequential(Wa, Ga, keys, grads, LR, EPS)
    assert bad == 2
    Wb, Gb = W.copy(), G.copy()
    oracle.push_sequential(Wb, Gb, keys[[0, 3, 4]], grads[[0, 3, 4]], LR, EPS)
    assert np.array_equal(Wa, Wb) and np.array_equal(Ga, Gb)


def test_mf_sequential_step_uses_the_pre_step_gradients():
    """The MF step's gradient rows are those of the merged step (grad_mf on
    the pre-step table); only their application differs."""
    K, d = 40, 4
    W, G = tables(K, d, 13)
    rng = np.random.default_rng(14)
    row, col = rng.integers(0, 25, 60).astype(np.int32), rng.integers(0, 15, 60).astype(np.int32)
    val = rng.standard_normal(60).astype(np.float32)
    keys, grads, loss, bad = oracle.grad_mf(W, row, col, val, 25, 0.01)
    Wa, Ga = W.copy(), G.copy()
    l2, b2 = oracle.step_mf_sequential(Wa, Ga, row, col, val, 25, 0.01, LR, EPS)
    assert (l2, b2) == (loss, bad)
    Wb, Gb = W.copy(), G.copy()
    oracle.push_sequential(Wb, Gb, keys, grads, LR, EPS)
    assert np.array_equal(Wa, Wb) and np.array_equal(Ga, Gb)

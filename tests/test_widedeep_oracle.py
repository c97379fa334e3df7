"""Pins of the Wide & Deep reference (oracle/widedeep.py): torch float64
autograd of the same model, central finite differences, the closed forms
with no hidden layer and with a zero output weight, and skipped samples."""
import numpy as np
import pytest
import torch

from oracle.widedeep import dense_layout, forward_backward, grad_ctr_wd, step_ctr_wd, unpack

E, F, WIDTH = 6, 4, 8          # embedding 6, wide weight at column 6, one pad column
HIDDEN = (9, 5)


def make(seed, K=30, B=11, hidden=HIDDEN, wscale=0.5):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((K, WIDTH)) * 0.3).astype(np.float32)
    W[:, E + 1:] = 0
    _, n = dense_layout(F * E, hidden)
    dense = (rng.standard_normal(n) * wscale).astype(np.float32)
    keys = rng.integers(0, K, (B, F)).astype(np.int64)
    keys[3, 1] = keys[3, 2]                 # a key twice in one sample
    label = (rng.random(B) < 0.4).astype(np.float32)
    return W, dense, keys, label


def torch_model(W, dense, keys, label, hidden):
    rows = torch.tensor(W[keys], dtype=torch.float64, requires_grad=True)      # per occurrence
    p = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True)
         for k, v in unpack(dense.astype(np.float64), F * E, hidden).items()}
    B = keys.shape[0]
    h = rows[:, :, :E].reshape(B, F * E)
    for i in range(len(hidden)):
        h = torch.relu(h @ p[f"W{i + 1}"] + p[f"b{i + 1}"])
    logit = h @ p["w"] + p["c"][0] + rows[:, :, E].sum(dim=1)
    y = torch.tensor(label, dtype=torch.float64)
    loss = torch.nn.functional.binary_cross_entropy_with_logits(logit, y, reduction="sum")
    loss.backward()
    return loss.item(), rows.grad.numpy(), {k: v.grad.numpy() for k, v in p.items()}


@pytest.mark.parametrize("hidden", [HIDDEN, (7,), ()])
def test_gradients_match_torch_autograd_float64(hidden):
    W, dense, keys, label = make(1, hidden=hidden)
    loss, valid, dx, dlogit, dflat = forward_backward(W, dense, keys, label, E, hidden)
    tl, trow, tp = torch_model(W, dense, keys, label, hidden)
    assert valid.all()
    assert loss == pytest.approx(tl, rel=1e-13)
    np.testing.assert_allclose(dx, trow[:, :, :E], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(dlogit[:, None].repeat(F, 1), trow[:, :, E], rtol=1e-12, atol=1e-15)
    assert not trow[:, :, E + 1:].any()
    d = unpack(dflat, F * E, hidden)
    for k in tp:
        np.testing.assert_allclose(d[k], tp[k], rtol=1e-11, atol=1e-13, err_msg=k)
    # the packed per-occurrence rows: [dx_f | dlogit | padding], rounded once to fp32
    okeys, grads, _, _, _ = grad_ctr_wd(W, dense, keys, label, E, hidden)
    assert np.array_equal(okeys, keys.ravel())
    np.testing.assert_allclose(grads, trow.reshape(-1, WIDTH).astype(np.float32), rtol=3e-7, atol=1e-12)


def test_gradients_match_central_finite_differences():
    W, dense, keys, label = make(2)
    W64 = W.astype(np.float64)
    _, _, dx, dlogit, dflat = forward_backward(W64, dense.astype(np.float64), keys, label, E, HIDDEN)
    h = 1e-6

    def L(Wm, dm):
        return forward_backward(Wm, dm, keys, label, E, HIDDEN)[0]

    k = keys[3, 1]
    for c in (0, 3, E):                       # two embedding entries and the wide weight of one key
        Wp, Wm = W64.copy(), W64.copy()
        Wp[k, c] += h
        Wm[k, c] -= h
        fd = (L(Wp, dense.astype(np.float64)) - L(Wm, dense.astype(np.float64))) / (2 * h)
        occ = np.argwhere(keys == k)
        an = sum((dx[b, f, c] if c < E else dlogit[b]) for b, f in occ)
        assert fd == pytest.approx(an, rel=1e-6, abs=1e-9)
    for i in (0, 17, dflat.size - 3, dflat.size - 1):
        dp, dm = dense.astype(np.float64).copy(), dense.astype(np.float64).copy()
        dp[i] += h
        dm[i] -= h
        fd = (L(W64, dp) - L(W64, dm)) / (2 * h)
        assert fd == pytest.approx(dflat[i], rel=1e-6, abs=1e-9)


def test_no_hidden_layer_is_logistic_regression():
    W, dense, keys, label = make(3, hidden=())
    loss, _, dx, dlogit, dflat = forward_backward(W, dense, keys, label, E, ())
    B = keys.shape[0]
    x = W[keys][:, :, :E].reshape(B, F * E).astype(np.float64)
    w, c = dense[:-1].astype(np.float64), float(dense[-1])
    logit = x @ w + c + W[keys][:, :, E].astype(np.float64).sum(1)
    a = 1 / (1 + np.exp(-logit)) - label
    np.testing.assert_allclose(dlogit, a, rtol=1e-13)
    np.testing.assert_allclose(dx.reshape(B, -1), np.outer(a, w), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dflat[:-1], x.T @ a, rtol=1e-12, atol=1e-15)
    assert dflat[-1] == pytest.approx(a.sum(), rel=1e-12)


def test_zero_output_weight_stops_the_deep_gradient():
    W, dense, keys, label = make(4)
    layout, n = dense_layout(F * E, HIDDEN)
    off_w = [o for nm, s, o in layout if nm == "w"][0]
    dense[off_w:off_w + HIDDEN[-1]] = 0
    _, _, dx, dlogit, dflat = forward_backward(W, dense, keys, label, E, HIDDEN)
    assert not dx.any()
    assert not dflat[:off_w].any()                     # every W_l and b_l
    c = float(dense[-1])
    wide = W[keys][:, :, E].astype(np.float64).sum(1)
    np.testing.assert_allclose(dlogit, 1 / (1 + np.exp(-(c + wide))) - label, rtol=1e-13)


def test_invalid_samples_are_skipped_and_step_is_grad_then_push():
    W, dense, keys, label = make(5)
    keys[2, 0] = W.shape[0]
    keys[7, 3] = -4
    okeys, grads, dflat, loss, bad = grad_ctr_wd(W, dense, keys, label, E, HIDDEN)
    assert bad == 2
    assert (okeys.reshape(-1, F)[[2, 7]] == -1).all() and not grads.reshape(-1, F, WIDTH)[[2, 7]].any()
    ok = np.ones(keys.shape[0], bool)
    ok[[2, 7]] = False
    l2 = forward_backward(W, dense, keys[ok], label[ok], E, HIDDEN)
    assert loss == pytest.approx(l2[0], rel=1e-14)
    np.testing.assert_allclose(dflat, l2[4], rtol=1e-12, atol=1e-15)
    import oracle
    G, acc = np.zeros_like(W), np.zeros_like(dense)
    W1, d1 = W.copy(), dense.copy()
    step_ctr_wd(W1, G, d1, acc, keys, label, E, HIDDEN, 0.1, 1e-10)
    W2, G2 = W.copy(), np.zeros_like(W)
    oracle.push(W2, G2, okeys, grads, 0.1, 1e-10)
    d2, a2 = oracle.adagrad_row(dense.copy(), np.zeros_like(dense), dflat.astype(np.float32), 0.1, 1e-10)
    assert np.array_equal(W1, W2) and np.array_equal(G, G2)
    assert np.array_equal(d1, d2) and np.array_equal(acc, a2)
    assert np.array_equal(W1[:, E + 1:], W[:, E + 1:])      # padding untouched

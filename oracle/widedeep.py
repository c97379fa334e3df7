"""Plain reference of the Wide & Deep click-through-rate step (Appendix C,
"Click-through-rate prediction": the Wide & Deep model trained with
minibatch SGD and AdaGrad).

TEST INFRASTRUCTURE ONLY: imported by the tests and the benchmark's CPU
leg, never by the product path.  Written in numpy float64 with matrix
products as library steps; the sparse push and the per-element AdaGrad are
the C oracle's (oracle/__init__.py).

Readings (the paper names the model, not its sizes or layout):
  * Table row of key k: [e_k (E values) | u_k (the key's wide weight) |
    zero padding to the row width].  The padding never enters the model, so
    its gradient is zero and AdaGrad leaves it unchanged.
  * Deep part: x = concat_f e_{key_f} (F*E values); h_0 = x;
    h_l = relu(h_{l-1} W_l + b_l) for the hidden layers; y_deep = h_L w + c.
    Wide part: the sum of the sample's wide weights.  logit = y_deep + wide;
    loss = softplus(logit) - label * logit (logistic).
  * Dense parameters, fp32, in one flat buffer: for each hidden layer W_l
    (fan_in x fan_out, row-major) then b_l, then w (H_L values) and c.
  * A sample with a key outside the table is skipped (no loss, no
    gradient), as in the embedding model.
  * Gradients come from the pre-step parameters.  Each key occurrence's
    gradient row [dx_f | dlogit | 0 ...] is rounded to fp32 and merged by
    the push; dense gradients are sums over the valid samples in fp64,
    rounded once to fp32, then one per-element AdaGrad step.
"""
from __future__ import annotations

import numpy as np

import oracle


def dense_layout(fan_in0: int, hidden):
    """[(name, shape, offset)] of the flat dense buffer and its length."""
    out, off, fan = [], 0, fan_in0
    for i, h in enumerate(hidden):
        out.append((f"W{i + 1}", (fan, h), off))
        off += fan * h
        out.append((f"b{i + 1}", (h,), off))
        off += h
        fan = h
    out.append(("w", (fan,), off))
    off += fan
    out.append(("c", (1,), off))
    off += 1
    return out, off


def unpack(dense, fan_in0, hidden):
    layout, n = dense_layout(fan_in0, hidden)
    assert dense.size == n
    return {name: dense[off:off + int(np.prod(shape))].reshape(shape) for name, shape, off in layout}


def forward_backward(W, dense, keys, label, E, hidden):
    """Loss and gradients of the valid samples, all in float64.
    Returns (loss, valid mask, dx [B, F, E], dlogit [B], dense gradient)."""
    K, width = W.shape
    B, F = keys.shape
    valid = ((keys >= 0) & (keys < K)).all(axis=1)
    kv = np.where(valid[:, None], keys, 0)
    rows = W[kv].astype(np.float64)                     # [B, F, width]
    x = rows[:, :, :E].reshape(B, F * E)
    wide = rows[:, :, E].sum(axis=1)
    p = unpack(dense.astype(np.float64), F * E, hidden)
    hs = [x]
    for i in range(len(hidden)):
        hs.append(np.maximum(hs[-1] @ p[f"W{i + 1}"] + p[f"b{i + 1}"], 0.0))
    logit = hs[-1] @ p["w"] + p["c"][0] + wide
    y = label.astype(np.float64)
    loss_b = np.logaddexp(0.0, logit) - y * logit
    dlogit = 1.0 / (1.0 + np.exp(-logit)) - y
    dlogit = np.where(valid, dlogit, 0.0)
    grads = {"w": hs[-1].T @ dlogit, "c": np.array([dlogit.sum()])}
    dh = np.outer(dlogit, p["w"])
    for i in range(len(hidden), 0, -1):
        dh = dh * (hs[i] > 0.0)
        grads[f"W{i}"] = hs[i - 1].T @ dh
        grads[f"b{i}"] = dh.sum(axis=0)
        dh = dh @ p[f"W{i}"].T
    layout, n = dense_layout(F * E, hidden)
    dflat = np.zeros(n, np.float64)
    for name, shape, off in layout:
        dflat[off:off + int(np.prod(shape))] = grads[name].ravel()
    dx = dh.reshape(B, F, E)
    return float(loss_b[valid].sum()), valid, dx, dlogit, dflat


def grad_ctr_wd(W, dense, keys, label, E, hidden):
    """Per-occurrence (key, fp32 gradient row) pairs in sample-major order,
    the fp64 dense gradient, the loss and the number of skipped samples."""
    K, width = W.shape
    B, F = keys.shape
    loss, valid, dx, dlogit, dflat = forward_backward(W, dense, keys, label, E, hidden)
    g = np.zeros((B, F, width), np.float64)
    g[:, :, :E] = dx
    g[:, :, E] = dlogit[:, None]
    okeys = np.where(valid[:, None], keys, -1).reshape(-1)
    grads = g.astype(np.float32).reshape(B * F, width)
    grads[~np.repeat(valid, F)] = 0.0
    return okeys, grads, dflat, loss, int((~valid).sum())


def step_ctr_wd(W, G, dense, dense_acc, keys, label, E, hidden, lr, eps):
    """One step: gradients from the pre-step parameters, the merging push
    into (W, G), per-element AdaGrad on the dense buffer (in place)."""
    okeys, grads, dflat, loss, bad = grad_ctr_wd(W, dense, keys, label, E, hidden)
    oracle.push(W, G, okeys, grads, lr, eps)
    w, a = oracle.adagrad_row(dense, dense_acc, dflat.astype(np.float32), lr, eps)
    dense[...] = w
    dense_acc[...] = a
    return loss, bad

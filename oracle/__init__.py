"""ctypes front end of the plain CPU oracle (``oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the package smoke check
and by the benchmark's CPU-baseline leg, never by the product path.  It
imports nothing from the GPU package and the GPU package imports nothing
from here.

Every function takes and returns numpy arrays; tables are float32
``[num_keys, dim]`` row-major and are updated in place by the ``step_*`` and
``push`` calls, exactly like the store they check.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc (no fast-math, no contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        L = C.CDLL(_LIB)
        p, i64, i32, f32, f64 = C.c_void_p, C.c_int64, C.c_int32, C.c_float, C.c_double
        sig = {
            "orc_pull": (i64, [p, i64, i32, p, i64, p]),
            "orc_dedup": (i64, [i64, p, i64, p, p, p, p]),
            "orc_adagrad_row": (None, [p, p, p, i32, f32, f32]),
            "orc_push": (i64, [p, p, i64, i32, f32, f32, p, i64, p]),
            "orc_adagrad_rowwise": (None, [p, p, p, i32, f32, f32]),
            "orc_push_rowwise": (i64, [p, p, i64, i32, f32, f32, p, i64, p]),
            "orc_push_sequential": (i64, [p, p, i64, i32, f32, f32, p, i64, p, p]),
            "orc_push_sequential_rowwise": (i64, [p, p, i64, i32, f32, f32, p, i64, p, p]),
            "orc_bf16_to_f32": (f32, [C.c_uint16]),
            "orc_f32_to_bf16": (C.c_uint16, [f32]),
            "orc_push_bf16": (i64, [p, p, i64, i32, f32, f32, p, i64, p]),
            "orc_f32_to_bf16_array": (None, [p, p, i64]),
            "orc_complex_score": (f64, [p, p, p, i32]),
            "orc_grad_mf": (f64, [p, i64, i32, p, p, p, i64, i64, f32, p, p, p]),
            "orc_grad_kge": (f64, [p, i64, i32, p, p, p, p, i64, i32, i32, i64, p, p, p]),
            "orc_grad_sgns": (f64, [p, i64, i32, p, p, p, i64, i32, i32, i64, p, p, p]),
            "orc_grad_ctr": (f64, [p, i64, i32, p, p, i64, i32, p, p, p]),
            "orc_step_mf": (f64, [p, p, i64, i32, f32, f32, p, p, p, i64, i64, f32, p]),
            "orc_step_kge": (f64, [p, p, i64, i32, f32, f32, p, p, p, p, i64, i32, i32, i64, p]),
            "orc_step_sgns": (f64, [p, p, i64, i32, f32, f32, p, p, p, i64, i32, i32, i64, p]),
            "orc_step_ctr": (f64, [p, p, i64, i32, f32, f32, p, p, i64, i32, p]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _table(W):
    assert W.dtype == np.float32 and W.flags.c_contiguous and W.ndim == 2
    return W


# ---------------------------------------------------------------------------
def pull(W, keys):
    W = _table(W)
    keys = _c(keys, np.int64)
    out = np.empty((keys.size, W.shape[1]), np.float32)
    bad = lib().orc_pull(_p(W), W.shape[0], W.shape[1], _p(keys), keys.size, _p(out))
    return out, int(bad)


def dedup(num_keys, keys):
    keys = _c(keys, np.int64)
    n = keys.size
    uniq = np.empty(max(n, 1), np.int64)
    perm = np.empty(max(n, 1), np.int32)
    offs = np.empty(n + 1, np.int32)
    nu = np.zeros(1, np.int32)
    bad = lib().orc_dedup(num_keys, _p(keys), n, _p(uniq), _p(perm), _p(offs), _p(nu))
    u = int(nu[0])
    return uniq[:u].copy(), perm[:n].copy(), offs[: u + 1].copy(), int(bad)


def adagrad_row(w, acc, g, lr, eps):
    w, acc, g = _c(w, np.float32), _c(acc, np.float32), _c(g, np.float32)
    lib().orc_adagrad_row(_p(w), _p(acc), _p(g), w.size, lr, eps)
    return w, acc


def push(W, G, keys, grads, lr, eps):
    W, G = _table(W), _table(G)
    keys = _c(keys, np.int64)
    grads = _c(grads, np.float32).reshape(keys.size, W.shape[1])
    return int(lib().orc_push(_p(W), _p(G), W.shape[0], W.shape[1], lr, eps, _p(keys), keys.size,
                              _p(grads)))


def adagrad_rowwise(w, acc, g, lr, eps):
    """Row-wise AdaGrad on one row; acc is the row's single accumulator."""
    w, g = _c(w, np.float32), _c(g, np.float32)
    a = np.array([acc], np.float32)
    lib().orc_adagrad_rowwise(_p(w), _p(a), _p(g), w.size, lr, eps)
    return w, a[0]


def push_rowwise(W, Gr, keys, grads, lr, eps):
    """The merged push with row-wise AdaGrad; Gr holds one accumulator per key."""
    W = _table(W)
    assert Gr.dtype == np.float32 and Gr.flags.c_contiguous and Gr.shape == (W.shape[0],)
    keys = _c(keys, np.int64)
    grads = _c(grads, np.float32).reshape(keys.size, W.shape[1])
    return int(lib().orc_push_rowwise(_p(W), _p(Gr), W.shape[0], W.shape[1], lr, eps, _p(keys), keys.size,
                                      _p(grads)))


def push_sequential(W, G, keys, grads, lr, eps, order=None, rowwise=False):
    """Write access without merging (the asynchronous update semantics):
    each occurrence's gradient row is its own AdaGrad step, the occurrences
    applied one after another in `order` (occurrence indices; None: index
    order).  rowwise: G holds one accumulator per key (row-wise AdaGrad).
    Returns the number of invalid keys."""
    W = _table(W)
    if rowwise:
        assert G.dtype == np.float32 and G.flags.c_contiguous and G.shape == (W.shape[0],)
    else:
        G = _table(G)
    keys = _c(keys, np.int64)
    grads = _c(grads, np.float32).reshape(keys.size, W.shape[1])
    o = None
    if order is not None:
        o = _c(order, np.int64)
        assert o.size == keys.size
    fn = lib().orc_push_sequential_rowwise if rowwise else lib().orc_push_sequential
    return int(fn(_p(W), _p(G), W.shape[0], W.shape[1], lr, eps, _p(keys), keys.size, _p(grads),
                  None if o is None else _p(o)))


def async_bounds(W0, G0, keys, grads, lr, eps, rowwise=False):
    """Per element of W, the interval [lo, hi] (fp64, exact arithmetic) that
    holds W after the unmerged push in ANY order of the occurrences.

    Occurrence j of key k takes the step lr * g_j / (sqrt(a_j) + eps), where
    a_j is k's accumulator just after j's own square was added:
    G0[k] + g_j^2 <= a_j <= G0[k] + (sum of all of k's squares).  Each step
    therefore lies between its values at those two ends, and the sum of the
    steps between the sums of their smaller and larger ends."""
    K, d = W0.shape
    keys = np.asarray(keys, np.int64)
    g = np.asarray(grads, np.float64).reshape(keys.size, d)
    ok = (keys >= 0) & (keys < K)
    keys, g = keys[ok], g[ok]
    if rowwise:
        t = (g * g).sum(axis=1) / d                   # one square per occurrence (the row mean)
        total = np.asarray(G0, np.float64).copy()
        np.add.at(total, keys, t)
        a_lo = (np.asarray(G0, np.float64)[keys] + t)[:, None]
        a_hi = total[keys][:, None]
    else:
        t = g * g
        total = np.asarray(G0, np.float64).copy()
        np.add.at(total, keys, t)
        a_lo = np.asarray(G0, np.float64)[keys] + t
        a_hi = total[keys]
    s1 = lr * g / (np.sqrt(a_lo) + eps)
    s2 = lr * g / (np.sqrt(a_hi) + eps)
    smin, smax = np.zeros((K, d)), np.zeros((K, d))
    np.add.at(smin, keys, np.minimum(s1, s2))
    np.add.at(smax, keys, np.maximum(s1, s2))
    W = np.asarray(W0, np.float64)
    return W - smax, W - smin


def step_mf_sequential(W, G, row, col, val, col_off, lam, lr, eps, order=None, rowwise=False):
    """An MF step with the asynchronous update semantics: every entry's two
    gradient rows from the pre-step table (occurrences 2b: row key, 2b+1:
    column key), then push_sequential in `order`.  Returns (loss, bad)."""
    keys, grads, loss, bad = grad_mf(W, row, col, val, col_off, lam)
    push_sequential(W, G, keys, grads, lr, eps, order, rowwise)
    return loss, bad


def step_rowwise(task, W, Gr, batch, lr, eps, **kw):
    """A task step with row-wise AdaGrad: the task's per-occurrence gradients
    from the pre-step table, then push_rowwise.  Returns (loss, bad)."""
    grad = {"mf": grad_mf, "kge": grad_kge, "sgns": grad_sgns, "ctr": grad_ctr}[task]
    keys, grads, loss, bad = grad(W, *batch, **kw)
    push_rowwise(W, Gr, keys, grads, lr, eps)
    return loss, bad


def bf16_to_f32(b):
    """Widen bf16 words (uint16) to fp32: exact, the word is the upper half."""
    b = np.asarray(b, np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16(x):
    """Round fp32 values to bf16 words (nearest, ties to even), element by element."""
    x = np.ascontiguousarray(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().orc_f32_to_bf16_array(_p(x), _p(out), x.size)
    return out


def push_bf16(Wb, G, keys, grads, lr, eps):
    """The merged push on a table of bf16 values (uint16 words) with fp32
    accumulators: per key the fp64 sum rounded to fp32, one per-element
    AdaGrad step on the widened values, the result narrowed to bf16."""
    assert Wb.dtype == np.uint16 and Wb.flags.c_contiguous and G.shape == Wb.shape
    G = _table(G)
    keys = _c(keys, np.int64)
    grads = _c(grads, np.float32).reshape(keys.size, Wb.shape[1])
    return int(lib().orc_push_bf16(_p(Wb), _p(G), Wb.shape[0], Wb.shape[1], lr, eps, _p(keys), keys.size,
                                   _p(grads)))


def step_mf_bf16(Wb, G, row, col, val, col_off, lam, lr, eps):
    """An MF step on bf16 values: gradients from the widened pre-step table,
    then push_bf16.  Returns (loss, bad)."""
    keys, grads, loss, bad = grad_mf(bf16_to_f32(Wb), row, col, val, col_off, lam)
    push_bf16(Wb, G, keys, grads, lr, eps)
    return loss, bad


def complex_score(s, r, o):
    s, r, o = _c(s, np.float32), _c(r, np.float32), _c(o, np.float32)
    return float(lib().orc_complex_score(_p(s), _p(r), _p(o), s.size // 2))


def grad_mf(W, row, col, val, col_off, lam):
    W = _table(W)
    row, col, val = _c(row, np.int32), _c(col, np.int32), _c(val, np.float32)
    B = row.size
    keys = np.empty(2 * B, np.int64)
    grads = np.empty((2 * B, W.shape[1]), np.float32)
    bad = C.c_int64(0)
    loss = lib().orc_grad_mf(_p(W), W.shape[0], W.shape[1], _p(row), _p(col), _p(val), B,
                             col_off, lam, _p(keys), _p(grads), C.byref(bad))
    return keys, grads, float(loss), int(bad.value)


def grad_kge(W, head, rel, tail, neg, n_head_neg, rel_off):
    W = _table(W)
    head, rel, tail = _c(head, np.int32), _c(rel, np.int32), _c(tail, np.int32)
    neg = _c(neg, np.int32)
    B = head.size
    n_neg = neg.size // max(B, 1) if B else 0
    per = 3 + n_neg
    keys = np.empty(B * per, np.int64)
    grads = np.empty((B * per, W.shape[1]), np.float32)
    bad = C.c_int64(0)
    loss = lib().orc_grad_kge(_p(W), W.shape[0], W.shape[1], _p(head), _p(rel), _p(tail), _p(neg),
                              B, n_neg, n_head_neg, rel_off, _p(keys), _p(grads), C.byref(bad))
    return keys, grads, float(loss), int(bad.value)


def grad_sgns(W, centre, ctx, neg, window, out_off):
    W = _table(W)
    centre, ctx, neg = _c(centre, np.int32), _c(ctx, np.int32), _c(neg, np.int32)
    B = centre.size
    slots = 2 * window
    n_neg = neg.size // max(B * slots, 1) if B else 0
    per = 1 + slots * (1 + n_neg)
    keys = np.empty(B * per, np.int64)
    grads = np.empty((B * per, W.shape[1]), np.float32)
    bad = C.c_int64(0)
    loss = lib().orc_grad_sgns(_p(W), W.shape[0], W.shape[1], _p(centre), _p(ctx), _p(neg), B,
                               window, n_neg, out_off, _p(keys), _p(grads), C.byref(bad))
    return keys, grads, float(loss), int(bad.value)


def grad_ctr(W, keys, label):
    W = _table(W)
    keys, label = _c(keys, np.int64), _c(label, np.float32)
    B = label.size
    F = keys.size // max(B, 1) if B else 0
    okeys = np.empty(B * F, np.int64)
    grads = np.empty((B * F, W.shape[1]), np.float32)
    bad = C.c_int64(0)
    loss = lib().orc_grad_ctr(_p(W), W.shape[0], W.shape[1], _p(keys), _p(label), B, F,
                              _p(okeys), _p(grads), C.byref(bad))
    return okeys, grads, float(loss), int(bad.value)


def step_mf(W, G, row, col, val, col_off, lam, lr, eps):
    W, G = _table(W), _table(G)
    row, col, val = _c(row, np.int32), _c(col, np.int32), _c(val, np.float32)
    bad = C.c_int64(0)
    loss = lib().orc_step_mf(_p(W), _p(G), W.shape[0], W.shape[1], lr, eps, _p(row), _p(col),
                             _p(val), row.size, col_off, lam, C.byref(bad))
    return float(loss), int(bad.value)


def step_kge(W, G, head, rel, tail, neg, n_head_neg, rel_off, lr, eps):
    W, G = _table(W), _table(G)
    head, rel, tail = _c(head, np.int32), _c(rel, np.int32), _c(tail, np.int32)
    neg = _c(neg, np.int32)
    B = head.size
    n_neg = neg.size // max(B, 1) if B else 0
    bad = C.c_int64(0)
    loss = lib().orc_step_kge(_p(W), _p(G), W.shape[0], W.shape[1], lr, eps, _p(head), _p(rel),
                              _p(tail), _p(neg), B, n_neg, n_head_neg, rel_off, C.byref(bad))
    return float(loss), int(bad.value)


def step_sgns(W, G, centre, ctx, neg, window, out_off, lr, eps):
    W, G = _table(W), _table(G)
    centre, ctx, neg = _c(centre, np.int32), _c(ctx, np.int32), _c(neg, np.int32)
    B = centre.size
    n_neg = neg.size // max(B * 2 * window, 1) if B else 0
    bad = C.c_int64(0)
    loss = lib().orc_step_sgns(_p(W), _p(G), W.shape[0], W.shape[1], lr, eps, _p(centre), _p(ctx),
                               _p(neg), B, window, n_neg, out_off, C.byref(bad))
    return float(loss), int(bad.value)


def step_ctr(W, G, keys, label, lr, eps):
    W, G = _table(W), _table(G)
    keys, label = _c(keys, np.int64), _c(label, np.float32)
    B = label.size
    F = keys.size // max(B, 1) if B else 0
    bad = C.c_int64(0)
    loss = lib().orc_step_ctr(_p(W), _p(G), W.shape[0], W.shape[1], lr, eps, _p(keys), _p(label),
                              B, F, C.byref(bad))
    return float(loss), int(bad.value)


# ---------------------------------------------------------------------------
# The same steps spread over host threads (for timing the oracle on all of a
# host's cores).  The work of a step splits into independent pieces: each
# unit's gradients depend only on the pre-step table, and each key's merge
# and AdaGrad update only on that key's occurrences (Appendix B.1.2: the
# updates of a parameter are merged into its store).  Threads take
# contiguous unit ranges for the first phase and disjoint key ranges for the
# second; every key's occurrences keep their order, so W and G come out bit
# for bit as from the one-thread step.  The loss is the sum of the ranges'
# losses, a different order of additions.
_GRAD = {"mf": "orc_grad_mf", "kge": "orc_grad_kge", "sgns": "orc_grad_sgns", "ctr": "orc_grad_ctr"}


def _grad_call(task, W, a, lo, hi, keys, grads, per):
    """Gradients of units [lo, hi) of the batch `a` into keys/grads at unit lo."""
    L = lib()
    bad = C.c_int64(0)
    K, d = W.shape
    ko, go = _p(keys[lo * per:]), _p(grads[lo * per:])
    if task == "mf":
        loss = L.orc_grad_mf(_p(W), K, d, _p(a["row"][lo:]), _p(a["col"][lo:]), _p(a["val"][lo:]), hi - lo,
                             a["col_off"], a["lam"], ko, go, C.byref(bad))
    elif task == "kge":
        loss = L.orc_grad_kge(_p(W), K, d, _p(a["head"][lo:]), _p(a["rel"][lo:]), _p(a["tail"][lo:]),
                              _p(a["neg"][lo:]), hi - lo, a["n_neg"], a["n_head_neg"], a["rel_off"], ko, go,
                              C.byref(bad))
    elif task == "sgns":
        loss = L.orc_grad_sgns(_p(W), K, d, _p(a["centre"][lo:]), _p(a["ctx"][lo:]), _p(a["neg"][lo:]), hi - lo,
                               a["window"], a["n_neg"], a["out_off"], ko, go, C.byref(bad))
    else:
        loss = L.orc_grad_ctr(_p(W), K, d, _p(a["keys"][lo:]), _p(a["label"][lo:]), hi - lo, a["F"], ko, go,
                              C.byref(bad))
    return float(loss), int(bad.value)


def _batch_args(task, batch):
    """Contiguous C-typed inputs of a task step, the unit count and the key
    occurrences per unit."""
    if task == "mf":
        row, col, val, col_off, lam = batch
        a = {"row": _c(row, np.int32), "col": _c(col, np.int32), "val": _c(val, np.float32), "col_off": col_off,
             "lam": lam}
        return a, a["row"].size, 2
    if task == "kge":
        head, rel, tail, neg, n_head_neg, rel_off = batch
        a = {"head": _c(head, np.int32), "rel": _c(rel, np.int32), "tail": _c(tail, np.int32),
             "neg": _c(neg, np.int32), "n_head_neg": n_head_neg, "rel_off": rel_off}
        B = a["head"].size
        a["n_neg"] = a["neg"].size // max(B, 1) if B else 0
        return a, B, 3 + a["n_neg"]
    if task == "sgns":
        centre, ctx, neg, window, out_off = batch
        a = {"centre": _c(centre, np.int32), "ctx": _c(ctx, np.int32), "neg": _c(neg, np.int32), "window": window,
             "out_off": out_off}
        B = a["centre"].size
        a["n_neg"] = a["neg"].size // max(B * 2 * window, 1) if B else 0
        return a, B, 1 + 2 * window * (1 + a["n_neg"])
    keys, label = batch
    a = {"keys": _c(keys, np.int64), "label": _c(label, np.float32)}
    B = a["label"].size
    a["F"] = a["keys"].size // max(B, 1) if B else 0
    return a, B, a["F"]


def step_threads(task, W, G, batch, lr, eps, threads):
    """One step of `task` ("mf", "kge", "sgns", "ctr"; batch = the arguments
    of grad_<task> after the table) on `threads` host threads: gradients of
    contiguous unit ranges, then the merged per-element AdaGrad push of
    disjoint key ranges.  W and G equal those of step_<task> bit for bit.
    Returns (loss, bad)."""
    from concurrent.futures import ThreadPoolExecutor

    W, G = _table(W), _table(G)
    a, B, per = _batch_args(task, batch)
    K, d = W.shape
    keys = np.empty(B * per, np.int64)
    grads = np.empty((B * per, d), np.float32)
    T = max(1, int(threads))
    cuts = [B * t // T for t in range(T + 1)]
    with ThreadPoolExecutor(T) as ex:
        parts = list(ex.map(lambda t: _grad_call(task, W, a, cuts[t], cuts[t + 1], keys, grads, per), range(T)))
        loss = sum(p[0] for p in parts)
        bad = sum(p[1] for p in parts)
        # disjoint key ranges, each range's occurrences in their original order
        part = np.where(keys >= 0, keys * T // K, 0).astype(np.uint8)
        order = np.argsort(part, kind="stable")
        ks, gs = keys[order], grads[order]
        del grads
        bounds = np.searchsorted(part[order], np.arange(T + 1))
        L = lib()

        def push_range(t):
            lo, hi = int(bounds[t]), int(bounds[t + 1])
            return int(L.orc_push(_p(W), _p(G), K, d, lr, eps, _p(ks[lo:]), hi - lo, _p(gs[lo:])))

        list(ex.map(push_range, range(T)))
    return loss, bad

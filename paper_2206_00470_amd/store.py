"""Python front end of the parameter store: torch tensors in, C ABI calls out.

Only argument marshalling happens here (pointers, sizes, the current HIP
stream, a cached workspace tensor); every step of the computation runs in
the HIP kernels of ``libadapm_hip.so``.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import _lib
from ._lib import check, lib


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, dtype, name: str):
    if not (t.is_cuda and t.dtype == dtype and t.is_contiguous()):
        raise TypeError(f"{name} must be a contiguous {dtype} CUDA tensor")
    return t


class Workspace:
    """A device byte buffer that grows to the largest request seen."""

    def __init__(self, device):
        self.device = device
        self.buf = None

    def get(self, nbytes: int):
        if nbytes == 0:
            return C.c_void_p(0), 0
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return C.c_void_p(self.buf.data_ptr()), self.buf.numel()


def interleaved_tables(W0: torch.Tensor, G0: torch.Tensor | None = None):
    """Copy [num_keys, dim] tables into one [num_keys, 2*dim] allocation and
    return the (W, G) row-strided views: each key's value row and
    accumulator row then sit side by side in HBM."""
    K, d = W0.shape
    T = torch.empty((K, 2 * d), dtype=torch.float32, device=W0.device)
    T[:, :d].copy_(W0)
    if G0 is None:
        T[:, d:].zero_()
    else:
        T[:, d:].copy_(G0)
    return T[:, :d], T[:, d:]


def padded_rowwise_table(W0: torch.Tensor, A0: torch.Tensor | None = None, pad: int = 4):
    """Copy a [num_keys, dim] value table into a [num_keys, dim + pad] tensor
    whose column dim holds each key's row-wise AdaGrad accumulator (zero, or
    A0); returns the (W, A) views for a row-wise Store.  pad = 4 keeps rows
    16-byte aligned when dim is a multiple of 4."""
    K, d = W0.shape
    T = torch.zeros((K, d + pad), dtype=torch.float32, device=W0.device)
    T[:, :d].copy_(W0)
    if A0 is not None:
        T[:, d].copy_(A0)
    return T[:, :d], T[:, d]


def interleaved_bf16_tables(W0: torch.Tensor, G0: torch.Tensor | None = None):
    """One allocation holding, per key, the bf16 values (rounded to nearest,
    ties to even) padded to 16 bytes, then the fp32 accumulators; returns
    the (W bf16, G fp32) row-strided views for a bf16 Store."""
    K, d = W0.shape
    vbytes = (2 * d + 15) // 16 * 16
    row = vbytes + 4 * d
    T = torch.zeros((K, row), dtype=torch.uint8, device=W0.device)
    W = T[:, :2 * d].view(torch.bfloat16)
    G = T[:, vbytes:].view(torch.float32)
    W.copy_(W0.to(torch.bfloat16))
    if G0 is not None:
        G.copy_(G0)
    return W, G


class Store:
    """A parameter store over caller-owned tables W (values) and G (AdaGrad
    accumulators), float32 CUDA tensors.  W is [num_keys, dim], dense or a
    row-strided view.

    G of shape [num_keys, dim] selects per-element AdaGrad; it may be dense
    or share W's row stride (for example the two halves of a
    [num_keys, 2*dim] tensor, see interleaved_tables).  G of shape
    [num_keys] selects row-wise AdaGrad (one accumulator per key, any
    stride: a separate vector or a column of W's row padding, see
    padded_rowwise_table)."""

    def __init__(self, W: torch.Tensor, G: torch.Tensor, lr: float = 0.1, eps: float = 1e-10, stream=None):
        if W.is_cuda and W.dtype == torch.bfloat16:
            self._init_bf16(W, G, lr, eps, stream)
            return
        if not (W.is_cuda and W.dtype == torch.float32 and W.dim() == 2 and W.stride(1) == 1):
            raise TypeError("W must be a float32 CUDA tensor [num_keys, dim] with unit column stride")
        if not (G.is_cuda and G.dtype == torch.float32):
            raise TypeError("G must be a float32 CUDA tensor")
        self.W, self.G = W, G
        self.num_keys, self.dim = W.shape
        self.row_stride = W.stride(0) if W.shape[0] > 1 else self.dim
        self.rowwise = G.dim() == 1
        self.lr, self.eps = lr, eps
        self.ws = Workspace(W.device)
        h = C.c_void_p()
        if self.rowwise:
            if G.shape[0] != self.num_keys:
                raise ValueError("a row-wise accumulator vector needs one value per key")
            astride = G.stride(0) if self.num_keys > 1 else 1
            check(lib().ps_create_rowwise(C.byref(h), self.num_keys, self.dim, self.row_stride, _ptr(W), _ptr(G),
                                          astride, lr, eps, _stream(stream)))
        else:
            if G.dim() != 2 or G.stride(1) != 1:
                raise TypeError("G must be [num_keys, dim] with unit column stride, or [num_keys]")
            if W.shape != G.shape:
                raise ValueError("W and G must have one shape")
            if W.shape[0] > 1 and W.stride(0) != G.stride(0):
                raise ValueError("W and G must share one row stride")
            check(lib().ps_create_strided(C.byref(h), self.num_keys, self.dim, self.row_stride, _ptr(W), _ptr(G),
                                          lr, eps, _stream(stream)))
        self._h = h

    def _init_bf16(self, W, G, lr, eps, stream):
        """bf16 values W [num_keys, dim] with fp32 accumulators G of the same
        shape, in separate allocations (rows may be strided)."""
        if not (W.dim() == 2 and W.stride(1) == 1 and G.is_cuda and G.dtype == torch.float32 and
                G.shape == W.shape and G.stride(1) == 1):
            raise TypeError("bf16 values need fp32 accumulators of the same shape, unit column strides")
        self.W, self.G = W, G
        self.num_keys, self.dim = W.shape
        self.row_stride = W.stride(0) if W.shape[0] > 1 else self.dim
        self.rowwise, self.bf16 = False, True
        self.lr, self.eps = lr, eps
        self.ws = Workspace(W.device)
        h = C.c_void_p()
        gs = G.stride(0) if G.shape[0] > 1 else self.dim
        check(lib().ps_create_bf16(C.byref(h), self.num_keys, self.dim, _ptr(W), self.row_stride, _ptr(G), gs, lr,
                                   eps, _stream(stream)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            check(lib().ps_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- sizing
    def workspace_bytes(self, op: int, units: int, per_unit: int = 1) -> int:
        return int(lib().ps_workspace_bytes(self.num_keys, self.dim, op, units, per_unit))

    def _ws(self, op, units, per_unit):
        return self.ws.get(self.workspace_bytes(op, units, per_unit))

    # ---------------------------------------------------------------- read / write
    def pull(self, keys: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        _dev(keys, torch.int64, "keys")
        n = keys.numel()
        if out is None:
            out = torch.empty((n, self.dim), dtype=torch.float32, device=self.W.device)
        _dev(out, torch.float32, "out")
        check(lib().ps_pull(self._h, _ptr(keys), n, _ptr(out), _stream(stream)))
        return out

    def push(self, keys: torch.Tensor, grads: torch.Tensor, stream=None):
        _dev(keys, torch.int64, "keys")
        _dev(grads, torch.float32, "grads")
        n = keys.numel()
        if grads.numel() != n * self.dim:
            raise ValueError("grads must hold n*dim floats")
        ws, wsb = self._ws(_lib.PS_OP_PUSH, n, 1)
        check(lib().ps_push(self._h, _ptr(keys), n, _ptr(grads), ws, wsb, _stream(stream)))

    def push_workspace(self, n: int) -> torch.Tensor:
        """A workspace of its own for push_prepare / push_apply of n keys."""
        return torch.empty(max(self.workspace_bytes(_lib.PS_OP_PUSH, n, 1), 1), dtype=torch.uint8,
                           device=self.W.device)

    def push_prepare(self, keys: torch.Tensor, ws: torch.Tensor, stream=None):
        """Key work of a push (sort, segments) into ws; reads no table row."""
        _dev(keys, torch.int64, "keys")
        check(lib().ps_push_prepare(self._h, _ptr(keys), keys.numel(), _ptr(ws), ws.numel(), _stream(stream)))

    def push_apply(self, n: int, grads: torch.Tensor, ws: torch.Tensor, stream=None):
        """Merge of a prepared push of n keys: grads into W and G."""
        _dev(grads, torch.float32, "grads")
        if grads.numel() != n * self.dim:
            raise ValueError("grads must hold n*dim floats")
        check(lib().ps_push_apply(self._h, n, _ptr(grads), _ptr(ws), ws.numel(), _stream(stream)))

    def push_noalloc(self, keys: torch.Tensor, grads: torch.Tensor, stream=None):
        """push() with the library's static device scratch as workspace: no
        device memory is allocated, here or in the library."""
        _dev(keys, torch.int64, "keys")
        _dev(grads, torch.float32, "grads")
        n = keys.numel()
        if grads.numel() != n * self.dim:
            raise ValueError("grads must hold n*dim floats")
        check(lib().ps_push_noalloc(self._h, _ptr(keys), n, _ptr(grads), _stream(stream)))

    def push_async(self, keys: torch.Tensor, grads: torch.Tensor, stream=None):
        """Unmerged push: every occurrence its own AdaGrad step, applied with
        atomic adds in no fixed order (the asynchronous update semantics)."""
        _dev(keys, torch.int64, "keys")
        _dev(grads, torch.float32, "grads")
        n = keys.numel()
        if grads.numel() != n * self.dim:
            raise ValueError("grads must hold n*dim floats")
        check(lib().ps_push_async(self._h, _ptr(keys), n, _ptr(grads), _stream(stream)))

    # ---------------------------------------------------------------- task steps
    def _loss(self, loss):
        if loss is None:
            loss = torch.empty(1, dtype=torch.float64, device=self.W.device)
        return _dev(loss, torch.float64, "loss")

    def step_mf(self, row, col, val, col_key_offset: int, lam: float, loss=None, stream=None):
        _dev(row, torch.int32, "row"), _dev(col, torch.int32, "col"), _dev(val, torch.float32, "val")
        B = row.numel()
        loss = self._loss(loss)
        ws, wsb = self._ws(_lib.PS_OP_STEP_MF, B, 2)
        check(lib().ps_step_mf(self._h, _ptr(row), _ptr(col), _ptr(val), B, col_key_offset, lam, _ptr(loss),
                               ws, wsb, _stream(stream)))
        return loss

    def step_mf_async(self, row, col, val, col_key_offset: int, lam: float, loss=None, stream=None):
        """The MF step with the unmerged update (see push_async)."""
        _dev(row, torch.int32, "row"), _dev(col, torch.int32, "col"), _dev(val, torch.float32, "val")
        B = row.numel()
        loss = self._loss(loss)
        ws, wsb = self._ws(_lib.PS_OP_STEP_MF_ASYNC, B, 2)
        check(lib().ps_step_mf_async(self._h, _ptr(row), _ptr(col), _ptr(val), B, col_key_offset, lam,
                                     _ptr(loss), ws, wsb, _stream(stream)))
        return loss

    def mf_workspace(self, B: int) -> torch.Tensor:
        """A workspace of its own for the two-phase MF step (one per batch in flight)."""
        return torch.empty(self.workspace_bytes(_lib.PS_OP_STEP_MF, B, 2), dtype=torch.uint8, device=self.W.device)

    def step_mf_prepare(self, row, col, val, col_key_offset: int, ws: torch.Tensor, stream=None):
        _dev(row, torch.int32, "row"), _dev(col, torch.int32, "col"), _dev(val, torch.float32, "val")
        B = row.numel()
        check(lib().ps_step_mf_prepare(self._h, _ptr(row), _ptr(col), _ptr(val), B, col_key_offset, _ptr(ws),
                                       ws.numel(), _stream(stream)))

    def step_mf_apply(self, B: int, lam: float, ws: torch.Tensor, loss=None, stream=None, rows_done=None):
        """rows_done: a torch.cuda.Event recorded once the row-key merge is enqueued."""
        loss = self._loss(loss)
        ev = C.c_void_p(rows_done.cuda_event) if rows_done is not None else C.c_void_p(0)
        check(lib().ps_step_mf_apply(self._h, B, lam, _ptr(loss), _ptr(ws), ws.numel(), _stream(stream), ev))
        return loss

    def step_kge(self, head, rel, tail, neg, n_head_neg: int, rel_key_offset: int, loss=None, stream=None):
        for t, nm in ((head, "head"), (rel, "rel"), (tail, "tail"), (neg, "neg")):
            _dev(t, torch.int32, nm)
        B = head.numel()
        n_neg = neg.numel() // B if B else 0
        loss = self._loss(loss)
        ws, wsb = self._ws(_lib.PS_OP_STEP_KGE, B, 3 + n_neg)
        check(lib().ps_step_kge(self._h, _ptr(head), _ptr(rel), _ptr(tail), _ptr(neg), B, n_neg, n_head_neg,
                                rel_key_offset, _ptr(loss), ws, wsb, _stream(stream)))
        return loss

    def kge_workspace(self, B: int, n_neg: int) -> torch.Tensor:
        """A workspace of its own for the two-phase ComplEx step (one per batch in flight)."""
        return torch.empty(self.workspace_bytes(_lib.PS_OP_STEP_KGE, B, 3 + n_neg), dtype=torch.uint8,
                           device=self.W.device)

    def step_kge_prepare(self, head, rel, tail, neg, rel_key_offset: int, ws: torch.Tensor, stream=None):
        """Key work of a ComplEx step (validity, sort, segments) into ws; reads no table row."""
        for t, nm in ((head, "head"), (rel, "rel"), (tail, "tail"), (neg, "neg")):
            _dev(t, torch.int32, nm)
        B = head.numel()
        n_neg = neg.numel() // B if B else 0
        check(lib().ps_step_kge_prepare(self._h, _ptr(head), _ptr(rel), _ptr(tail), _ptr(neg), B, n_neg,
                                        rel_key_offset, _ptr(ws), ws.numel(), _stream(stream)))

    def step_kge_apply(self, head, rel, tail, neg, n_head_neg: int, rel_key_offset: int, ws: torch.Tensor,
                       loss=None, stream=None):
        """Gradients and merge of a prepared ComplEx step; ids as given to the prepare."""
        for t, nm in ((head, "head"), (rel, "rel"), (tail, "tail"), (neg, "neg")):
            _dev(t, torch.int32, nm)
        B = head.numel()
        n_neg = neg.numel() // B if B else 0
        loss = self._loss(loss)
        check(lib().ps_step_kge_apply(self._h, _ptr(head), _ptr(rel), _ptr(tail), _ptr(neg), B, n_neg, n_head_neg,
                                      rel_key_offset, _ptr(loss), _ptr(ws), ws.numel(), _stream(stream)))
        return loss

    def sgns_workspace(self, B: int, window: int, n_neg: int) -> torch.Tensor:
        """A workspace of its own for the two-phase skip-gram step (one per batch in flight)."""
        return torch.empty(self.workspace_bytes(_lib.PS_OP_STEP_SGNS, B, 1 + 2 * window * (1 + n_neg)),
                           dtype=torch.uint8, device=self.W.device)

    def step_sgns_prepare(self, centre, ctx, neg, window: int, out_key_offset: int, ws: torch.Tensor, stream=None):
        """Key work of a skip-gram step (validity, sort, segments) into ws; reads no table row."""
        for t, nm in ((centre, "centre"), (ctx, "ctx"), (neg, "neg")):
            _dev(t, torch.int32, nm)
        B = centre.numel()
        n_neg = neg.numel() // (B * 2 * window) if B and window else 0
        check(lib().ps_step_sgns_prepare(self._h, _ptr(centre), _ptr(ctx), _ptr(neg), B, window, n_neg,
                                         out_key_offset, _ptr(ws), ws.numel(), _stream(stream)))

    def step_sgns_apply(self, centre, ctx, neg, window: int, out_key_offset: int, ws: torch.Tensor, loss=None,
                        stream=None):
        """Gradients and merges of a prepared skip-gram step; ids as given to the prepare."""
        for t, nm in ((centre, "centre"), (ctx, "ctx"), (neg, "neg")):
            _dev(t, torch.int32, nm)
        B = centre.numel()
        n_neg = neg.numel() // (B * 2 * window) if B and window else 0
        loss = self._loss(loss)
        check(lib().ps_step_sgns_apply(self._h, _ptr(centre), _ptr(ctx), _ptr(neg), B, window, n_neg,
                                       out_key_offset, _ptr(loss), _ptr(ws), ws.numel(), _stream(stream)))
        return loss

    def step_sgns(self, centre, ctx, neg, window: int, out_key_offset: int, loss=None, stream=None):
        for t, nm in ((centre, "centre"), (ctx, "ctx"), (neg, "neg")):
            _dev(t, torch.int32, nm)
        B = centre.numel()
        n_neg = neg.numel() // (B * 2 * window) if B else 0
        loss = self._loss(loss)
        ws, wsb = self._ws(_lib.PS_OP_STEP_SGNS, B, 1 + 2 * window * (1 + n_neg))
        check(lib().ps_step_sgns(self._h, _ptr(centre), _ptr(ctx), _ptr(neg), B, window, n_neg, out_key_offset,
                                 _ptr(loss), ws, wsb, _stream(stream)))
        return loss

    def step_ctr(self, keys, label, loss=None, stream=None):
        _dev(keys, torch.int64, "keys"), _dev(label, torch.float32, "label")
        B = label.numel()
        F = keys.numel() // B if B else 0
        loss = self._loss(loss)
        ws, wsb = self._ws(_lib.PS_OP_STEP_CTR, B, max(F, 1))
        check(lib().ps_step_ctr(self._h, _ptr(keys), _ptr(label), B, F, _ptr(loss), ws, wsb, _stream(stream)))
        return loss

    def ctr_workspace(self, B: int, F: int) -> torch.Tensor:
        """A workspace of its own for the two-phase CTR step (one per batch in flight)."""
        return torch.empty(self.workspace_bytes(_lib.PS_OP_STEP_CTR, B, max(F, 1)), dtype=torch.uint8,
                           device=self.W.device)

    def step_ctr_prepare(self, keys, F: int, ws: torch.Tensor, stream=None):
        """Key work of a CTR step (validity, sort, segments) into ws; reads no table row."""
        _dev(keys, torch.int64, "keys")
        B = keys.numel() // F if F > 0 else 0
        check(lib().ps_step_ctr_prepare(self._h, _ptr(keys), B, F, _ptr(ws), ws.numel(), _stream(stream)))

    def step_ctr_apply(self, keys, label, ws: torch.Tensor, loss=None, stream=None):
        """Gradients and merge of a prepared CTR step; keys as given to the prepare."""
        _dev(keys, torch.int64, "keys"), _dev(label, torch.float32, "label")
        B = label.numel()
        F = keys.numel() // B if B else 1
        loss = self._loss(loss)
        check(lib().ps_step_ctr_apply(self._h, _ptr(keys), _ptr(label), B, F, _ptr(loss), _ptr(ws), ws.numel(),
                                      _stream(stream)))
        return loss

    def step_ctr_wd(self, keys, label, dense, dense_acc, emb_dim: int, hidden, loss=None, stream=None):
        """Wide & Deep CTR step: rows [embedding (emb_dim) | wide weight | ...],
        an MLP of the given hidden widths over the F embeddings; `dense` and
        `dense_acc` are the flat fp32 dense parameters and accumulators."""
        _dev(keys, torch.int64, "keys"), _dev(label, torch.float32, "label")
        _dev(dense, torch.float32, "dense"), _dev(dense_acc, torch.float32, "dense_acc")
        B = label.numel()
        F = keys.numel() // B if B else 1
        hid = (C.c_int32 * max(len(hidden), 1))(*hidden)
        loss = self._loss(loss)
        nbytes = int(lib().ps_ctr_wd_workspace_bytes(self.num_keys, self.dim, B, F, emb_dim, len(hidden), hid))
        ws, wsb = self.ws.get(nbytes)
        check(lib().ps_step_ctr_wd(self._h, _ptr(keys), _ptr(label), B, F, emb_dim, len(hidden), hid, _ptr(dense),
                                   _ptr(dense_acc), _ptr(loss), ws, wsb, _stream(stream)))
        return loss

    # ---------------------------------------------------------------- status and timing
    def error(self, stream=None) -> int:
        """Synchronize, then return and clear the sticky device status."""
        return int(lib().ps_get_error(self._h, _stream(stream)))

    def set_timing(self, on):
        """True: time every kernel id; False: off; an int: bit mask of kernel ids."""
        mask = -1 if on is True else (0 if on is False else int(on))
        check(lib().ps_set_timing(self._h, mask))

    def read_timing(self, kernel_id: int):
        ms, n = C.c_double(0.0), C.c_int64(0)
        check(lib().ps_read_timing(self._h, kernel_id, C.byref(ms), C.byref(n)))
        return ms.value, n.value

    def probe_gather(self, keys: torch.Tensor, sink: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """Instrumentation: read the value rows keys (int32) in order, as a
        gather-bound kernel would, without its arithmetic; returns the
        per-workgroup fp64 sums of what was read (sink)."""
        _dev(keys, torch.int32, "keys")
        if sink is None:
            sink = torch.empty(_lib.PS_PROBE_GRID, dtype=torch.float64, device=self.W.device)
        _dev(sink, torch.float64, "sink")
        if sink.numel() < _lib.PS_PROBE_GRID:
            raise ValueError(f"sink needs {_lib.PS_PROBE_GRID} values")
        check(lib().ps_probe_gather(self._h, _ptr(keys), keys.numel(), _ptr(sink), _stream(stream)))
        return sink


class StagedStore(Store):
    """A store whose full tables live in pinned host memory (the home store)
    while HBM holds a table of slots for the keys of acted-upon intents:
    intent signalling and adaptive action timing for one worker, the GPU.

    W0: initial values [num_keys, dim] (numpy or CPU tensor; accumulators
    start at zero, or from G0).  ranges: ascending first keys of the key
    ranges (the first is 0); slots: the slot capacity of each range.  A key
    offset that a step takes must begin a range.  The home rows are one
    pinned [num_keys, 2*dim] tensor (values | accumulators), the slots one
    [sum(slots), 2*dim] device tensor.

    Protocol: intent(keys, c_start, c_end) ahead of use; advance_clock()
    before each batch's step, on the step's stream; round() (or auto()) to
    act on intents; flush() before reading home_tables()."""

    def __init__(self, W0, ranges, slots, lr: float = 0.1, eps: float = 1e-10, device="cuda", stream=None,
                 G0=None):
        W0 = torch.as_tensor(W0, dtype=torch.float32)
        K, d = W0.shape
        home = torch.empty((K, 2 * d), dtype=torch.float32, pin_memory=True)
        home[:, :d].copy_(W0)
        if G0 is None:
            home[:, d:].zero_()
        else:
            home[:, d:].copy_(torch.as_tensor(G0, dtype=torch.float32))
        total = int(sum(slots))
        T = torch.zeros((total, 2 * d), dtype=torch.float32, device=device)
        self.home = home
        self.W, self.G = T[:, :d], T[:, d:]
        self.key_slot = torch.empty(K, dtype=torch.int32, device=device)
        self.num_keys, self.dim = K, d
        self.row_stride = 2 * d
        self.rowwise = False
        self.lr, self.eps = lr, eps
        self.ws = Workspace(torch.device(device))
        self.ranges, self.slots = list(ranges), list(slots)
        rb = (C.c_int64 * len(ranges))(*ranges)
        rs = (C.c_int64 * len(slots))(*slots)
        h = C.c_void_p()
        hp = home.data_ptr()
        check(lib().ps_create_staged(C.byref(h), K, d, C.c_void_p(hp), C.c_void_p(hp + 4 * d), 2 * d, _ptr(self.W),
                                     _ptr(self.G), 2 * d, _ptr(self.key_slot), len(ranges), rb, rs, lr, eps,
                                     _stream(stream)))
        self._h = h

    def set_action_timing(self, alpha: float = 0.1, p: float = 0.9999, lambda0: float = 10.0):
        check(lib().ps_set_action_timing(self._h, alpha, p, lambda0))

    def intent(self, keys, c_start: int, c_end: int):
        """Intent(keys, C_start, C_end): host keys (numpy, list or CPU tensor)."""
        k = np.ascontiguousarray(np.asarray(keys, dtype=np.int64).ravel())
        check(lib().ps_intent(self._h, C.c_void_p(k.ctypes.data), k.size, c_start, c_end))

    def advance_clock(self, stream=None):
        check(lib().ps_advance_clock(self._h, _stream(stream)))

    def round(self, wait: bool = False):
        check(lib().ps_stage_round(self._h, int(wait)))

    def auto(self, on: bool = True):
        check(lib().ps_stage_auto(self._h, int(on)))

    def flush(self, stream=None):
        check(lib().ps_stage_flush(self._h, _stream(stream)))

    def stats(self) -> dict:
        n = len(_lib.STAGE_STATS)
        v = (C.c_int64 * n)()
        lam = C.c_double(0.0)
        check(lib().ps_stage_stats(self._h, v, n, C.byref(lam)))
        d = dict(zip(_lib.STAGE_STATS, list(v)))
        d["lambda"] = lam.value
        return d

    def resident(self) -> np.ndarray:
        cnt = C.c_int64(0)
        check(lib().ps_stage_resident(self._h, None, 0, C.byref(cnt)))
        out = np.empty(cnt.value, np.int64)
        check(lib().ps_stage_resident(self._h, C.c_void_p(out.ctypes.data), out.size, C.byref(cnt)))
        return out[:cnt.value]

    def home_tables(self):
        """(values, accumulators) of the home store as numpy views (current after flush())."""
        d = self.dim
        a = self.home.numpy()
        return a[:, :d], a[:, d:]


def action_timing(lam_prev: float, c_prev: int, c_now: int, alpha: float = 0.1, p: float = 0.9999):
    """Algorithm 1 as the library computes it: (new estimate, horizon)."""
    lam, h = C.c_double(0.0), C.c_int64(0)
    check(lib().ps_action_timing(lam_prev, c_prev, c_now, alpha, p, C.byref(lam), C.byref(h)))
    return lam.value, h.value


def dedup(num_keys: int, keys: torch.Tensor, err: torch.Tensor | None = None, stream=None):
    """Stable duplicate-key merge order of `keys`: (uniq, perm, offsets, U)."""
    _dev(keys, torch.int64, "keys")
    n = keys.numel()
    dev = keys.device
    uniq = torch.empty(max(n, 1), dtype=torch.int64, device=dev)
    perm = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    offs = torch.empty(n + 1, dtype=torch.int32, device=dev)
    nu = torch.empty(1, dtype=torch.int32, device=dev)
    nbytes = int(lib().ps_workspace_bytes(num_keys, 1, _lib.PS_OP_DEDUP, n, 1)) if n else 0
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    check(lib().ps_dedup(num_keys, _ptr(keys), n, _ptr(uniq), _ptr(perm), _ptr(offs), _ptr(nu), _ptr(err),
                         _ptr(ws), nbytes, _stream(stream)))
    U = int(nu.item())
    return uniq[:U], perm[:n], offs[:U + 1], U

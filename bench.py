#!/usr/bin/env python3
"""Throughput of the sparse parameter-store training step on one MI355X.

Default workload: matrix factorization of a synthetic 10,000,000 x 1,000,000
matrix (rows uniform, columns Zipf 1.1), rank-100 fp32 factors with fp32
AdaGrad accumulators (11M keys x 100, 8.8 GB of W+G in HBM), 1,048,576
entries per step.  One step = ps_step_mf: key intake, stable radix sort of
the 2,097,152 key occurrences, segment boundaries, per-entry gradients from
the pulled rows, fp64 per-key merge and the AdaGrad row update.

--workload selects one of the other task shapes (mf_tiny, kge, sgns, ctr).

Prints one JSON line: rows pulled + pushed per second (2 row accesses per
key occurrence) over exactly --steps timed steps, each on its own
pre-generated batch resident in HBM, and their median from HIP events; the
roofline of the dominant kernel measured with HIP events during the timed
steps (only that kernel is bracketed there: every event costs the GPU a few
microseconds; the warm-up steps pick it, and a few extra steps with every
big kernel bracketed give the per-kernel breakdown); push-only and
pull-only rates; kernel launches per step; and the CPU oracle timed on the
host, on one core and on all of them.

Algorithmic bytes: the fused step reads the batch's inputs once and, per
distinct key, its value and accumulator rows once and writes them once
(inputs + 4 U R); a kernel's share is the inputs it reads plus the keys it
updates.  The bytes the kernels actually move for gradient rows, records
and row gathers are reported beside them as kernel bytes.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0   # MI355X HBM3E
HOST_LINK_GBPS = 64.0    # PCIe 5.0 x16, one direction
MFMA_F64_TFLOPS = 78.6   # MI355X dense fp64 matrix peak


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mf", choices=["mf", "mf_tiny", "mf_colorder", "kge", "kge2x100", "sgns",
                                                           "sgns_w2v", "ctr", "ctr_wd"])
    ap.add_argument("--rank", type=int, default=0,
                    help="MF workloads: factor rank in place of the configuration's (rows of more than 512 "
                         "floats, such as the paper's rank 1,000, have pull and push only: use with --ops-only)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="bound on the CPU-oracle sample (0 = skip)")
    ap.add_argument("--no-ops", action="store_true", help="skip the pull-only / push-only measurements")
    ap.add_argument("--ops-only", action="store_true",
                    help="only the pull-only / push-only measurements (for counter runs of those calls)")
    ap.add_argument("--layout", default="interleaved", choices=["interleaved", "dense"],
                    help="W and G rows of a key side by side in one allocation, or two dense tables "
                         "(row-wise update: the accumulator in each W row's padding, or a separate vector)")
    ap.add_argument("--update", default="elementwise", choices=["elementwise", "rowwise", "async"],
                    help="AdaGrad with one accumulator per element (the paper's), or per key (an update "
                         "variant with half the table traffic), or per element applied without merging "
                         "(async: every occurrence its own step, atomic adds in no fixed order; MF only)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a 4 GiB device-to-device copy (reference for HBM counters)")
    ap.add_argument("--no-overlap", action="store_true",
                    help="one step call per step instead of overlapping the next batch's key work (sort, "
                         "segments; MF: records) on a second stream with this batch's table update")
    ap.add_argument("--values", default="f32", choices=["f32", "bf16"],
                    help="fp32 values, or bf16 values with fp32 accumulators (an update variant; MF workloads)")
    ap.add_argument("--staged", action="store_true",
                    help="home tables in pinned host memory, HBM slots for the keys of acted-upon intents; "
                         "intents signalled --lookahead batches ahead, rounds on the library's thread")
    ap.add_argument("--lookahead", type=int, default=2, help="staged: batches between intent and use")
    ap.add_argument("--graph", action="store_true",
                    help="capture the timed steps in one HIP graph and time its replay (for the launch-bound "
                         "small configurations); the roofline then comes from the eager breakdown steps")
    return ap.parse_args()


# device code of the sort, merge and task kernels and their launches: the
# committed counters stay valid while these files are unchanged
COUNTER_SOURCES = ("common.hpp", "fp64math.hpp", "push.hpp", "sort.hpp", "tasks.hpp", "api.hip")


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2206_00470_amd", "csrc")
    for name in COUNTER_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_summary(name: str):
    """A committed rocprofv3 counter summary (profiles/counters_<name>.json),
    if it was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", f"counters_{name}.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    return data if data.get("source_hash") == source_hash() else None


def counter_traffic(workload: str, kernel: str):
    """HBM bytes per launch of one kernel from the committed counters."""
    data = counter_summary(workload)
    k = (data or {}).get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


# ---------------------------------------------------------------------------- workloads
class Bench:
    """One workload: its table, resident step batches, the step call, the
    algorithmic bytes of its two big kernels and the oracle step."""

    def __init__(self, name, dev, nbatches, rowwise=False, values="f32", unmerged=False, rank=0):
        import torch
        from paper_2206_00470_amd import workloads as wls

        self.name = name
        self.rowwise = rowwise
        self.values = values
        self.unmerged = unmerged
        self.task = {"mf_tiny": "mf", "mf_colorder": "mf", "kge2x100": "kge", "sgns_w2v": "sgns"}.get(name, name)
        cfgs = {"mf": wls.MF_10Mx1M, "mf_tiny": wls.MF_TINY, "mf_colorder": wls.MF_10Mx1M_COLORDER,
                "kge": wls.KGE_COMPLEX, "kge2x100": wls.KGE_COMPLEX_2x100, "sgns": wls.SGNS_1M,
                "sgns_w2v": wls.SGNS_1M_W2V, "ctr": wls.CTR_33M, "ctr_wd": wls.CTR_33M_WD}
        self.cfg = cfg = cfgs[name]
        if rank:
            from dataclasses import replace
            self.cfg = cfg = replace(cfg, rank=rank, name=f"{cfg.name.rsplit('_r', 1)[0]}_r{rank}")
        self.wl = wls.workload(cfg)
        self.dev = dev
        self.dim = cfg.dim
        self.R = 4 * cfg.dim                              # an fp32 row (gradients, accumulators)
        self.RV = (2 if values == "bf16" else 4) * cfg.dim   # a value row
        self.W = self.wl.init_table()
        if self.task == "ctr_wd":
            self.dense0 = self.wl.init_dense()
            self.D = torch.from_numpy(self.dense0).to(dev)
            self.A = torch.zeros_like(self.D)
        T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        self.T = T
        self.batches, self.host_batches, self.occ, self.uniq = [], [], [], []

        def gen(i):
            bt = self.wl.batch(i)
            keys = self.keys_of(bt)
            return bt, keys.size, np.unique(keys).size

        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(min(host_threads(), max(1, nbatches))) as ex:
            for bt, n, u in ex.map(gen, range(nbatches)):
                self.host_batches.append(bt)
                self.batches.append({k: T(v) for k, v in bt.__dict__.items()})
                self.occ.append(n)
                self.uniq.append(u)

    def keys_of(self, bt):
        c = self.cfg
        if self.task == "mf":
            return np.concatenate([bt.row.astype(np.int64), c.n_rows + bt.col.astype(np.int64)])
        if self.task == "kge":
            return np.concatenate([bt.head, c.n_ent + bt.rel.astype(np.int64), bt.tail, bt.neg.ravel()]).astype(np.int64)
        if self.task == "sgns":
            ctx = bt.ctx.astype(np.int64)
            neg = bt.neg.astype(np.int64)
            present = ctx >= 0
            return np.concatenate([bt.centre.astype(np.int64), c.vocab + ctx[present],
                                   c.vocab + neg[present].ravel()])
        return bt.keys.ravel()

    def step(self, store, i, loss):
        c, b = self.cfg, self.batches[i % len(self.batches)]
        if self.task == "mf" and self.unmerged:
            store.step_mf_async(b["row"], b["col"], b["val"], c.n_rows, c.lam, loss=loss)
        elif self.task == "mf":
            store.step_mf(b["row"], b["col"], b["val"], c.n_rows, c.lam, loss=loss)
        elif self.task == "kge":
            store.step_kge(b["head"], b["rel"], b["tail"], b["neg"], c.n_head_neg, c.n_ent, loss=loss)
        elif self.task == "sgns":
            store.step_sgns(b["centre"], b["ctx"], b["neg"], c.window, c.vocab, loss=loss)
        elif self.task == "ctr_wd":
            store.step_ctr_wd(b["keys"], b["label"], self.D, self.A, c.emb_dim, c.deep, loss=loss)
        else:
            store.step_ctr(b["keys"], b["label"], loss=loss)

    def mlp_flops(self, B):
        """fp64 products of one Wide & Deep step: per hidden layer the
        forward, the weight gradient and the input gradient, 2 B fan_in
        fan_out flops each."""
        c = self.cfg
        fan, fl = c.n_fields * c.emb_dim, 0.0
        for h in c.deep:
            fl += 3 * 2.0 * B * fan * h
            fan = h
        return fl

    def run_overlapped_task(self, store, first, count, loss, after_step=None):
        """ComplEx, skip-gram or CTR steps first .. first+count-1 with the
        two-phase step: the key work of batch i+1 (validity, sort, segments)
        runs on a second stream while batch i forms its gradients and updates
        the table on the current one; two workspaces, events for the order.
        The results equal those of the one-call step, step by step."""
        import torch
        c, t = self.cfg, self.task
        main = torch.cuda.current_stream()
        b = lambda i: self.batches[i % len(self.batches)]
        if not hasattr(self, "_ovl_task"):
            if t == "ctr":
                B = max(x["label"].numel() for x in self.batches)
                mk = lambda: store.ctr_workspace(B, b(0)["keys"].numel() // b(0)["label"].numel())
            elif t == "kge":
                B = max(x["head"].numel() for x in self.batches)
                mk = lambda: store.kge_workspace(B, b(0)["neg"].numel() // b(0)["head"].numel())
            else:
                B = max(x["centre"].numel() for x in self.batches)
                mk = lambda: store.sgns_workspace(B, c.window, c.n_neg)
            self._ovl_task = (torch.cuda.Stream(), [mk(), mk()], [torch.cuda.Event(), torch.cuda.Event()],
                              [torch.cuda.Event(), torch.cuda.Event()])
        side, ws, prepared, applied = self._ovl_task
        if t == "ctr":
            F = b(0)["keys"].numel() // b(0)["label"].numel()
            prep = lambda x, w, st: store.step_ctr_prepare(x["keys"], F, w, stream=st)
            app = lambda x, w, st: store.step_ctr_apply(x["keys"], x["label"], w, loss=loss, stream=st)
        elif t == "kge":
            prep = lambda x, w, st: store.step_kge_prepare(x["head"], x["rel"], x["tail"], x["neg"], c.n_ent, w,
                                                           stream=st)
            app = lambda x, w, st: store.step_kge_apply(x["head"], x["rel"], x["tail"], x["neg"], c.n_head_neg,
                                                        c.n_ent, w, loss=loss, stream=st)
        else:
            prep = lambda x, w, st: store.step_sgns_prepare(x["centre"], x["ctx"], x["neg"], c.window, c.vocab, w,
                                                            stream=st)
            app = lambda x, w, st: store.step_sgns_apply(x["centre"], x["ctx"], x["neg"], c.window, c.vocab, w,
                                                         loss=loss, stream=st)
        side.wait_stream(main)
        prep(b(first), ws[0], side)
        prepared[0].record(side)
        for k in range(count):
            main.wait_event(prepared[k % 2])
            app(b(first + k), ws[k % 2], main)
            applied[k % 2].record(main)
            if after_step is not None:
                after_step(k)
            if k + 1 < count:
                if k >= 1:
                    side.wait_event(applied[(k + 1) % 2])   # that workspace's apply is done
                prep(b(first + k + 1), ws[(k + 1) % 2], side)
                prepared[(k + 1) % 2].record(side)

    def run_overlapped(self, store, first, count, loss, after_step=None):
        """MF steps first .. first+count-1 with the two-phase step: the key work
        of batch i+1 (sort, segments, records) runs on a second stream while
        batch i updates the table on the current one; two workspaces, events
        for the order.  The results equal those of ps_step_mf step by step."""
        import torch
        c = self.cfg
        main = torch.cuda.current_stream()
        if not hasattr(self, "_ovl"):
            nB = self.batches[0]["row"].numel()
            self._ovl = (torch.cuda.Stream(), [store.mf_workspace(nB), store.mf_workspace(nB)],
                         [torch.cuda.Event(), torch.cuda.Event()], [torch.cuda.Event(), torch.cuda.Event()],
                         torch.cuda.Event())
            self._ovl[4].record(main)   # creates the event, whose handle the library records into
        side, ws, prepared, applied, rows_done = self._ovl
        b = lambda i: self.batches[i % len(self.batches)]
        side.wait_stream(main)
        store.step_mf_prepare(b(first)["row"], b(first)["col"], b(first)["val"], c.n_rows, ws[0], stream=side)
        prepared[0].record(side)
        for k in range(count):
            bt = b(first + k)
            main.wait_event(prepared[k % 2])
            store.step_mf_apply(bt["row"].numel(), c.lam, ws[k % 2], loss=loss, stream=main, rows_done=rows_done)
            applied[k % 2].record(main)
            if after_step is not None:
                after_step(k)
            if k + 1 < count:
                nx = b(first + k + 1)
                if k >= 1:
                    side.wait_event(applied[(k + 1) % 2])
                side.wait_event(rows_done)   # overlap the column-key merge, not the row-key merge
                store.step_mf_prepare(nx["row"], nx["col"], nx["val"], c.n_rows, ws[(k + 1) % 2], stream=side)
                prepared[(k + 1) % 2].record(side)

    def alg_bytes(self, i):
        """Algorithmic (useful) bytes per launch of the merge kernel(s) and of
        the task-gradient kernel for batch i; shared per-unit rows count once."""
        c, bt = self.cfg, self.host_batches[i % len(self.host_batches)]
        n, U, R = self.occ[i % len(self.occ)], self.uniq[i % len(self.uniq)], self.R
        # per distinct key: W read and written, and G (a row, or one value when row-wise)
        RV = self.RV
        tab = 2.0 * RV + 8.0 if self.rowwise else 2.0 * RV + 2.0 * R
        table = tab * U
        if self.task == "mf" and self.unmerged:
            # gradient rows: row, col, val in, each distinct key's row read once, two
            # gradient rows out per entry; unmerged update: every gradient row read and
            # each distinct key's W and G read and written once
            B = bt.row.size
            return {"async": n * R + tab * U, "taskgrad": B * 12.0 + U * RV + 2.0 * B * R}
        if self.task == "mf":
            B = bt.row.size
            Ucol = np.unique(bt.col).size
            Urow = U - Ucol
            # row-key merge: a 16-byte record per entry, the entry's column row (one read per
            # distinct column key), the column-occurrence gradient row out, and the row keys'
            # W and G; column-key merge: the stored gradient rows and the column keys' W and G;
            # record scatter: col, val, two ranks in, one record out
            return {"rowmerge": B * (16.0 + R) + Ucol * RV + tab * Urow,
                    "segreduce": B * R + tab * Ucol,
                    "taskgrad": B * (4.0 + 4.0 + 8.0 + 16.0)}
        if self.task == "ctr":
            # gradient rows in occurrence order, read by the merge through the sort permutation
            B, F = bt.keys.shape
            return {"segreduce": n * (4.0 + R) + table,
                    "taskgrad": B * (4.0 + F * (8.0 + R + R))}
        if self.task == "ctr_wd":
            # "mlp" counts flops of the fp64 products, not bytes
            return {"segreduce": n * R + table, "mlp": self.mlp_flops(bt.keys.shape[0])}
        if self.task == "kge":
            B, nn = bt.neg.shape
            return {"segreduce": n * 4.0 + 3 * B * R + B * nn * 8.0 + 2 * B * 2 * R + table,
                    "taskgrad": B * (12.0 + 4 * nn + (3 + nn) * R + 3 * R + 4 * R + 8 * nn)}
        B = bt.centre.size                       # sgns
        pairs = int((bt.ctx >= 0).sum())
        out_occ = pairs * (1 + c.n_neg)
        return {"segreduce": n * 4.0 + out_occ * 8.0 + 2 * B * R + table,
                "taskgrad": B * (4.0 + 4 * bt.ctx.shape[1] * (1 + c.n_neg)) + (B + out_occ) * R + B * R
                            + out_occ * 8.0}

    def input_bytes(self, i):
        """Bytes of the step's batch as the caller hands it over (ids, values,
        labels)."""
        bt = self.host_batches[i % len(self.host_batches)]
        return float(sum(v.nbytes for v in bt.__dict__.values()))

    def sec8_bytes(self, i):
        """Algorithmic bytes of the fused step (the batch's inputs read once,
        then per distinct key its value and accumulator rows read and
        written once: inputs + 4 U R for per-element AdaGrad) and each
        kernel's share of them: the inputs it reads plus the keys it
        updates.  Gradient rows, records, gathers of rows for the task
        arithmetic and sort traffic are the implementation's, not in these
        bytes (they are in alg_bytes)."""
        c, bt = self.cfg, self.host_batches[i % len(self.host_batches)]
        U, R, RV = self.uniq[i % len(self.uniq)], self.R, self.RV
        tab = 2.0 * RV + 8.0 if self.rowwise else 2.0 * RV + 2.0 * R
        inp = self.input_bytes(i)
        out = {"step": inp + tab * U, "inputs": inp, "per_key": tab, "U": U}
        if self.task == "mf" and self.unmerged:
            out.update({"async": tab * U, "taskgrad": inp})
        elif self.task == "mf":
            Ucol = np.unique(bt.col).size
            out.update({"rowmerge": inp + tab * (U - Ucol), "segreduce": tab * Ucol, "taskgrad": inp})
        elif self.task == "ctr_wd":
            out.update({"segreduce": tab * U, "mlp": self.mlp_flops(bt.keys.shape[0])})
        else:
            out.update({"segreduce": tab * U, "taskgrad": inp})
        return out

    def oracle_args(self, bt):
        c = self.cfg
        return {"mf": lambda: (bt.row, bt.col, bt.val, c.n_rows, c.lam),
                "kge": lambda: (bt.head, bt.rel, bt.tail, bt.neg, c.n_head_neg, c.n_ent),
                "sgns": lambda: (bt.centre, bt.ctx, bt.neg, c.window, c.vocab),
                "ctr": lambda: (bt.keys, bt.label)}[self.task]()

    def threadable(self):
        """Whether the oracle step has a threaded form (step_threads): the
        per-element fp32 steps of the four tasks, merged."""
        return self.task in ("mf", "kge", "sgns", "ctr") and not (self.rowwise or self.unmerged
                                                                  or self.values == "bf16")

    def oracle_step(self, W, G, i, threads=1):
        import oracle
        c, bt = self.cfg, self.wl.batch(i)
        lr, eps = c.opt.lr, c.opt.eps
        if threads > 1 and self.threadable():
            oracle.step_threads(self.task, W, G, self.oracle_args(bt), lr, eps, threads)
            return self.keys_of(bt).size
        if self.values == "bf16":
            oracle.step_mf_bf16(W, G, bt.row, bt.col, bt.val, c.n_rows, c.lam, lr, eps)
            return self.keys_of(bt).size
        if self.task == "ctr_wd":
            from oracle.widedeep import step_ctr_wd
            if not hasattr(self, "_dense_host"):
                self._dense_host = self.dense0.copy()
                self._acc_host = np.zeros_like(self._dense_host)
            step_ctr_wd(W, G, self._dense_host, self._acc_host, bt.keys, bt.label, c.emb_dim, c.deep, lr, eps)
            return self.keys_of(bt).size
        if self.rowwise:
            oracle.step_rowwise(self.task, W, G, self.oracle_args(bt), lr, eps)
        elif self.task == "mf" and self.unmerged:
            oracle.step_mf_sequential(W, G, bt.row, bt.col, bt.val, c.n_rows, c.lam, lr, eps)
        elif self.task == "mf":
            oracle.step_mf(W, G, bt.row, bt.col, bt.val, c.n_rows, c.lam, lr, eps)
        elif self.task == "kge":
            oracle.step_kge(W, G, bt.head, bt.rel, bt.tail, bt.neg, c.n_head_neg, c.n_ent, lr, eps)
        elif self.task == "sgns":
            oracle.step_sgns(W, G, bt.centre, bt.ctx, bt.neg, c.window, c.vocab, lr, eps)
        else:
            oracle.step_ctr(W, G, bt.keys, bt.label, lr, eps)
        return self.keys_of(bt).size


def key_ranges(wb):
    """First keys of the key ranges a staged store needs for this task (each
    key offset a step takes starts a range)."""
    c = wb.cfg
    if wb.task == "mf":
        return [0, c.n_rows]
    if wb.task == "kge":
        return [0, c.n_ent]
    if wb.task == "sgns":
        return [0, c.vocab]
    return [0]


def run_staged(args, wb, dev):
    """Steps on a staged store: each step advances the clock, runs the step
    and signals the intent of the batch `lookahead` steps ahead (its distinct
    keys, as a data loader would); rounds run on the library's thread.
    Returns the fields of the JSON line that differ from the in-HBM run."""
    import torch

    from paper_2206_00470_amd import StagedStore, _lib
    cfg, nb, L = wb.cfg, len(wb.batches), args.lookahead
    begin = key_ranges(wb)
    ends = begin[1:] + [cfg.num_keys]
    ukeys = [np.unique(wb.keys_of(bt)) for bt in wb.host_batches]
    per = [max(int(((u >= b) & (u < e)).sum()) for u in ukeys) for b, e in zip(begin, ends)]
    # room for the batches in flight: the active one, the one expiring, L ahead
    slots = [min(e - b, int((L + 2) * p * 1.05) + 64) for b, e, p in zip(begin, ends, per)]
    t0 = time.time()
    store = StagedStore(wb.W, begin, slots, cfg.opt.lr, cfg.opt.eps, device=dev)
    print(f"# staged store: {sum(slots)} slots for {cfg.num_keys} keys, home tables pinned in "
          f"{time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    for c in range(1, L + 1):
        store.intent(ukeys[(c - 1) % nb], c, c + 1)
    clock = [0]

    def step(i):
        store.advance_clock()
        clock[0] += 1
        wb.step(store, i, loss)
        store.intent(ukeys[(i + L) % nb], clock[0] + L, clock[0] + L + 1)

    store.set_timing(1 << _lib.PS_KERNEL_STAGE)
    store.auto(True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    store.auto(False)
    store.read_timing(_lib.PS_KERNEL_STAGE)   # reset
    st0 = store.stats()
    store.auto(True)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t
    store.auto(False)
    assert store.error() == 0
    st1 = store.stats()
    mv_ms, mv_n = store.read_timing(_lib.PS_KERNEL_STAGE)
    moved = (st1["staged"] - st0["staged"]) + (st1["evicted"] - st0["evicted"])
    R = wb.R
    link_bytes = moved * 2.0 * R          # a value row and an accumulator row cross the link per move
    achieved = link_bytes / (mv_ms * 1e-3) / 1e9 if mv_ms > 0 else None
    store.close()
    staging = {"lookahead": L, "ranges": begin, "slots": slots, "home_GB": round(cfg.num_keys * 2 * R / 1e9, 2),
               "slots_GB": round(sum(slots) * 2 * R / 1e9, 2),
               "staged_per_step": (st1["staged"] - st0["staged"]) / args.steps,
               "evicted_per_step": (st1["evicted"] - st0["evicted"]) / args.steps,
               "forced_in_timed_steps": st1["forced"] - st0["forced"],
               "rounds_in_timed_steps": st1["rounds"] - st0["rounds"],
               "stalls_in_timed_steps": st1["stalled"] - st0["stalled"],
               "rate_estimate": round(st1["lambda"], 4),
               "host_planning_ms_per_round": round((st1["plan_us"] - st0["plan_us"]) / 1e3
                                                   / max(1, (st1["rounds"] - st0["rounds"]) + (st1["forced"] - st0["forced"])), 4),
               "host_planning_ms_per_step": round((st1["plan_us"] - st0["plan_us"]) / 1e3 / args.steps, 4),
               "link_GBps_over_step_time": round(link_bytes / elapsed / 1e9, 2),
               "move_kernel_ms_per_step": round(mv_ms / args.steps, 4)}
    roofline = {"bound": "host-link", "kernel": "k_move_rows", "achieved": round(achieved, 2) if achieved else None,
                "peak": HOST_LINK_GBPS, "unit": "GB/s", "frac": round(achieved / HOST_LINK_GBPS, 4) if achieved else None,
                "traffic": None, "avg_ms": round(mv_ms / max(mv_n, 1), 4),
                "alg_bytes_per_launch": int(link_bytes / max(mv_n, 1))}
    return elapsed, staging, roofline


def host_threads():
    """Threads for the all-core oracle: the cores this process may run on,
    capped by OMP_NUM_THREADS when that is set (the host share of one GPU)."""
    n = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS")
    if cap and cap.isdigit() and int(cap) > 0:
        n = min(n, int(cap))
    return max(1, n)


def cpu_baseline(args, wb, rowwise):
    """The oracle on the host on a bounded sample of the same workload (whole
    steps on the full table): single-threaded, and on all the host's cores
    (step_threads: gradients of unit ranges, then the merge of key ranges,
    one range per thread), each for about half of --cpu-seconds.  Also the
    host's memcpy bandwidth, for context."""
    if args.cpu_seconds <= 0:
        return None
    cfg = wb.cfg
    W = wb.W.copy()
    G = np.zeros(W.shape[0], np.float32) if rowwise else np.zeros_like(W)
    if wb.values == "bf16":
        import oracle
        W = oracle.f32_to_bf16(W)
    from threadpoolctl import threadpool_limits

    def run(threads, budget, first):
        done, rows, t0 = 0, 0, time.perf_counter()
        with threadpool_limits(threads):      # numpy's products (Wide & Deep) on as many threads
            while True:
                rows += 2 * wb.oracle_step(W, G, first + done, threads)
                done += 1
                if time.perf_counter() - t0 >= budget:
                    break
        t = time.perf_counter() - t0
        return rows / t, done, t

    T = host_threads()
    v1, n1, t1 = run(1, args.cpu_seconds / 2, 1000)
    res = {"value": v1, "unit": "rows/s", "cores": 1, "kind": "oracle",
           "sample": f"{n1} step(s) of the same workload on the full {cfg.num_keys}x{cfg.dim} table, "
                     f"single-threaded C oracle, {t1:.1f} s"}
    if T > 1 and (wb.threadable() or wb.task == "ctr_wd"):
        vT, nT, tT = run(T, args.cpu_seconds / 2, 2000)
        multi = {"value": vT, "unit": "rows/s", "cores": T, "kind": "oracle",
                 "sample": f"{nT} step(s) of the same workload on the full {cfg.num_keys}x{cfg.dim} table, the C "
                           f"oracle on {T} threads (unit ranges, then key ranges), {tT:.1f} s"}
        # the faster of the two is the baseline (small batches run faster on one thread)
        if vT >= v1:
            res = dict(multi, single_core=res)
        else:
            res = dict(res, all_cores=multi)
    a = np.ones(1 << 28, np.float32)
    b = np.empty_like(a)
    np.copyto(b, a)
    t0 = time.perf_counter()
    for _ in range(3):
        np.copyto(b, a)
    res["host_memcpy_GBps"] = round(3 * 2 * a.nbytes / (time.perf_counter() - t0) / 1e9, 1)
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the store is a single-device build and --gpus {args.gpus} "
              "is not supported (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2206_00470_amd import Store, _lib

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    t0 = time.time()
    nb = max(1, args.steps + args.warmup)        # a distinct batch for every warm-up and timed step
    rowwise = args.update == "rowwise"
    unmerged = args.update == "async"
    bf16 = args.values == "bf16"
    if unmerged and (bf16 or args.staged or not args.workload.startswith("mf")):
        print("--update async runs the MF workloads on fp32 values, in HBM", file=sys.stderr)
        sys.exit(2)
    if bf16 and (rowwise or args.staged or not args.workload.startswith("mf")):
        print("--values bf16 runs the MF workloads with per-element AdaGrad, in HBM", file=sys.stderr)
        sys.exit(2)
    if args.rank and (not args.workload.startswith("mf") or (args.rank > 512 and not args.ops_only)):
        print("--rank applies to the MF workloads; ranks above 512 need --ops-only (pull and push only)",
              file=sys.stderr)
        sys.exit(2)
    wb = Bench(args.workload, dev, nb, rowwise, args.values, unmerged, rank=args.rank)
    cfg = wb.cfg
    metric = ("param rows pulled+pushed/sec (MF 10m x 1m, rank 100)" if args.workload == "mf"
              else f"param rows pulled+pushed/sec ({cfg.name})")
    if args.staged:
        if rowwise or args.graph:
            print("--staged runs per-element AdaGrad, eagerly", file=sys.stderr)
            sys.exit(2)
        elapsed, staging, roofline = run_staged(args, wb, dev)
        occ = float(np.mean([wb.occ[(args.warmup + i) % nb] for i in range(args.steps)]))
        ms_per_step = elapsed * 1e3 / args.steps
        line = {
            "metric": metric + ", home table in host memory", "value": 2.0 * occ / (ms_per_step * 1e-3),
            "unit": "rows/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "f32", "data": "synthetic",
            "config": {"workload": cfg.name, "num_keys": cfg.num_keys, "dim": cfg.dim, "update": "elementwise",
                       "launch": "eager", "key_occurrences_per_step": occ, "batches_resident": nb,
                       "staging": staging},
            "roofline": roofline,
            "cpu_baseline": cpu_baseline(args, wb, False),
        }
        print(json.dumps(line), flush=True)
        return
    if bf16 and args.layout == "interleaved":
        from paper_2206_00470_amd.store import interleaved_bf16_tables
        Wt, Gt = interleaved_bf16_tables(torch.from_numpy(wb.W).to(dev))
    elif bf16:
        Wt = torch.from_numpy(wb.W).to(dev).to(torch.bfloat16)   # nearest, ties to even
        Gt = torch.zeros(wb.W.shape, dtype=torch.float32, device=dev)
    elif rowwise and args.layout == "interleaved":
        from paper_2206_00470_amd.store import padded_rowwise_table
        Wt, Gt = padded_rowwise_table(torch.from_numpy(wb.W).to(dev))
    elif rowwise:
        Wt = torch.from_numpy(wb.W).to(dev)
        Gt = torch.zeros(cfg.num_keys, dtype=torch.float32, device=dev)
    elif args.layout == "interleaved":
        from paper_2206_00470_amd.store import interleaved_tables
        Wt, Gt = interleaved_tables(torch.from_numpy(wb.W).to(dev))
    else:
        Wt = torch.from_numpy(wb.W).to(dev)
        Gt = torch.zeros_like(Wt)
    store = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    print(f"# setup {time.time() - t0:.1f}s: {cfg.name}, table {cfg.num_keys}x{cfg.dim}, {nb} batches resident",
          file=sys.stderr, flush=True)

    ops = {}
    if args.ops_only:
        ops = measure_ops(args, wb, store, dev, rowwise, unmerged)
        copy = calibrate_copy(dev) if args.calibrate_copy else None
        print(json.dumps({"metric": "push / pull alone (" + cfg.name + ")", "ops": ops, "copy_calibration": copy}),
              flush=True)
        store.close()
        return

    KID = {"segreduce": _lib.PS_KERNEL_SEGREDUCE, "taskgrad": _lib.PS_KERNEL_TASKGRAD,
           "rowmerge": _lib.PS_KERNEL_MF_ROWMERGE, "scatter": _lib.PS_KERNEL_SCATTER, "mlp": _lib.PS_KERNEL_MLP,
           "async": _lib.PS_KERNEL_ASYNC}
    names = list(wb.alg_bytes(0))                 # kernels with algorithmic bytes for this workload

    # (MF tiny is launch-bound: the overlap's second stream costs more than it hides, eagerly and in a
    # graph replay, 0.063 -> 0.078 ms; skip-gram's key sort already ends beside its 5.7 ms gradient
    # kernel, and overlapping it with the merges instead gained nothing: 11.62 -> 11.73 ms)
    overlap = not args.no_overlap and not unmerged and (
        (args.workload in ("mf", "mf_colorder") and not args.graph) or wb.task in ("ctr", "kge"))
    run_ovl = wb.run_overlapped_task if wb.task in ("ctr", "kge", "sgns") else wb.run_overlapped

    def run_steps(first, count, mask, marks=None):
        """count steps from batch `first` with the kernels in `mask` bracketed by HIP
        events (and, with marks, an event on the current stream after each step);
        returns host seconds and {name: (total ms, launches)}."""
        for k in KID.values():
            store.read_timing(k)                  # reset
        store.set_timing(mask)
        torch.cuda.synchronize()
        if marks is not None:
            marks[0].record()
        t = time.perf_counter()
        if overlap:
            run_ovl(store, first, count, loss,
                              after_step=(lambda k: marks[k + 1].record()) if marks is not None else None)
        else:
            for i in range(count):
                wb.step(store, first + i, loss)
                if marks is not None:
                    marks[i + 1].record()
        torch.cuda.synchronize()
        secs = time.perf_counter() - t
        store.set_timing(False)
        assert store.error() == 0
        return secs, {name: store.read_timing(k) for name, k in KID.items()}

    # warm-up steps, then the per-kernel breakdown: a few steps with every big
    # kernel timed (instrumentation only, not part of the timed figure; run on
    # batches after the timed ones), which also pick the dominant kernel
    run_steps(0, args.warmup, 0)
    nprof = max(1, min(args.steps, 5))
    _, kt_all = run_steps(args.warmup + args.steps, nprof, _lib.PS_TIMING_ALL)
    dom = max(names, key=lambda k: kt_all[k][0])

    # ------------------------------------------------------------ timed steps
    # Each HIP event costs the GPU a few microseconds, so only the dominant
    # kernel is bracketed while the step time is measured (plus one event per
    # step on the stream, for the median).
    step_ms = []
    if args.graph:
        # the same steps, captured once (the workspace is already sized) and replayed
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            if overlap:
                run_ovl(store, args.warmup, args.steps, loss)
            else:
                for i in range(args.steps):
                    wb.step(store, args.warmup + i, loss)
        g.replay()                          # untimed first replay
        torch.cuda.synchronize()
        t = time.perf_counter()
        g.replay()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t
        assert store.error() == 0
        # four more replays, each timed with events: the median replay per step
        for _ in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            step_ms.append(e0.elapsed_time(e1) / args.steps)
        step_ms.append(elapsed * 1e3 / args.steps)
    else:
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        elapsed, kt = run_steps(args.warmup, args.steps, 1 << KID[dom], marks)
        step_ms = [marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)]
    launches = launches_per_step(wb, store, args.warmup, loss)

    idx = [args.warmup + i for i in range(args.steps)]
    idx_prof = [args.warmup + args.steps + i for i in range(nprof)]
    occ = float(np.mean([wb.occ[i % nb] for i in idx]))
    U_avg = float(np.mean([wb.uniq[i % nb] for i in idx]))
    ms_per_step = elapsed * 1e3 / args.steps
    rows_per_s = 2.0 * occ / (ms_per_step * 1e-3)
    # launches per step of the merge kernel: SGNS merges output rows, then input rows
    # (MF's row-key merge is timed on its own, "rowmerge")
    seg_launches_per_step = 2 if wb.task == "sgns" else 1

    def kernel_entry(name, timing, steps, bidx):
        ms, cnt = timing
        kbytes = float(np.mean([wb.alg_bytes(i)[name] for i in bidx]))
        sbytes = float(np.mean([wb.sec8_bytes(i)[name] for i in bidx]))
        per_step_ms = ms / max(steps, 1)
        return {"avg_ms": ms / max(cnt, 1), "ms_per_step": per_step_ms, "launches": cnt,
                "alg_bytes_per_step": sbytes,
                "alg_GBps": sbytes / (per_step_ms * 1e-3) / 1e9 if cnt else None,
                "kernel_bytes_per_step": kbytes,
                "kernel_GBps": kbytes / (per_step_ms * 1e-3) / 1e9 if cnt else None,
                "launches_per_step": seg_launches_per_step if name == "segreduce" else
                (3 * len(wb.cfg.deep) if name == "mlp" else 1)}

    kernels = {name: kernel_entry(name, kt_all[name], nprof, idx_prof) for name in names}
    # from the timed steps (graph mode: from the eager breakdown steps)
    dk = kernels[dom] if args.graph else kernel_entry(dom, kt[dom], args.steps, idx)
    kernels["scatter"] = {"ms_per_step": kt_all["scatter"][0] / nprof, "launches": kt_all["scatter"][1]}
    symbol = {"segreduce": "k_segreduce<%s>" % {"mf": "SrcSorted", "kge": "SrcKGE", "sgns": "SrcSGNS",
                                                 "ctr": "SrcIndirect", "ctr_wd": "SrcSorted"}[wb.task],
              "rowmerge": "k_segreduce<SrcMFRow>", "mlp": "k_gemm_f64", "async": "k_push_async",
              "taskgrad": {"mf": "k_mf_grad_rows" if unmerged else "k_mf_pack", "kge": "k_kge_grad", "sgns": "k_sgns_grad",
                           "ctr": "k_ctr_grad", "ctr_wd": "k_wd_head"}[wb.task]}[dom]
    traffic = counter_traffic(args.workload + ("_rowwise" if rowwise else "") + ("_bf16" if bf16 else "")
                              + ("_async" if unmerged else ""), symbol)
    lpl = dk["launches_per_step"]
    alg_launch = dk["alg_bytes_per_step"] / lpl
    step_alg = float(np.mean([wb.sec8_bytes(i)["step"] for i in idx]))
    roofline = {
        "bound": "hbm",
        "kernel": symbol,
        "achieved": round(dk["alg_GBps"], 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(dk["alg_GBps"] / HBM_PEAK_GBPS, 4),
        "traffic": int(traffic) if traffic else None,
        "traffic_over_alg": round(traffic / alg_launch, 3) if traffic else None,
        "avg_ms": round(dk["avg_ms"], 4),
        "alg_bytes_per_launch": int(alg_launch),
        "alg_bytes": "the fused step's bytes (inputs read once, each distinct key's value and accumulator "
                     "rows read and written once) that this kernel accounts for: the inputs it reads and "
                     "the keys it updates",
        "kernel_bytes_per_launch": int(dk["kernel_bytes_per_step"] / lpl),
        "kernel_GBps": round(dk["kernel_GBps"], 1),
        "step": {"alg_bytes": int(step_alg), "GBps": round(step_alg / (ms_per_step * 1e-3) / 1e9, 1),
                 "frac": round(step_alg / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)},
    }
    if dom == "mlp":
        tf = dk["alg_GBps"] / 1e3            # "bytes" of the mlp entry are flops
        roofline = {"bound": "mfma", "kernel": symbol, "dtype": "f64", "achieved": round(tf, 2),
                    "peak": MFMA_F64_TFLOPS, "unit": "TFLOP/s", "frac": round(tf / MFMA_F64_TFLOPS, 4),
                    "traffic": None, "avg_ms": round(dk["avg_ms"], 4),
                    "alg_flops_per_launch": int(dk["alg_bytes_per_step"] / dk["launches_per_step"]),
                    "step": roofline["step"]}

    if not args.no_ops:
        ops = measure_ops(args, wb, store, dev, rowwise, unmerged)
        if wb.task == "sgns" and not bf16:
            ops["gather_ceiling"] = gather_ceilings(wb, store, dev, kernels, idx[0], ops.get("merge_distinct_keys"))
        elif wb.task in ("kge", "ctr") and not bf16:
            ops["gather_ceiling"] = task_gather_ceiling(wb, store, dev, kernels, idx[0])

    copy = calibrate_copy(dev) if args.calibrate_copy else None

    cpu = cpu_baseline(args, wb, rowwise)

    line = {
        "metric": metric + (", row-wise AdaGrad" if rowwise else "") + (", bf16 values" if bf16 else "")
                  + (", unmerged (asynchronous) updates" if unmerged else ""),
        "value": rows_per_s,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "median_ms_per_step": round(float(np.median(step_ms)), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64" if wb.task == "ctr_wd" else "f32",   # the Wide & Deep MLP runs in fp64
        "data": "synthetic",
        "config": {"workload": cfg.name, "num_keys": cfg.num_keys, "dim": cfg.dim, "layout": args.layout,
                   "update": args.update, "values": args.values,
                   "launch": "hip graph replay" if args.graph else "eager",
                   "next_key_work_overlapped": overlap,
                   "key_occurrences_per_step": occ, "avg_unique_keys_per_step": U_avg,
                   "batches_resident": nb, "distinct_batch_per_timed_step": nb >= args.warmup + args.steps,
                   "kernel_launches_per_step": launches},
        "roofline": roofline,
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kernels.items()},
        "kernels_from": f"{nprof} steps before the timed ones with every big kernel timed (the timed steps "
                        f"time only {dom})"
                        if not args.graph else f"{nprof} eager steps with every big kernel timed; the timed steps "
                                               f"are one HIP-graph replay",
        "median_from": "HIP events on the stream after each timed step" if not args.graph else
                       "the timed replay and four more, each over all steps",
        "ops": ops,
        "copy_calibration": copy,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    store.close()


def calibrate_copy(dev):
    """A 4 GiB device-to-device copy of known size: the reference for the HBM
    counters, and the copy bandwidth of this part."""
    import torch
    a = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    a.fill_(1.0)
    for _ in range(2):
        b.copy_(a)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    tcp = (time.perf_counter() - t1) / 5
    out = {"bytes_read": a.numel() * 4, "bytes_written": b.numel() * 4, "ms": round(tcp * 1e3, 4),
           "GBps": round(2 * a.numel() * 4 / tcp / 1e9, 1)}
    del a, b
    torch.cuda.empty_cache()
    return out


def launches_per_step(wb, store, i, loss):
    """Kernel launches of one step: the step captured into a HIP graph (not
    replayed) and its kernel nodes counted."""
    import ctypes as C

    import torch
    try:
        hip = C.CDLL("libamdhip64.so")
        wb.step(store, i, loss)           # eager first: the step's workspace exists before the capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph(keep_graph=True)
        with torch.cuda.graph(g):
            wb.step(store, i, loss)
        graph = C.c_void_p(g.raw_cuda_graph())
        n = C.c_size_t(0)
        if hip.hipGraphGetNodes(graph, None, C.byref(n)) != 0:
            return None
        nodes = (C.c_void_p * n.value)()
        if hip.hipGraphGetNodes(graph, nodes, C.byref(n)) != 0:
            return None
        kinds = C.c_int(0)
        count = 0
        for nd in nodes:
            if hip.hipGraphNodeGetType(C.c_void_p(nd), C.byref(kinds)) == 0 and kinds.value == 0:
                count += 1            # hipGraphNodeTypeKernel
        g.reset()
        torch.cuda.synchronize()
        return count
    except (OSError, RuntimeError, AttributeError):
        return None


def pipelined_push(store, keys, grads, n, reps):
    """Seconds per push of `reps` pushes back to back, the key work of push
    i+1 (ps_push_prepare, second stream, two workspaces) beside the merge
    of push i (ps_push_apply)."""
    import torch
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    ws = [store.push_workspace(n), store.push_workspace(n)]
    prepared = [torch.cuda.Event(), torch.cuda.Event()]
    applied = [torch.cuda.Event(), torch.cuda.Event()]

    def run(count):
        side.wait_stream(main)
        store.push_prepare(keys, ws[0], stream=side)
        prepared[0].record(side)
        for k in range(count):
            main.wait_event(prepared[k % 2])
            store.push_apply(n, grads, ws[k % 2], stream=main)
            applied[k % 2].record(main)
            if k + 1 < count:
                if k >= 1:
                    side.wait_event(applied[(k + 1) % 2])
                store.push_prepare(keys, ws[(k + 1) % 2], stream=side)
                prepared[(k + 1) % 2].record(side)

    run(2)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(main)
    run(reps)
    e1.record(main)
    torch.cuda.synchronize()
    assert store.error() == 0
    del ws
    return e0.elapsed_time(e1) * 1e-3 / reps


def measure_ops(args, wb, store, dev, rowwise, unmerged):
    """ps_push and ps_pull alone on one batch's key occurrences (random
    gradient rows), each rep timed with HIP events; reported as medians.
    Also the merge kernel alone on as many distinct random keys (the bare
    read-modify-write pattern), and with unmerged updates the unmerged push."""
    import torch

    from paper_2206_00470_amd import _lib
    cfg = wb.cfg
    bt = wb.wl.batch(100)
    keys_np = wb.keys_of(bt)
    n = int(keys_np.size)
    U = int(np.unique(keys_np).size)
    keys = torch.from_numpy(keys_np).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    grads = torch.randn((n, cfg.dim), generator=gen, dtype=torch.float32, device=dev)
    out = torch.empty((n, cfg.dim), dtype=torch.float32, device=dev)
    reps = 10

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record()
        for r in range(reps):
            fn()
            ev[r + 1].record()
        torch.cuda.synchronize()
        assert store.error() == 0
        return float(np.median([ev[r].elapsed_time(ev[r + 1]) for r in range(reps)])) * 1e-3

    tp = timed(lambda: store.push(keys, grads))
    tl = timed(lambda: store.pull(keys, out=out))
    tpp = pipelined_push(store, keys, grads, n, reps)
    R, RV = wb.R, wb.RV
    tab = 2.0 * RV + 8.0 if rowwise else 2.0 * RV + 2.0 * R
    push_alg = 8.0 * n + n * R + tab * U
    pull_alg = 8.0 * n + U * RV + n * R
    oc = counter_summary(args.workload + "_ops") if not (rowwise or unmerged or wb.values == "bf16") else None
    push_traffic = int(oc["push_hbm_bytes"]) if oc and "push_hbm_bytes" in oc else None
    ops = {
        "push": {"ms": round(tp * 1e3, 4), "rows_per_s": n / tp, "alg_GBps": round(push_alg / tp / 1e9, 1),
                 "frac_of_peak": round(push_alg / tp / 1e9 / HBM_PEAK_GBPS, 4), "occurrences": n, "unique_keys": U,
                 "roofline": {"bound": "hbm", "achieved": round(push_alg / tp / 1e9, 1), "peak": HBM_PEAK_GBPS,
                              "unit": "GB/s", "frac": round(push_alg / tp / 1e9 / HBM_PEAK_GBPS, 4),
                              "alg_bytes": int(push_alg), "traffic": push_traffic,
                              "traffic_over_alg": round(push_traffic / push_alg, 3) if push_traffic else None,
                              "what": "8 n (keys) + n R (gradient rows) + per distinct key its value and "
                                      "accumulator rows read and written, over the whole ps_push (sort, "
                                      "segments, merge, finalize)"}},
        "push_pipelined": {"ms": round(tpp * 1e3, 4), "rows_per_s": n / tpp,
                           "alg_GBps": round(push_alg / tpp / 1e9, 1),
                           "frac_of_peak": round(push_alg / tpp / 1e9 / HBM_PEAK_GBPS, 4),
                           "roofline": {"bound": "hbm", "achieved": round(push_alg / tpp / 1e9, 1),
                                        "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                        "frac": round(push_alg / tpp / 1e9 / HBM_PEAK_GBPS, 4),
                                        "alg_bytes": int(push_alg)},
                           "what": f"{reps} pushes back to back, each push's key work (ps_push_prepare) on a "
                                   "second stream beside the previous push's merge (ps_push_apply); time per push"},
        "pull": {"ms": round(tl * 1e3, 4), "rows_per_s": n / tl, "alg_GBps": round(pull_alg / tl / 1e9, 1),
                 "frac_of_peak": round(pull_alg / tl / 1e9 / HBM_PEAK_GBPS, 4)},
        "median_of": reps,
    }
    if unmerged:
        ta = timed(lambda: store.push_async(keys, grads))
        ops["push_async"] = {"ms": round(ta * 1e3, 4), "rows_per_s": n / ta,
                             "alg_GBps": round((n * R + tab * U) / ta / 1e9, 1)}
    if not args.ops_only and not unmerged:
        # the bare read-modify-write pattern through the merge kernel: U distinct
        # random keys, one contiguous gradient row each (no duplicates to merge)
        ukeys = torch.from_numpy(np.sort(np.random.default_rng(11).choice(cfg.num_keys, U, replace=False))).to(dev)
        ugrads = grads[:U]
        store.push(ukeys, ugrads)
        store.read_timing(_lib.PS_KERNEL_SEGREDUCE)
        store.set_timing(1 << _lib.PS_KERNEL_SEGREDUCE)
        for _ in range(reps):
            store.push(ukeys, ugrads)
        store.set_timing(False)
        mms, mcnt = store.read_timing(_lib.PS_KERNEL_SEGREDUCE)
        merge_ms = mms / max(mcnt, 1)
        rmw_alg = U * R + tab * U
        ops["merge_distinct_keys"] = {"keys": U, "merge_ms": round(merge_ms, 4),
                                      "alg_GBps": round(rmw_alg / (merge_ms * 1e-3) / 1e9, 1),
                                      "what": "merge kernel alone on a push of distinct random keys: W and G "
                                              "read-modify-write plus one gradient row per key"}
        del ukeys, ugrads
    del keys, grads, out
    torch.cuda.empty_cache()
    return ops


def probe_ms(store, keys_np, sink, dev, reps=10):
    """Median time (ms) of the gather probe over the row sequence keys_np."""
    import torch
    keys = torch.from_numpy(keys_np.astype(np.int32)).to(dev)
    for _ in range(2):
        store.probe_gather(keys, sink)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record()
    for r in range(reps):
        store.probe_gather(keys, sink)
        ev[r + 1].record()
    torch.cuda.synchronize()
    return float(np.median([ev[r].elapsed_time(ev[r + 1]) for r in range(reps)]))


def task_gather_ceiling(wb, store, dev, kernels, i):
    """ComplEx and CTR: the gradient kernel's row reads of batch i (ComplEx:
    per triple the head, relation and tail rows, then every negative's row;
    CTR: per sample its field rows, which the kernel reads twice, the second
    time from the caches) through the gather probe (median of 10), beside
    the rate the kernel reaches on them in the breakdown steps."""
    import torch

    from paper_2206_00470_amd import _lib
    c, bt = wb.cfg, wb.host_batches[i % len(wb.host_batches)]
    if wb.task == "kge":
        keys = np.concatenate([bt.head.astype(np.int64)[:, None], (c.n_ent + bt.rel.astype(np.int64))[:, None],
                               bt.tail.astype(np.int64)[:, None], bt.neg.astype(np.int64)], axis=1).ravel()
        what = "the ComplEx gradient kernel: per triple its head, relation and tail rows, then its negatives' rows"
    else:
        keys = bt.keys.astype(np.int64).ravel()
        what = "the CTR gradient kernel: per sample its field rows (read twice by the kernel, counted once)"
    sink = torch.empty(_lib.PS_PROBE_GRID, dtype=torch.float64, device=dev)
    t = probe_ms(store, keys, sink, dev) * 1e-3
    rows = int(keys.size)
    probe = rows * wb.R / t / 1e9
    kms = kernels.get("taskgrad", {}).get("ms_per_step")
    kgb = rows * wb.R / (kms * 1e-3) / 1e9 if kms else None
    return {"grad_stream": {"rows": rows, "probe_ms": round(t * 1e3, 4), "probe_GBps": round(probe, 1),
                            "kernel": "taskgrad", "kernel_ms": round(kms, 4) if kms else None,
                            "kernel_GBps": round(kgb, 1) if kgb else None,
                            "kernel_frac_of_probe": round(kgb / probe, 3) if kgb else None, "what": what},
            "what": "rows read per second by the gather probe (ps_probe_gather: the same reads without the "
                    "kernel's arithmetic) against the kernel's row bytes per second"}


def gather_ceilings(wb, store, dev, kernels, i, ops_mdk=None):
    """Skip-gram: how fast this part serves each of the step's two row-gather
    streams — the gradient kernel's output rows in centre order, and the
    output-key merge's centre rows in sorted output-key order — measured by
    the gather probe on the same row sequences of batch i (median of 10),
    beside the rate the step's kernels reach on them (their row bytes over
    their time per step in the breakdown steps)."""
    import torch

    from paper_2206_00470_amd import _lib
    c, bt = wb.cfg, wb.host_batches[i % len(wb.host_batches)]
    ctx = bt.ctx.astype(np.int64)
    present = ctx >= 0
    rows = np.concatenate([ctx[:, :, None], bt.neg.astype(np.int64)], axis=2)   # [B, slots, 1 + n_neg]
    out_keys = (c.vocab + rows[present]).ravel()            # per centre and present slot: context, negatives
    centre_of = np.repeat(np.broadcast_to(bt.centre.astype(np.int64)[:, None], ctx.shape)[present], rows.shape[2])
    order = np.argsort(out_keys, kind="stable")
    R = wb.R
    B = int(bt.centre.size)
    n_out = int(out_keys.size)
    streams = {"grad_stream": (out_keys, "taskgrad", "the gradient kernel: every output occurrence's row "
                                                      "(1.2 GB output table), centre after centre"),
               "merge_stream": (centre_of[order], "segreduce", "the output-key merge: each output "
                                                                "occurrence's centre input row, in sorted "
                                                                "output-key order")}
    sink = torch.empty(_lib.PS_PROBE_GRID, dtype=torch.float64, device=dev)
    out = {}
    for name, (keys_np, kname, what) in streams.items():
        t = probe_ms(store, keys_np, sink, dev) * 1e-3
        probe = n_out * R / t / 1e9
        # the gradient kernel also reads the B centre rows, the merge (its input-key
        # launch) the B stored centre gradient rows
        kms = kernels.get(kname, {}).get("ms_per_step")
        kgb = (n_out + B) * R / (kms * 1e-3) / 1e9 if kms else None
        out[name] = {"rows": n_out, "probe_ms": round(t * 1e3, 4), "probe_GBps": round(probe, 1),
                     "kernel": kname, "kernel_ms": round(kms, 4) if kms else None,
                     "kernel_GBps": round(kgb, 1) if kgb else None,
                     "kernel_frac_of_probe": round(kgb / probe, 3) if kgb else None, "what": what}
    # the merge also reads and writes each distinct output key's W and G rows,
    # which the probe does not: add that read-modify-write at the rate of the
    # merge kernel alone on distinct keys (ops.merge_distinct_keys)
    mdk = ops_mdk or {}
    if mdk.get("merge_ms") and out["merge_stream"]["kernel_ms"]:
        u_out = int(np.unique(out_keys).size)
        rmw_ms = mdk["merge_ms"] * u_out / mdk["keys"]
        ceil_ms = out["merge_stream"]["probe_ms"] + rmw_ms
        out["merge_stream"]["with_rmw"] = {
            "distinct_output_keys": u_out, "rmw_ms": round(rmw_ms, 4), "ceiling_ms": round(ceil_ms, 4),
            "kernel_frac_of_ceiling": round(ceil_ms / out["merge_stream"]["kernel_ms"], 3),
            "what": "probe time of the gathers plus the distinct-key merge's time scaled to the step's "
                    "distinct output keys, against the merge kernels' time per step"}
    out["what"] = ("rows read per second by the gather probe (ps_probe_gather: the same reads without the "
                   "kernels' arithmetic) against the kernels' row bytes per second")
    return out


if __name__ == "__main__":
    main()

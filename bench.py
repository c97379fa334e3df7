#!/usr/bin/env python3
"""Throughput of the sparse parameter-store training step on one MI355X.

Workload: matrix factorization of a synthetic 10,000,000 x 1,000,000 matrix
(rows uniform, columns Zipf 1.1), rank-100 fp32 factors with fp32 AdaGrad
accumulators (11M keys x 100, 8.8 GB of W+G in HBM), 1,048,576 entries per
step.  One step = ps_step_mf: key intake, stable radix sort of the 2,097,152
key occurrences, segment boundaries, per-entry gradients from the pulled
rows, fp64 per-key merge and the AdaGrad row update.

Prints one JSON line: rows pulled + pushed per second (2 x 2,097,152 row
accesses per step), the roofline of the dominant kernel measured with HIP
events during the timed steps, the push-only and pull-only rates, and the
CPU oracle timed on the host.
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="bound on the CPU-oracle sample (0 = skip)")
    ap.add_argument("--no-ops", action="store_true", help="skip the pull-only / push-only measurements")
    return ap.parse_args()


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2206_00470_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_traffic(kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "counters_mf_10Mx1M.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("source_hash") != source_hash():
        return None
    k = data.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the store is a single-device build and --gpus {args.gpus} "
              "is not supported (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2206_00470_amd import Store, _lib
    from paper_2206_00470_amd.workloads import MF_10Mx1M, MFWorkload, random_push

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cfg = MF_10Mx1M
    wl = MFWorkload(cfg)
    dev = torch.device("cuda:0")
    B = cfg.batch
    n = 2 * B
    R = 4 * cfg.dim

    t0 = time.time()
    W = wl.init_table()
    Wt = torch.from_numpy(W).to(dev)
    Gt = torch.zeros_like(Wt)
    store = Store(Wt, Gt, cfg.opt.lr, cfg.opt.eps)

    nb = max(1, min(args.steps + args.warmup, 8))
    batches, uniq = [], []
    for i in range(nb):
        bt = wl.batch(i)
        batches.append((torch.from_numpy(bt.row).to(dev), torch.from_numpy(bt.col).to(dev),
                        torch.from_numpy(bt.val).to(dev)))
        keys = np.concatenate([bt.row.astype(np.int64), cfg.n_rows + bt.col.astype(np.int64)])
        uniq.append(np.unique(keys).size)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    print(f"# setup {time.time() - t0:.1f}s: table {cfg.num_keys}x{cfg.dim}, {nb} batches resident",
          file=sys.stderr, flush=True)

    def step(i):
        r, c, v = batches[i % nb]
        store.step_mf(r, c, v, cfg.n_rows, cfg.lam, loss=loss)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    assert store.error() == 0

    # ------------------------------------------------------------ timed steps
    for k in range(4):
        store.read_timing(k)            # reset
    store.set_timing(True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    store.set_timing(False)
    assert store.error() == 0
    kt = {name: store.read_timing(k) for name, k in
          (("segreduce", _lib.PS_KERNEL_SEGREDUCE), ("taskgrad", _lib.PS_KERNEL_TASKGRAD),
           ("scatter", _lib.PS_KERNEL_SCATTER))}

    ms_per_step = elapsed * 1e3 / args.steps
    rows_per_s = 2.0 * n * args.steps / elapsed
    U_avg = float(np.mean([uniq[(args.warmup + i) % nb] for i in range(args.steps)]))

    # algorithmic bytes per launch (useful bytes only)
    alg = {
        # gradient rows read in sorted order + W and G read and written for each distinct key
        "segreduce": n * R + 4.0 * U_avg * R,
        # entry inputs + two gathered rows + two gradient rows written + two rank words
        "taskgrad": B * (12.0 + 2 * R + 2 * R + 8.0),
    }
    kernels = {}
    for name, nbytes in alg.items():
        ms, cnt = kt[name]
        avg_ms = ms / max(cnt, 1)
        kernels[name] = {"avg_ms": avg_ms, "launches": cnt, "alg_bytes": nbytes,
                         "alg_GBps": nbytes / (avg_ms * 1e-3) / 1e9 if cnt else None}
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"])
    dk = kernels[dom]
    kernel_symbol = {"segreduce": "k_segreduce", "taskgrad": "k_mf_grad"}[dom]
    roofline = {
        "bound": "hbm",
        "kernel": kernel_symbol,
        "achieved": round(dk["alg_GBps"], 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(dk["alg_GBps"] / HBM_PEAK_GBPS, 4),
        "traffic": counter_traffic(kernel_symbol),
        "avg_ms": round(dk["avg_ms"], 4),
        "alg_bytes_per_launch": int(dk["alg_bytes"]),
    }

    # ------------------------------------------------------------ push-only / pull-only
    ops = {}
    if not args.no_ops:
        keys_np, grads_np = random_push(cfg.num_keys, n, cfg.dim, 7)
        bt = wl.batch(100)
        keys_np = np.concatenate([bt.row.astype(np.int64)[:, None],
                                  cfg.n_rows + bt.col.astype(np.int64)[:, None]], axis=1).ravel()
        U = np.unique(keys_np).size
        keys = torch.from_numpy(keys_np).to(dev)
        grads = torch.from_numpy(grads_np).to(dev)
        del grads_np
        out = torch.empty((n, cfg.dim), dtype=torch.float32, device=dev)
        reps = 10
        for _ in range(2):
            store.push(keys, grads)
            store.pull(keys, out=out)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(reps):
            store.push(keys, grads)
        torch.cuda.synchronize()
        tp = (time.perf_counter() - t1) / reps
        t1 = time.perf_counter()
        for _ in range(reps):
            store.pull(keys, out=out)
        torch.cuda.synchronize()
        tl = (time.perf_counter() - t1) / reps
        assert store.error() == 0
        push_alg = 8.0 * n + n * R + 4.0 * U * R
        pull_alg = 8.0 * n + U * R + n * R
        ops = {
            "push": {"ms": round(tp * 1e3, 4), "rows_per_s": n / tp, "alg_GBps": round(push_alg / tp / 1e9, 1),
                     "frac_of_peak": round(push_alg / tp / 1e9 / HBM_PEAK_GBPS, 4), "unique_keys": int(U)},
            "pull": {"ms": round(tl * 1e3, 4), "rows_per_s": n / tl, "alg_GBps": round(pull_alg / tl / 1e9, 1)},
        }
        del keys, grads, out

    # ------------------------------------------------------------ CPU oracle on the host
    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        G = np.zeros_like(W)
        done, tc0 = 0, time.perf_counter()
        while True:
            bt = wl.batch(1000 + done)
            oracle.step_mf(W, G, bt.row, bt.col, bt.val, cfg.n_rows, cfg.lam, cfg.opt.lr, cfg.opt.eps)
            done += 1
            if time.perf_counter() - tc0 >= args.cpu_seconds:
                break
        tc = time.perf_counter() - tc0
        cpu = {"value": 2.0 * n * done / tc, "unit": "rows/s", "cores": 1, "kind": "oracle",
               "sample": f"{done} step(s) of {B} entries on the full {cfg.num_keys}x{cfg.dim} table, "
                         f"single-threaded C oracle, {tc:.1f} s"}

    line = {
        "metric": "param rows pulled+pushed/sec (MF 10m x 1m, rank 100)",
        "value": rows_per_s,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "num_keys": cfg.num_keys, "dim": cfg.dim,
                   "entries_per_step": B, "key_occurrences_per_step": n,
                   "avg_unique_keys_per_step": U_avg, "batches_resident": nb},
        "step_alg_GBps": round((B * 12.0 + 4.0 * U_avg * R) / (ms_per_step * 1e-3) / 1e9, 1),
        "roofline": roofline,
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kernels.items()},
        "ops": ops,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    store.close()


if __name__ == "__main__":
    main()

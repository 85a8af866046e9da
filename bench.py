#!/usr/bin/env python3
"""Throughput of sequentially-correct sparse SGD on one MI355X.

A step is one pass of the whole path over the workload, inputs resident in
HBM: conflict levels (pdb_schedule: transpose, previous writers, levels,
grouping) and one SGD epoch (pdb_sgd_epoch / pdb_mf_epoch), weights reset to
w0 at the start of the step (--epochs E: E epochs on the step's schedule;
--batch B: mini-batches of B examples; --delay D: bounded-delay SGD; --dense W:
full-batch gradient descent on dense workload W, one step = the workload's
iterations).  `value` = stored entries updated per second over the K timed
steps (ratings per second for matrix completion; example-feature pairs times
iterations for dense gradient descent).

Default workload: 10M examples x 1M features, 50 entries per example with
Zipf(1.2) feature ids, binary values, logistic loss, lr 0.01.

Prints one JSON line.  `roofline` prices the dominant kernel (the epoch)
against HBM bandwidth with its algorithmic bytes; `cpu_baseline` times the
CPU oracle on a bounded prefix of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

_ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, _ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "sequentially-correct nnz-updates/sec per epoch + achieved HBM GB/s fraction"


def algorithmic_bytes(g, L, mf=False, U=None, nb=None):
    """Bytes one epoch must move at least once.  Mini-batches (U union
    entries over nb batches): each stored entry's column (and value) once, each
    example's row bound and label, each union feature's weight read and
    written once, and the batch order."""
    if U is not None:
        per_nz = 4 + (4 if g["val"] is not None else 0)
        return g["nnz"] * per_nz + g["n"] * (8 + 4) + U * 8 + nb * (4 + 8) + L * 8
    if mf:
        # per rating: user, item, rating, perm (16 B) + read and write of a
        # 128-byte user row and a 128-byte item row (512 B); level_ptr per level
        return g["n"] * (16 + 512) + L * 8
    per_nz = 4 + 8 + (4 if g["val"] is not None else 0)   # col, w read + write, val
    per_ex = 8 + 4 + 4                                      # row_ptr, y, perm
    return g["nnz"] * per_nz + g["n"] * per_ex + L * 8


def source_digest(batch=False, stale=False, dense=False):
    """Digest of the sources of the priced epoch kernel: a traffic record
    taken on other sources is not reported."""
    h = hashlib.sha256()
    main = "dense.hip" if dense else ("stale.hip" if stale else ("batch.hip" if batch else "apply.hip"))
    for f in (main, "pdb_math.h", "pdb_words.h", "pdb_internal.h"):
        with open(os.path.join(_ROOT, "paper_1508_00703_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic(workload, digest):
    """HBM bytes per epoch launch from the committed counter summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(_ROOT, "profiles", "traffic_%s.md" % workload)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if line.startswith("traffic_json:"):
            vals = json.loads(line.split(":", 1)[1])
    if vals.get("source_digest") != digest:
        return None
    return vals.get("hbm_bytes_per_launch")


def trimmed_mean(xs):
    xs = sorted(xs)
    if len(xs) >= 10:
        xs = xs[2:-2]
    return sum(xs) / len(xs)


def cpu_baseline(g, cfg_id, budget_s, gpu_levels=None, batch=0, delay=-1):
    """The oracle (one-pass levels + grouping + natural-order epoch), single
    thread, on the first rows of the same workload (with batch > 0: batch
    levels + grouping + the mini-batch epoch)."""
    import numpy as np

    import oracle

    mf = cfg_id == 5

    def run(rows):
        rp = g["row_ptr"][:rows + 1]
        col = g["col"][:rp[-1]]
        t0 = time.perf_counter()
        if delay >= 0:
            oracle.prev_writer(rp, col, g["d"])
            val = None if g["val"] is None else g["val"][:rp[-1]]
            oracle.stale_epoch(rp, col, val, g["y"][:rows], np.zeros(g["d"], np.float32), g["lr"],
                               g["loss"], oracle.NATURAL, delay)
            return time.perf_counter() - t0, int(rp[-1]), None
        if batch:
            level, perm, level_ptr, L = oracle.batch_schedule(rp, col, g["d"], batch)
            val = None if g["val"] is None else g["val"][:rp[-1]]
            oracle.batch_epoch(rp, col, val, g["y"][:rows], np.zeros(g["d"], np.float32), g["lr"],
                               g["loss"], oracle.NATURAL, batch)
            return time.perf_counter() - t0, int(rp[-1]), level
        level, perm, level_ptr, L = oracle.schedule(rp, col, g["d"])
        if mf:
            oracle.mf_epoch(g["user"][:rows], g["item"][:rows], g["rating"][:rows], g["U0"],
                            g["V0"], g["lr"], g["reg"], oracle.NATURAL)
        else:
            val = None if g["val"] is None else g["val"][:rp[-1]]
            oracle.sgd_epoch(rp, col, val, g["y"][:rows], np.zeros(g["d"], np.float32), g["lr"],
                             g["loss"], oracle.NATURAL)
        return time.perf_counter() - t0, int(rp[-1]), level

    n = g["n"]
    probe = min(n, 20000)
    t, _, _ = run(probe)
    rows = int(min(n, max(probe, probe * budget_s / max(t, 1e-6))))
    if batch:
        rows = min(n, max(batch, rows // batch * batch))  # whole batches
    t, nnz_s, level = run(rows)
    units = rows if mf else nnz_s
    res = {"value": units / t, "unit": "ratings/s" if mf else "nnz-updates/s", "cores": 1,
           "kind": "oracle",
           "sample": "first %d of %d %s (%d stored entries), %s + natural-order %sepoch, "
                     "%.1f s" % (
                         rows, n, "ratings" if mf else "examples", nnz_s,
                         "previous writers" if delay >= 0 else
                         "one-pass %slevels + grouping" % ("batch " if batch else ""),
                         "mini-batch (B=%d) " % batch if batch else
                         ("delay-%d " % delay if delay >= 0 else ""), t),
           "host_cpu": platform.processor() or platform.machine()}
    if gpu_levels is not None and level is not None:
        k = len(level) if batch else rows
        res["sample_levels_equal_gpu"] = bool(np.array_equal(gpu_levels[:k], level[:k]))
    return res


DENSE_LDS_FLOATS = 36864  # the tile stays in LDS when cb + rb (rounded to 4) + rb cb fit


def dense_cpu_baseline(g, budget_s):
    """The oracle's natural-order full-batch gradient descent, single thread,
    on the whole matrix for as many iterations as fit the budget."""
    import numpy as np

    import oracle

    w0 = np.zeros(g["d"], np.float32)
    t0 = time.perf_counter()
    oracle.dense_gd(g["X"], g["y"], w0, g["lr"], g["loss"], oracle.NATURAL, 1)
    t1 = time.perf_counter() - t0
    iters = int(max(1, min(g["iters"], budget_s / max(t1, 1e-6))))
    t0 = time.perf_counter()
    oracle.dense_gd(g["X"], g["y"], w0, g["lr"], g["loss"], oracle.NATURAL, iters)
    t = time.perf_counter() - t0
    return {"value": g["n"] * g["d"] * iters / t, "unit": "nnz-updates/s", "cores": 1,
            "kind": "oracle",
            "sample": "all %d x %d entries, %d of %d iterations, natural order, %.1f s" % (
                g["n"], g["d"], iters, g["iters"], t),
            "host_cpu": platform.processor() or platform.machine()}


def run_dense(args):
    """Dense full-batch gradient descent: a step is one pdb_dense_gd call of
    the workload's iterations from w = 0."""
    import numpy as np
    import torch

    import datagen
    from paper_1508_00703_amd import native

    native.load()
    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    g = datagen.generate_dense(args.dense)
    print("generated %s: %d x %d in %.1f s" % (g["name"], g["n"], g["d"], time.perf_counter() - t0),
          file=sys.stderr, flush=True)
    n, d, iters = g["n"], g["d"], g["iters"]
    X = torch.from_numpy(np.ascontiguousarray(g["X"])).to(dev)
    y = torch.from_numpy(g["y"]).to(dev)
    w = torch.zeros(d, dtype=torch.float32, device=dev)
    rb, cb = native.pdb_dense_plan(n, d)
    ws = native.workspace(native.pdb_dense_workspace_bytes(n, d, rb, cb), dev)
    resident = cb + ((rb + 3) // 4) * 4 + rb * cb <= DENSE_LDS_FLOATS
    stream = torch.cuda.current_stream(dev)
    ev = []

    def step(timed):
        w.zero_()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        native.pdb_dense_gd(X, y, w, float(g["lr"]), g["loss"], iters, rb, cb, ws=ws)
        b.record(stream)
        if timed:
            ev.append((a, b))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    if native.pdb_workspace_status(ws) != native.PDB_OK:
        raise SystemExit("device-side failure during warmup")
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(True)
        print("step %d done" % k, file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if native.pdb_workspace_status(ws) != native.PDB_OK:
        raise SystemExit("device-side failure during the timed steps")
    call_ms = [a.elapsed_time(b) for a, b in ev]
    ms = trimmed_mean(call_ms)
    # bytes the algorithm must move per call: X once when its tiles stay on
    # chip, else X twice per iteration (the dot products need every column of
    # the new weights, the gradient every row's step); y once, w read + written
    xbytes = 4 * n * d * (1 if resident else 2 * iters)
    abytes = xbytes + 4 * n + 8 * d
    achieved = abytes / (ms * 1e-3) / 1e9
    workload = "dense%d" % args.dense
    digest = source_digest(dense=True)
    out = {
        "metric": METRIC,
        "value": n * d * iters * args.steps / elapsed,
        "unit": "nnz-updates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "%s: %s, %d iterations of full-batch gradient descent" % (
                       workload, g["name"], iters),
                   "n": n, "d": d, "iters": iters, "seed": g["seed"], "row_block": rb,
                   "col_block": cb, "workers": -(-n // rb) * -(-d // cb),
                   "tile": "resident in LDS" if resident else "streamed every iteration"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": read_traffic(workload, digest),
                     "kernel": "k_dense_gd (all iterations)", "algorithmic_bytes": abytes,
                     "call_ms": ms, "call_ms_all": call_ms, "source_digest": digest,
                     "us_per_iteration": ms * 1e3 / max(iters, 1)},
        "epoch_ms": ms,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = dense_cpu_baseline(g, args.cpu_budget)
    print(json.dumps(out))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--epochs", type=int, default=1,
                    help="epochs per step on the step's one schedule (the schedule is cached)")
    ap.add_argument("--delay", type=int, default=-1,
                    help="bounded-delay SGD (pdb_stale_epoch) with this delay; -1 = sequential")
    ap.add_argument("--batch", type=int, default=0,
                    help="mini-batch gradient descent with this many examples per batch "
                         "(pdb_batch_schedule + pdb_batch_epoch); 0 = SGD")
    ap.add_argument("--dense", type=int, default=0, choices=[0, 1, 2],
                    help="full-batch gradient descent on dense workload 1 (5000 x 960, "
                         "200 iterations) or 2 (500 x 1M, 50 iterations); 0 = sparse")
    ap.add_argument("--method", type=int, default=0,
                    help="0 auto, 1 chain-scan, 2 dataflow, 3 spine")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES of device memory once (a plain copy kernel of known "
                         "size, for scaling HBM traffic counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the path does not shard across GPUs "
              "(see DESIGN.md, 'More than one GPU'); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copied_bytes": src.numel() * 4}))
        return

    if args.dense:
        run_dense(args)
        return

    import datagen
    from paper_1508_00703_amd import native

    native.load()
    dev = torch.device("cuda:0")
    cfg_id = args.config
    mf = cfg_id == 5
    batch = args.batch
    delay = args.delay
    if (batch or delay >= 0) and mf:
        raise SystemExit("--batch and --delay apply to the sparse SGD workloads (configs 1-4)")
    if batch and delay >= 0:
        raise SystemExit("--batch and --delay are separate workloads")
    t0 = time.perf_counter()
    g = datagen.generate_mf(cfg_id) if mf else datagen.generate(cfg_id)
    t_gen = time.perf_counter() - t0
    print("generated %s: n=%d nnz=%d in %.1f s" % (g["name"], g["n"], g["nnz"], t_gen),
          file=sys.stderr, flush=True)

    if batch:
        # the workload's mini-batch form: lr / B, the step of the batch's mean gradient
        g = dict(g)
        g["lr"] = np.float32(g["lr"] / batch)
    n, d, nnz = g["n"], g["d"], g["nnz"]
    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], None if mf else g["val"], dev)
    bt = native.Batches(n, nnz, batch, dev) if batch else None
    prev_row = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev) if delay >= 0 else None
    lv = native.Levels(bt.nb if batch else n, nnz, dev)
    ws_s = native.workspace(native.pdb_schedule_workspace_bytes(n, d, nnz), dev)
    ws_e = native.workspace(
        native.pdb_stale_workspace_bytes(nnz) if delay >= 0 else native.pdb_epoch_workspace_bytes(
            (g["n_users"] + g["n_items"]) * g["rank"] if mf else d), dev)
    if mf:
        user = torch.from_numpy(g["user"]).to(dev)
        item = torch.from_numpy(g["item"]).to(dev)
        rating = torch.from_numpy(g["rating"]).to(dev)
        U0 = torch.from_numpy(g["U0"]).to(dev)
        V0 = torch.from_numpy(g["V0"]).to(dev)
        U, V = U0.clone(), V0.clone()
    else:
        y = torch.from_numpy(g["y"]).to(dev)
        w0 = torch.zeros(d, dtype=torch.float32, device=dev)
        w = w0.clone()
    stream = torch.cuda.current_stream(dev)
    ev = []
    sched_ms = []
    info = {}

    def step(timed):
        nonlocal info
        # events on the library's stream: the schedule's pair starts once the
        # previous step's epoch has finished on the device
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record(stream)
        if batch:
            info = native.pdb_batch_schedule(csr, n, d, bt, lv, args.method, ws=ws_s)
        elif delay >= 0:
            # bounded delay needs only each entry's previous writer
            native.pdb_prev_writer(csr, n, d, prev_row, lv.prev_nz, ws=ws_s)
        else:
            info = native.pdb_schedule(csr, None, n, d, lv, args.method, ws=ws_s)
        s1.record(stream)
        sched_ms.append((s0, s1))
        if mf:
            U.copy_(U0)
            V.copy_(V0)
        else:
            w.copy_(w0)
        for _ in range(args.epochs):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            if mf:
                native.pdb_mf_epoch(user, item, rating, n, U, g["n_users"], V, g["n_items"],
                                    g["rank"], float(g["lr"]), float(g["reg"]), lv, ws=ws_e)
            elif batch:
                native.pdb_batch_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], bt, lv,
                                       ws=ws_e)
            elif delay >= 0:
                native.pdb_stale_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], delay, lv,
                                       ws=ws_e)
            else:
                native.pdb_sgd_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], lv, ws=ws_e)
            b.record(stream)
            if timed:
                ev.append((a, b))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    if native.pdb_workspace_status(ws_e) != native.PDB_OK:
        raise SystemExit("device-side failure during warmup")
    sched_ms.clear()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(True)
        print("step %d done" % k, file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if native.pdb_workspace_status(ws_e) != native.PDB_OK:
        raise SystemExit("device-side failure during the timed steps")
    elapsed = t1 - t0
    epoch_ms = [a.elapsed_time(b) for a, b in ev]
    ep = trimmed_mean(epoch_ms)
    L = lv.L_host
    units = n if mf else nnz
    value = units * args.epochs * args.steps / elapsed
    abytes = (algorithmic_bytes(g, L, U=bt.U_host, nb=bt.nb) if batch
              else algorithmic_bytes(g, L, mf))
    achieved = abytes / (ep * 1e-3) / 1e9
    workload = "c%d" % cfg_id + ("-b%d" % batch if batch else "") + \
        ("-d%d" % delay if delay >= 0 else "")
    # the epoch kernel the library runs (the rule of pdb_sgd_epoch / pdb_mf_epoch)
    mode = int(os.environ.get("PDB_EPOCH_MODE", "0"))
    syncfree = mode == 2 or (mode == 0 and L > 0 and n >= 8 * L)
    if batch:
        kernel = "k_batch_syncfree (mini-batch epoch)" if mode != 1 else \
            "k_batch_levels (mini-batch epoch)"
    elif delay >= 0:
        kernel = ("k_stale_window or k_stale_epoch (bounded-delay epoch; the library picks "
                  "per call, windowed on chain-like inputs)")
    elif syncfree:
        kernel = "k_mf_syncfree (epoch)" if mf else "k_sgd_syncfree (epoch)"
    else:
        kernel = "k_levels_apply (epoch)"
    digest = source_digest(bool(batch), delay >= 0)
    traffic = read_traffic(workload, digest)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "ratings/s" if mf else "nnz-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "epochs_per_step": args.epochs,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "%s: %s%s%s" % (workload, g["name"],
                                                ", mini-batches of %d" % batch if batch else "",
                                                ", delay %d" % delay if delay >= 0 else ""),
                   "n": n, "d": d, "nnz": nnz,
                   "seed": g["seed"], "levels": None if delay >= 0 else L,
                   "max_level_width": None if delay >= 0 else lv.max_width_host,
                   "schedule_method": info.get("method_used"),
                   "schedule_rounds": info.get("rounds")},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": kernel, "algorithmic_bytes": abytes,
                     "epoch_ms": ep, "epoch_ms_all": epoch_ms, "source_digest": digest,
                     # levels run one after another: the epoch is a dependent
                     # chain of L levels, so the time per level is the figure
                     # that bounds it when levels are narrow
                     **({"levels": L, "ns_per_level": ep * 1e6 / max(L, 1)} if delay < 0 else {})},
        "schedule_ms": trimmed_mean([a.elapsed_time(b) for a, b in sched_ms]),
        "epoch_ms": ep,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(g, cfg_id, args.cpu_budget,
                                           None if delay >= 0 else lv.level.cpu().numpy(),
                                           batch, delay)
    print(json.dumps(out))


if __name__ == "__main__":
    main()

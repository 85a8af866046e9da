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

Prints one JSON line.  `parity` compares the last step's result with the CPU
oracle on the whole workload (levels bit-exact, weights within 1e-5 of the
natural summation order and bitwise equal to the matched one); `value` is
0 and `invalid` says why when any of them fails.  `roofline` prices the
dominant kernel (the epoch) against HBM bandwidth with its algorithmic
bytes, next to the copy rate the library's stream kernel reaches on the same
GPU; `cpu_baseline` times the CPU oracle on a bounded prefix of the same
workload.  --microbench prints the copy, hand-over and barrier figures alone.
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
NATURAL_TOL = 1e-5


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
    """Digest of the sources of the priced epoch kernel: a counter record
    taken on other sources is not reported."""
    h = hashlib.sha256()
    main = "dense.hip" if dense else ("stale.hip" if stale else ("batch.hip" if batch else "apply.hip"))
    for f in (main, "pdb_math.h", "pdb_words.h", "pdb_internal.h"):
        with open(os.path.join(_ROOT, "paper_1508_00703_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_profile(kind, workload, digest):
    """The JSON record of profiles/<kind>_<workload>.md (a line starting with
    '<kind>_json:'), if it was taken on the current kernel source; else None."""
    path = os.path.join(_ROOT, "profiles", "%s_%s.md" % (kind, workload))
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if line.startswith("%s_json:" % kind):
            vals = json.loads(line.split(":", 1)[1])
    if vals.get("source_digest") != digest:
        return None
    return vals


def read_traffic(workload, digest):
    """HBM bytes per epoch launch from the committed counter summary."""
    rec = read_profile("traffic", workload, digest)
    return None if rec is None else rec.get("hbm_bytes_per_launch")


def read_l2(workload, digest):
    """L2 hits, misses and hit rate of the epoch kernel per launch."""
    rec = read_profile("l2", workload, digest)
    if rec is None:
        return None
    return {k: rec[k] for k in ("hit_rate", "hits_per_launch", "misses_per_launch", "kernel")
            if k in rec}


def trimmed_mean(xs):
    xs = sorted(xs)
    if len(xs) >= 10:
        xs = xs[2:-2]
    return sum(xs) / len(xs)


def host_cpu():
    """lscpu's model name and the host threads this process may use."""
    model = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count()
    return {"model": model, "nproc": nproc, "threads_in_host": os.cpu_count()}


def copy_peak(dev, nbytes=1 << 30, reps=10):
    """The library's streaming copy of nbytes, timed with events: read plus
    written bytes per second (GB/s), trimmed mean of reps runs."""
    import torch

    from paper_1508_00703_amd import native

    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream(dev)
    for _ in range(2):
        native.pdb_mb_copy(src, dst)
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        native.pdb_mb_copy(src, dst)
        b.record(stream)
        times.append((a, b))
    torch.cuda.synchronize()
    ms = trimmed_mean([a.elapsed_time(b) for a, b in times])
    del src, dst
    return 2.0 * nbytes / (ms * 1e-3) / 1e9


def microbench(args):
    """Copy rate, device-scope hand-over latency and grid-barrier cost."""
    import torch

    from paper_1508_00703_amd import native

    native.load()
    dev = torch.device("cuda:0")
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    out = {"microbench": True, "device": torch.cuda.get_device_name(dev), "compute_units": cus,
           "copy_gbs": {}, "hop_ns": {}, "barrier_ns": {}}
    for gib in (1, 4):
        out["copy_gbs"]["%d GiB" % gib] = copy_peak(dev, gib << 30)
        print("copy %d GiB done" % gib, file=sys.stderr, flush=True)
    for partner in (1, 8, 9, 255):
        ns, xa, xb = native.pdb_mb_hop(20000, partner, dev)
        out["hop_ns"]["block 0 (XCD %d) <-> block %d (XCD %d)" % (xa, partner, xb)] = ns
        print("hop %d done" % partner, file=sys.stderr, flush=True)
    for blocks in (8, 64, cus):
        out["barrier_ns"]["%d blocks" % blocks] = native.pdb_mb_barrier(5000, blocks, dev)
        print("barrier %d done" % blocks, file=sys.stderr, flush=True)
    print(json.dumps(out))


def cpu_baseline(g, cfg_id, budget_s, batch=0, delay=-1, epochs=1):
    """The oracle (one-pass levels + grouping + natural-order epoch), single
    thread, on the first rows of the same workload (with batch > 0: batch
    levels + grouping + the mini-batch epoch; with delay >= 0: previous
    writers + the bounded-delay epoch).  Returns the record and, when the
    prefix is the whole workload, the oracle's schedule and natural result
    (reused by the parity check)."""
    import numpy as np

    import oracle

    mf = cfg_id == 5

    def run(rows):
        rp = g["row_ptr"][:rows + 1]
        col = g["col"][:rp[-1]]
        val = None if mf or g["val"] is None else g["val"][:rp[-1]]
        t0 = time.perf_counter()
        if delay >= 0:
            oracle.prev_writer(rp, col, g["d"])
            res = oracle.stale_epoch(rp, col, val, g["y"][:rows], np.zeros(g["d"], np.float32),
                                     g["lr"], g["loss"], oracle.NATURAL, delay)
            return time.perf_counter() - t0, int(rp[-1]), None, res
        if batch:
            sched = oracle.batch_schedule(rp, col, g["d"], batch)
            res = oracle.batch_epoch(rp, col, val, g["y"][:rows], np.zeros(g["d"], np.float32),
                                     g["lr"], g["loss"], oracle.NATURAL, batch)
            return time.perf_counter() - t0, int(rp[-1]), sched, res
        sched = oracle.schedule(rp, col, g["d"])
        if mf:
            res = oracle.mf_epoch(g["user"][:rows], g["item"][:rows], g["rating"][:rows], g["U0"],
                                  g["V0"], g["lr"], g["reg"], oracle.NATURAL)
        else:
            res = oracle.sgd_epoch(rp, col, val, g["y"][:rows], np.zeros(g["d"], np.float32),
                                   g["lr"], g["loss"], oracle.NATURAL)
        return time.perf_counter() - t0, int(rp[-1]), sched, res

    n = g["n"]
    probe = min(n, 20000)
    t, _, _, _ = run(probe)
    rows = int(min(n, max(probe, probe * budget_s / max(t, 1e-6))))
    if batch:
        rows = min(n, max(batch, rows // batch * batch))  # whole batches
    t, nnz_s, sched, res = run(rows)
    units = rows if mf else nnz_s
    cpu = host_cpu()
    rec = {"value": units / t, "unit": "ratings/s" if mf else "nnz-updates/s", "cores": 1,
           "kind": "oracle",
           "sample": "first %d of %d %s (%d stored entries), %s + natural-order %sepoch, "
                     "%.1f s, one thread" % (
                         rows, n, "ratings" if mf else "examples", nnz_s,
                         "previous writers" if delay >= 0 else
                         "one-pass %slevels + grouping" % ("batch " if batch else ""),
                         "mini-batch (B=%d) " % batch if batch else
                         ("delay-%d " % delay if delay >= 0 else ""), t),
           "host_cpu": cpu["model"], "host_nproc": cpu["nproc"],
           "host_threads": cpu["threads_in_host"]}
    whole = rows == n and epochs == 1
    return rec, (sched if whole else None), (res if whole else None)


def parity_check(g, cfg_id, gpu_levels, gpu_result, sched=None, natural=None, batch=0, delay=-1,
                 epochs=1):
    """The last step's result against the oracle on the whole workload:
    levels (and grouping) bit-exact, weights within NATURAL_TOL of the natural
    summation order and bitwise equal to the matched one (the summation order
    the kernels use).  sched / natural: the oracle's schedule and natural
    result when already computed on the whole workload."""
    import numpy as np

    import oracle

    t0 = time.perf_counter()
    mf = cfg_id == 5
    out = {"scope": "whole workload", "tol_natural": NATURAL_TOL}
    if delay < 0 and gpu_levels is not None:
        if sched is None:
            sched = (oracle.batch_schedule(g["row_ptr"], g["col"], g["d"], batch) if batch
                     else oracle.schedule(g["row_ptr"], g["col"], g["d"]))
        level, perm, level_ptr, L = sched
        lv_level, lv_perm, lv_ptr, lv_L = gpu_levels
        out["levels_equal"] = bool(lv_L == L and np.array_equal(lv_level, level) and
                                   np.array_equal(lv_perm, perm) and
                                   np.array_equal(lv_ptr[:L + 1], level_ptr))
    else:
        out["levels_equal"] = None  # bounded delay runs on previous writers, not levels

    def epochs_of(mode):
        if mf:
            U, V = g["U0"], g["V0"]
            for _ in range(epochs):
                U, V = oracle.mf_epoch(g["user"], g["item"], g["rating"], U, V, g["lr"], g["reg"],
                                       mode)
            return [U, V]
        w = np.zeros(g["d"], np.float32)
        args = (g["row_ptr"], g["col"], g["val"], g["y"])
        for _ in range(epochs):
            if batch:
                w = oracle.batch_epoch(*args, w, g["lr"], g["loss"], mode, batch)
            elif delay >= 0:
                w = oracle.stale_epoch(*args, w, g["lr"], g["loss"], mode, delay)
            else:
                w = oracle.sgd_epoch(*args, w, g["lr"], g["loss"], mode)
        return [w]

    nat = ([natural] if not mf else list(natural)) if natural is not None else epochs_of(
        oracle.NATURAL)
    mat = epochs_of(oracle.MATCHED)
    out["max_abs_dw_natural"] = float(max(np.max(np.abs(a - b), initial=0.0)
                                          for a, b in zip(gpu_result, nat)))
    out["bitwise_matched"] = bool(all(np.array_equal(a.view(np.int32), b.view(np.int32))
                                      for a, b in zip(gpu_result, mat)))
    out["ok"] = bool(out["levels_equal"] is not False and out["bitwise_matched"] and
                     out["max_abs_dw_natural"] <= NATURAL_TOL)
    out["oracle_s"] = time.perf_counter() - t0
    return out


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
    cpu = host_cpu()
    return {"value": g["n"] * g["d"] * iters / t, "unit": "nnz-updates/s", "cores": 1,
            "kind": "oracle",
            "sample": "all %d x %d entries, %d of %d iterations, natural order, %.1f s, "
                      "one thread" % (g["n"], g["d"], iters, g["iters"], t),
            "host_cpu": cpu["model"], "host_nproc": cpu["nproc"],
            "host_threads": cpu["threads_in_host"]}


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
    got = w.cpu().numpy()
    if args.no_parity:
        parity = None
    else:
        import oracle

        t0 = time.perf_counter()
        w0 = np.zeros(d, np.float32)
        nat = oracle.dense_gd(g["X"], g["y"], w0, g["lr"], g["loss"], oracle.NATURAL, iters)
        mat = oracle.dense_gd(g["X"], g["y"], w0, g["lr"], g["loss"], oracle.MATCHED, iters, rb,
                              cb, 32)
        tol = 1e-4 * float(np.abs(nat).max(initial=0.0)) + 1e-6
        parity = {"scope": "whole workload", "levels_equal": None,
                  "max_abs_dw_natural": float(np.max(np.abs(got - nat), initial=0.0)),
                  "tol_natural": tol,
                  "bitwise_matched": bool(np.array_equal(got.view(np.int32), mat.view(np.int32))),
                  "oracle_s": time.perf_counter() - t0}
        parity["ok"] = parity["bitwise_matched"] and parity["max_abs_dw_natural"] <= tol
    ok = parity is not None and parity["ok"]
    peak = copy_peak(dev)
    out = {
        "metric": METRIC,
        "value": n * d * iters * args.steps / elapsed if ok else 0.0,
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
        "parity": parity,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": read_traffic(workload, digest),
                     "l2": read_l2(workload, digest),
                     "peak_measured": peak, "frac_of_measured": achieved / peak,
                     "kernel": "k_dense_gd (all iterations)", "algorithmic_bytes": abytes,
                     "call_ms": ms, "call_ms_all": call_ms, "source_digest": digest,
                     "us_per_iteration": ms * 1e3 / max(iters, 1)},
        "epoch_ms": ms,
    }
    if parity is None:
        out["invalid"] = "parity not checked (--no-parity): the value is not counted"
    elif not parity["ok"]:
        out["invalid"] = "parity with the oracle failed: the value is not counted"
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = dense_cpu_baseline(g, args.cpu_budget)
    print(json.dumps(out))


def widest_level(native, g, lv, lp, L, mf, dev, stream, run_one, reps=20):
    """The epoch kernel on the widest level alone: a one-level schedule over
    that level's examples, run level by level (they share no feature), timed
    with events on the library's stream.  The whole epoch is bounded by its
    chain of levels; this is the bandwidth the apply reaches where a level is
    wide.  Bytes as algorithmic_bytes, for the level's examples only."""
    import numpy as np
    import torch

    widths = np.diff(lp[:L + 1])
    lvl = int(np.argmax(widths))
    width = int(widths[lvl])
    rec = {"level": lvl + 1, "width": width}
    if width < 64:
        rec["skipped"] = "narrow (fewer than 64 examples)"
        return rec
    b0, b1 = int(lp[lvl]), int(lp[lvl + 1])
    sub = native.Levels(0, 0, dev, with_prev_nz=False)
    sub.perm = lv.perm[b0:b1]
    sub.level = lv.level
    sub.level_ptr = torch.tensor([0, width], dtype=torch.int64, device=dev)
    sub.n_levels.fill_(1)
    sub.prev_nz = lv.prev_nz
    sub.L_host = 1
    sub.max_width_host = width
    if mf:
        nbytes = width * (16 + 512) + 8
    else:
        rows = lv.perm[b0:b1].cpu().numpy().astype(np.int64)
        m = g["row_ptr"][rows + 1] - g["row_ptr"][rows]
        per_nz = 4 + 8 + (4 if g["val"] is not None else 0)
        nbytes = int(m.sum()) * per_nz + width * (8 + 4 + 4) + 8
        rec["entries"] = int(m.sum())
    opt1 = native.options(epoch_mode=1)
    run_one(sub, opt1)  # warm-up
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        run_one(sub, opt1)
        b.record(stream)
        times.append((a, b))
    torch.cuda.synchronize()
    us = trimmed_mean([a.elapsed_time(b) for a, b in times]) * 1e3
    gbs = nbytes / (us * 1e-6) / 1e9
    rec.update({"algorithmic_bytes": nbytes, "us_per_call": us, "achieved_gbs": gbs,
                "frac": gbs / HBM_PEAK_GBS, "kernel": "k_levels_apply (one level)"})
    return rec


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
                    help="schedule method: 0 auto, 1 chain-scan, 2 dataflow, 3 spine, 4 chain, "
                         "5 walk, 6 short-row walk")
    ap.add_argument("--epoch-mode", type=int, default=0, choices=[0, 1, 2],
                    help="epoch execution: 0 auto, 1 level by level, 2 sync-free")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true",
                    help="skip the oracle comparison (the value is then reported as unchecked)")
    ap.add_argument("--microbench", action="store_true",
                    help="only the copy rate, device-scope hand-over and grid-barrier figures")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES of device memory once with the library's copy kernel "
                         "(a plain copy of known size, for scaling HBM traffic counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the path does not shard across GPUs; "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.calibrate_copy:
        from paper_1508_00703_amd import native

        native.load()
        nbytes = args.calibrate_copy // 16 * 16
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        native.pdb_mb_copy(src, dst)
        torch.cuda.synchronize()
        print(json.dumps({"copied_bytes": nbytes, "kernel": "k_mb_copy"}))
        return

    if args.microbench:
        microbench(args)
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
    opt = native.options(epoch_mode=args.epoch_mode)
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
            info = native.pdb_batch_schedule(csr, n, d, bt, lv, args.method, ws=ws_s, opt=opt)
        elif delay >= 0:
            # bounded delay needs only each entry's previous writer
            native.pdb_prev_writer(csr, n, d, prev_row, lv.prev_nz, ws=ws_s)
        else:
            info = native.pdb_schedule(csr, None, n, d, lv, args.method, ws=ws_s, opt=opt)
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
                                    g["rank"], float(g["lr"]), float(g["reg"]), lv, ws=ws_e,
                                    opt=opt)
            elif batch:
                native.pdb_batch_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], bt, lv,
                                       ws=ws_e, opt=opt)
            elif delay >= 0:
                native.pdb_stale_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], delay, lv,
                                       ws=ws_e, opt=opt)
            else:
                native.pdb_sgd_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], lv, ws=ws_e,
                                     opt=opt)
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
    mode = args.epoch_mode
    one_cu = mf and L > 0 and n < 16 * L and (g["n_users"] + g["n_items"]) * 256 <= 2 ** 32
    syncfree = mode == 2 or (mode == 0 and L > 0 and (n >= 8 * L or one_cu))
    if batch:
        kernel = "k_batch_syncfree (mini-batch epoch)" if mode != 1 else \
            "k_batch_levels (mini-batch epoch)"
    elif delay >= 0:
        kernel = ("k_stale_window or k_stale_epoch (bounded-delay epoch; the library picks "
                  "per call, windowed on chain-like inputs)")
    elif syncfree:
        kernel = ("k_mf_onecu (epoch)" if one_cu else "k_mf_syncfree (epoch)") if mf \
            else "k_sgd_syncfree (epoch)"
    else:
        kernel = "k_levels_apply (epoch)"
    digest = source_digest(bool(batch), delay >= 0)

    # the last step's result and levels, copied out after the timed region
    gpu_result = [U.cpu().numpy(), V.cpu().numpy()] if mf else [w.cpu().numpy()]
    gpu_levels = None
    if delay < 0:
        gpu_levels = (lv.level.cpu().numpy(), lv.perm.cpu().numpy(), lv.level_ptr.cpu().numpy(),
                      L)
    # the apply on the widest level alone (outside the timed steps and after
    # the result was copied out; it changes the weights, which are not used
    # again)
    widest = None
    width_stats = {}
    if delay < 0 and not batch and L > 0:
        widths = np.diff(gpu_levels[2][:L + 1])
        width_stats = {"mean_level_width": float(widths.mean()),
                       "median_level_width": float(np.median(widths))}
        if mf:
            def run_one(sub, o):
                native.pdb_mf_epoch(user, item, rating, n, U, g["n_users"], V, g["n_items"],
                                    g["rank"], float(g["lr"]), float(g["reg"]), sub, ws=ws_e,
                                    opt=o)
        else:
            def run_one(sub, o):
                native.pdb_sgd_epoch(csr, y, n, d, w, float(g["lr"]), g["loss"], sub, ws=ws_e,
                                     opt=o)
        widest = widest_level(native, g, lv, gpu_levels[2], L, mf, dev, stream, run_one)
        if native.pdb_workspace_status(ws_e) != native.PDB_OK:
            raise SystemExit("device-side failure on the widest level")
    peak = copy_peak(dev)
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
                   **width_stats,
                   "schedule_method": info.get("method_used"),
                   "schedule_rounds": info.get("rounds"), "epoch_mode": args.epoch_mode},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": read_traffic(workload, digest),
                     "l2": read_l2(workload, digest),
                     "peak_measured": peak, "frac_of_measured": achieved / peak,
                     "kernel": kernel, "algorithmic_bytes": abytes,
                     "epoch_ms": ep, "epoch_ms_all": epoch_ms, "source_digest": digest,
                     # levels run one after another: the epoch is a dependent
                     # chain of L levels, so the time per level is the figure
                     # that bounds it when levels are narrow
                     **({"levels": L, "ns_per_level": ep * 1e6 / max(L, 1)} if delay < 0 else {})},
        "schedule_ms": trimmed_mean([a.elapsed_time(b) for a, b in sched_ms]),
        "epoch_ms": ep,
    }
    if widest is not None:
        out["roofline"]["widest_level"] = widest

    sched = natural = None
    if not args.no_cpu_baseline:
        out["cpu_baseline"], sched, natural = cpu_baseline(g, cfg_id, args.cpu_budget, batch,
                                                           delay, args.epochs)
        print("cpu baseline done", file=sys.stderr, flush=True)
    if args.no_parity:
        out["parity"] = None
        out["invalid"] = "parity not checked (--no-parity): the value is not counted"
        out["value"] = 0.0
    else:
        out["parity"] = parity_check(g, cfg_id, gpu_levels, gpu_result, sched, natural, batch,
                                     delay, args.epochs)
        print("parity check done", file=sys.stderr, flush=True)
        if not out["parity"]["ok"]:
            out["invalid"] = "parity with the oracle failed: the value is not counted"
            out["value"] = 0.0
    if mf:
        # each rating updates a 32-component user row and item row
        out["param_updates_per_s"] = out["value"] * 2 * g["rank"]
    print(json.dumps(out))


if __name__ == "__main__":
    main()

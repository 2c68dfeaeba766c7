#!/usr/bin/env python3
"""Benchmark of the LRAM lookup hot path on one MI355X.

One step = the whole path on one batch: lram_forward (wrap, closest point,
reduction to F, candidate scan, top-32, locations, weights, gather-reduce) then
lram_backward (the same search, value-gradient scatter into an fp32 gradient
table, query gradient).  Inputs are resident in HBM before timing starts; the
gradient table accumulates across steps (it is zeroed once, outside timing).

Prints one JSON line (rank 0, N = 1).  ``value`` is fwd+bwd lookups per second;
``roofline`` covers the kernel that takes longest per step, priced with
compulsory HBM bytes (each distinct table row counted once per launch) over its
average launch time measured with HIP events on its own stream;
``cpu_baseline`` times the CPU oracle on a bounded sample of the same lookups.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def pick_workload(W, name, torch):
    w = W.WORKLOADS[name]
    free, total = torch.cuda.mem_get_info()
    st = 4 if w.dtype == "f32" else 2
    need = w.table_bytes + (w.N * w.m * 4 if w.backward else 0) + w.L * (32 + w.m * 4 + w.m * st + 32) + (3 << 30)
    log("device memory: free %.1f GB of %.1f GB; %s needs %.1f GB" % (free / 1e9, total / 1e9, name, need / 1e9))
    return w, need <= free


def unique_rows(lram, q, K, torch):
    """Number of distinct table rows the batch touches (for compulsory bytes)."""
    L = q.shape[0] * q.shape[1]
    seen = None
    chunk = 1 << 20
    qf = q.reshape(-1, 8)
    for s in range(0, L, chunk):
        slot, _, _ = lram.neighbors(qf[s:s + chunk], K, want_d2=False)
        u = torch.unique(slot[slot >= 0])
        seen = u if seen is None else torch.unique(torch.cat([seen, u]))
        del slot
    return int(seen.numel())


def cpu_info() -> dict:
    """The host CPU as lscpu reports it (model, sockets, cores, threads)."""
    info = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=30).stdout
        for line in out.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in ("Model name", "Socket(s)", "Core(s) per socket", "Thread(s) per core", "CPU(s)",
                             "CPU max MHz", "L3"):
                info[k.strip()] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return info


def _omp_threads(n):
    """Thread count of the oracle's OpenMP enumeration for the calling thread."""
    try:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))
    except OSError:
        pass


def _oracle_pass(oracle, qs, rows, g, K, threads):
    """The oracle's fwd+bwd on a sample, data-parallel over `threads` threads:
    the neighbour enumeration (C, OpenMP), then forward, dq and the value
    gradient of lookup chunks (numpy, which releases the interpreter lock),
    then the chunks' gradient rows merged per row partition.  Returns seconds."""
    from concurrent.futures import ThreadPoolExecutor

    n = qs.shape[0]
    _omp_threads(threads)
    t0 = time.perf_counter()
    nb = oracle.neighbors(qs, K)
    bounds = [(i * n // threads, (i + 1) * n // threads) for i in range(threads)]

    def algebra(b):
        sl = slice(*b)
        nbs = {k: v[sl] for k, v in nb.items()}
        oracle.forward(nbs, rows[sl])
        oracle.grad_query(nbs, rows[sl], g[sl])
        return oracle.grad_table_rows(nbs, g[sl])

    def merge(p):
        us, accs = [], []
        for u, a in parts:
            k = (u % threads) == p
            us.append(u[k])
            accs.append(a[k])
        u = np.concatenate(us)
        uniq, inv = np.unique(u, return_inverse=True)
        acc = np.zeros((uniq.size, g.shape[1]), np.float64)
        np.add.at(acc, inv, np.concatenate(accs))
        return uniq.size

    with ThreadPoolExecutor(threads) as ex:
        parts = list(ex.map(algebra, bounds))
        rows_out = sum(ex.map(merge, range(threads)))
    assert rows_out > 0
    return time.perf_counter() - t0


def cpu_baseline(oracle, W, w, q_np, table, G, target_s, torch):
    """The oracle timed on the host cores: median of 3 passes over a random
    sample of the workload's lookups on every core of the GPU's share (at most
    16), and median of 3 on one core.  Value rows are copied from the GPU
    table beforehand (untimed)."""
    qf = q_np.reshape(-1, 8)
    Gf = G.reshape(-1, w.m)
    rng = np.random.default_rng(123)
    threads = max(1, min(16, len(os.sched_getaffinity(0))))

    def sample(n):
        idx = np.sort(rng.choice(qf.shape[0], n, replace=False))
        qs = qf[idx]
        _omp_threads(threads)
        sl = torch.from_numpy(oracle.neighbors(qs, w.K)["slot"]).to(table.device).long()
        rows = table[sl.clamp(min=0)].float()
        rows[sl < 0] = 0
        g = Gf[torch.from_numpy(idx).to(table.device)].cpu().numpy().astype(np.float64)
        return qs, rows.cpu().numpy(), g

    def timed(n, nthreads, budget):
        """Median of 3 passes; the sample grows until one pass takes ~budget s."""
        while True:
            qs, rows, g = sample(n)
            t = _oracle_pass(oracle, qs, rows, g, w.K, nthreads)
            if t >= 0.5 * budget or n >= qf.shape[0]:
                break
            n = int(min(qf.shape[0], max(2 * n, n * budget / max(t, 1e-3))))
        ts = sorted([t] + [_oracle_pass(oracle, qs, rows, g, w.K, nthreads) for _ in range(2)])
        return n, ts

    n_all, t_all = timed(4096, threads, target_s / 5)
    n_one, t_one = timed(1024, 1, target_s / 10)
    _omp_threads(threads)
    return {"value": n_all / t_all[1], "unit": "lookups/s (fwd+bwd)", "cores": threads, "kind": "oracle",
            "cpu": cpu_info(), "one_core": {"value": n_one / t_one[1], "lookups": n_one, "seconds": t_one},
            "seconds": t_all,
            "sample": "%d random lookups of the %s batch, median of 3 passes (%.2f / %.2f / %.2f s) on %d threads: "
                      "neighbour enumeration in C (OpenMP), forward, dq and value gradient in numpy over lookup "
                      "chunks, gradient rows merged per row partition; one core: %d lookups, median %.2f s; value "
                      "rows copied from the GPU table untimed" % (
                          n_all, w.name, t_all[0], t_all[1], t_all[2], threads, n_one, t_one[1])}


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary
    (FETCH_SIZE and WRITE_SIZE, copy-calibrated), or None if there is none or the
    kernel sources changed since the counters were taken."""
    from paper_2107_03474_amd.build import source_digest

    path = os.path.join(ROOT, "profiles", "counters_%s.json" % workload)
    try:
        prof = json.load(open(path))
        if prof.get("source_sha256") != source_digest():
            return None
        return prof["kernels"][kernel]["traffic_bytes"]
    except (OSError, KeyError, ValueError):
        return None


def copy_rate(torch, dev, nbytes=1 << 30, reps=10):
    """Attainable HBM rate: read + write bytes of a plain device-to-device copy per second."""
    a = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    rate = 2 * nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    return rate


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=15)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="k14-m32-bf16-zipf")
    ap.add_argument("--mode", default="auto", choices=["auto", "atomic", "sorted", "merged"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-compare", action="store_true",
                    help="skip timing the other scatter modes and the step variants (no shared order, saved lists)")
    ap.add_argument("--no-order", action="store_true",
                    help="no shared lookup order in the timed step (the backward sorts on its own)")
    ap.add_argument("--no-theta", action="store_true", help="skip timing the activation layer path")
    ap.add_argument("--no-k", action="store_true", help="skip timing the variable-k lookups")
    ap.add_argument("--no-subnetwork", action="store_true", help="skip timing the memory subnetwork slice")
    ap.add_argument("--no-training", action="store_true", help="skip the access statistics and the Adam step")
    ap.add_argument("--no-graph", action="store_true", help="skip the small-batch eager vs graph-replay timing")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip timing the other full-size workloads (K = 8 fp32 m = 64, K = 12 bf16 m = 64)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: there is no multi-GPU path (each GPU would run the same "
              "kernels on its own shard of the table). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2107_03474_amd as lram
    import workloads as W

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    if args.calibrate_copy:
        a = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read_per_launch": a.numel() * 4,
                          "bytes_written_per_launch": a.numel() * 4, "launches": 5}), flush=True)
        return
    lram.load()
    w, fits = pick_workload(W, args.workload, torch)
    if not fits:
        log("%s does not fit in device memory; falling back to k12-m64-bf16-proj" % w.name)
        w, fits = pick_workload(W, "k12-m64-bf16-proj", torch)
        if not fits:
            raise SystemExit("no workload fits")
    log("workload %s: %s" % (w.name, w.desc))
    t0 = time.time()
    q_np = W.queries(w)
    q = torch.from_numpy(q_np).to(dev)
    table = W.make_table(w, dev)
    G = W.grad_out(w, dev)
    gtab = torch.zeros((w.N, w.m), dtype=torch.float32, device=dev)
    out = torch.empty((w.B, w.H, w.m), dtype=table.dtype, device=dev)
    gq = torch.empty((w.B, w.H, 8), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    log("inputs ready in %.1f s" % (time.time() - t0))
    U = unique_rows(lram, q, w.K, torch)
    log("distinct rows touched: %d of %d slots (%.1f%%)" % (U, w.L * 32, 100.0 * U / (w.L * 32)))

    stream = torch.cuda.current_stream()
    mode = lram.resolved_mode(w.B, w.H, args.mode)
    # the merged scatter sorts the lookups by closest lattice point anyway: the
    # step does it once, first, and the forward and the backward both use it
    ordered = mode == "merged" and not args.no_order
    log("value-gradient scatter: %s%s" % (mode, ", lookups ordered once per step" if ordered else ""))
    nbytes = lram.backward_workspace_bytes(w.B, w.H, w.m, mode)
    wsp = torch.empty(nbytes, dtype=torch.uint8, device=dev) if nbytes and not ordered else None
    obuf = torch.empty(lram.order_layout(w.B, w.H)[0], dtype=torch.uint8, device=dev) if ordered else None

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        if ordered:
            lram.order(q, w.K, obuf)
        if ev:
            ev[1].record(stream)
        lram.forward(q, table, w.K, out=out, order=obuf)
        if ev:
            ev[2].record(stream)
        lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=mode, workspace=wsp, order=obuf)
        if ev:
            ev[3].record(stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log("warmup %d done" % i)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(ev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    order_t = [ev[k][0].elapsed_time(ev[k][1]) for k in range(args.steps)]
    fwd_t = [ev[k][1].elapsed_time(ev[k][2]) for k in range(args.steps)]
    bwd_t = [ev[k][2].elapsed_time(ev[k][3]) for k in range(args.steps)]
    step_t = [ev[k][0].elapsed_time(ev[k][3]) for k in range(args.steps)]
    order_ms, fwd_ms, bwd_ms = float(np.mean(order_t)), float(np.mean(fwd_t)), float(np.mean(bwd_t))
    ms_step = wall * 1e3 / args.steps
    log("timed %d steps: %.3f ms/step (order %.3f ms, forward %.3f ms, backward %.3f ms; median step %.3f ms)" % (
        args.steps, ms_step, order_ms, fwd_ms, bwd_ms, float(np.median(step_t))))
    timing = {"events_ms": {"order": {"mean": order_ms, "median": float(np.median(order_t))},
                            "forward": {"mean": fwd_ms, "median": float(np.median(fwd_t))},
                            "backward": {"mean": bwd_ms, "median": float(np.median(bwd_t))},
                            "step": {"mean": float(np.mean(step_t)), "median": float(np.median(step_t)),
                                     "min": float(np.min(step_t)), "max": float(np.max(step_t))}},
              "protocol": "%d warm-up steps, then %d timed steps back to back; HIP events on the launch stream "
                          "around each call; value and ms_per_step from the host clock around all %d" % (
                              args.warmup, args.steps, args.steps)}

    # the same step without the shared order (the backward sorts on its own),
    # and with the saved neighbour lists (the backward skips its search): not
    # part of `value`
    variants = {}
    if not args.no_compare:
        def timed_pair(f_fwd, f_bwd, reps=5):
            f_fwd()
            f_bwd()
            torch.cuda.synchronize()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            tf = tb = 0.0
            for _ in range(reps):
                e[0].record(stream)
                f_fwd()
                e[1].record(stream)
                f_bwd()
                e[2].record(stream)
                torch.cuda.synchronize()
                tf += e[0].elapsed_time(e[1]) / reps
                tb += e[1].elapsed_time(e[2]) / reps
            return tf, tb

        if ordered:
            nws = lram.backward_workspace_bytes(w.B, w.H, w.m, mode)
            wsu = torch.empty(nws, dtype=torch.uint8, device=dev)
            tf, tb = timed_pair(lambda: lram.forward(q, table, w.K, out=out),
                                lambda: lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=mode,
                                                      workspace=wsu))
            variants["unordered"] = {"fwd_ms": tf, "bwd_ms": tb, "step_ms": tf + tb,
                                     "what": "forward in lookup order; the backward sorts by closest point itself"}
            log("without the shared order: forward %.3f ms, backward %.3f ms" % (tf, tb))
            del wsu
        nl = lram.new_lists(q)
        tf, tb = timed_pair(lambda: lram.forward(q, table, w.K, out=out, order=obuf, lists=nl),
                            lambda: lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=mode,
                                                  workspace=wsp, order=obuf, lists=nl))
        variants["saved_lists"] = {"fwd_ms": tf, "bwd_ms": tb, "step_ms": tf + tb + order_ms,
                                   "what": "the forward also writes the 32 (location, weight, code) entries of "
                                           "every lookup (384 B); the backward reads them instead of searching"}
        log("with saved neighbour lists: forward %.3f ms, backward %.3f ms" % (tf, tb))
        del nl
    # what the accumulate-into contract spares every step: clearing the whole
    # gradient table (outside the timed steps, not part of `value`)
    ez = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ez[0].record()
    gtab.zero_()
    ez[1].record()
    torch.cuda.synchronize()
    zero_ms = ez[0].elapsed_time(ez[1])
    log("clearing the %.1f GB gradient table: %.2f ms" % (gtab.numel() * 4 / 1e9, zero_ms))

    # the other value-gradient scatters, timed the same way for comparison (not part of `value`)
    # backward calls as a caller without an order makes them (the merged one
    # sorting on its own); sorted is the bit-reproducible scatter
    by_scatter = {mode: variants["unordered"]["bwd_ms"] if "unordered" in variants else bwd_ms}
    del wsp
    for other in ("atomic", "sorted", "merged"):
        if other == mode or args.no_compare:
            continue
        nbytes = lram.backward_workspace_bytes(w.B, w.H, w.m, other)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=dev) if nbytes else None
        lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=other, workspace=ws)
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record(stream)
        for _ in range(5):
            lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=other, workspace=ws)
        e[1].record(stream)
        torch.cuda.synchronize()
        by_scatter[other] = e[0].elapsed_time(e[1]) / 5
        del ws
        log("backward with the %s scatter: %.3f ms" % (other, by_scatter[other]))

    # the activation layer of Sec. 2.3 in front of the same lookups (not part of `value`)
    theta = None
    if not args.no_theta:
        z = torch.from_numpy(W.theta_inputs(w)).to(dev)
        gz = torch.empty_like(z)
        nbytes = lram.backward_workspace_bytes(w.B, w.H, w.m, mode)
        wsp = torch.empty(nbytes, dtype=torch.uint8, device=dev) if nbytes else None
        lram.theta_forward(z, table, w.K, out=out)
        lram.theta_backward(z, table, w.K, G, grad_table=gtab, grad_z=gz, mode=mode, workspace=wsp)
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        tf = tb = 0.0
        for _ in range(5):
            e[0].record(stream)
            lram.theta_forward(z, table, w.K, out=out)
            e[1].record(stream)
            lram.theta_backward(z, table, w.K, G, grad_table=gtab, grad_z=gz, mode=mode, workspace=wsp)
            e[2].record(stream)
            torch.cuda.synchronize()
            tf += e[0].elapsed_time(e[1]) / 5
            tb += e[1].elapsed_time(e[2]) / 5
        theta = {"fwd_ms": tf, "bwd_ms": tb, "lookups_per_s": w.L / ((tf + tb) * 1e-3),
                 "fwd_lookups_per_s": w.L / (tf * 1e-3), "scatter": mode,
                 "input": "z [B, H, 16]: the workload's queries as arguments, Rayleigh moduli"}
        log("activation layer + lookup: forward %.3f ms, backward %.3f ms" % (tf, tb))
        del z, gz, wsp

    # coverage vs bandwidth: the same lookups truncated to k = 16, 32, 64 or
    # untruncated (not part of `value`); coverage = mean share of the kernel's
    # total weight on a 65,536-lookup sample
    by_k = None
    if not args.no_k:
        by_k = {}
        qs = q.reshape(-1, 8)[:65536]
        tot_all = lram.neighbors(qs, w.K, want_d2=False, k=lram.ALL)[1].double().sum(1)
        nws = lram.backward_workspace_bytes(w.B, w.H, w.m, "merged")
        wsm = torch.empty(nws, dtype=torch.uint8, device=dev)
        for kk in (16, 32, 64, lram.ALL):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            lram.forward(q, table, w.K, out=out, k=kk)
            lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, k=kk, mode="atomic")
            lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, k=kk, mode="merged", workspace=wsm)
            torch.cuda.synchronize()
            e[0].record(stream)
            for _ in range(3):
                lram.forward(q, table, w.K, out=out, k=kk)
            e[1].record(stream)
            for _ in range(3):
                lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, k=kk, mode="atomic")
            e[2].record(stream)
            for _ in range(3):
                lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, k=kk, mode="merged", workspace=wsm)
            e[3].record(stream)
            torch.cuda.synchronize()
            cov = (lram.neighbors(qs, w.K, want_d2=False, k=kk)[1].double().sum(1) / tot_all).mean().item()
            name = "all" if kk == lram.ALL else str(kk)
            by_k[name] = {"fwd_ms": e[0].elapsed_time(e[1]) / 3, "bwd_atomic_ms": e[1].elapsed_time(e[2]) / 3,
                          "bwd_merged_ms": e[2].elapsed_time(e[3]) / 3, "coverage": cov}
            log("k=%s: forward %.3f ms, backward %.3f ms atomic / %.3f ms merged, weight coverage %.6f" % (
                name, by_k[name]["fwd_ms"], by_k[name]["bwd_atomic_ms"], by_k[name]["bwd_merged_ms"], cov))
        del wsm

    st = 4 if w.dtype == "f32" else 2
    L = w.L
    fwd_bytes = L * (32 + w.m * st) + U * w.m * st
    bwd_bytes = L * (32 + w.m * 4 + 32) + U * (w.m * st + 2 * w.m * 4)
    fwd_req = L * (32 + w.m * st + 32 * w.m * st)
    bwd_req = L * (32 + w.m * 4 + 32 + 32 * (w.m * st + 2 * w.m * 4))
    if bwd_ms >= fwd_ms:
        # the atomic backward is one kernel; the other modes time every kernel
        # of the call between the same events (merged: the gated atomic kernel
        # and the fused kernel, plus the cell keys and the lookup sort when no
        # order is shared; sorted: the fused kernel, the pair sort and the
        # segmented reduction)
        kname = {"atomic": "k_backward_atomic", "merged": "backward_pass_merged",
                 "sorted": "backward_pass_sorted"}[mode]
        kms, kbytes, kreq = bwd_ms, bwd_bytes, bwd_req
    else:
        kname, kms, kbytes, kreq = "k_forward", fwd_ms, fwd_bytes, fwd_req
    achieved = kbytes / (kms * 1e-3) / 1e9
    traffic = measured_traffic(w.name, kname)
    fwd_traffic = measured_traffic(w.name, "k_forward")
    attainable = copy_rate(torch, dev)
    log("attainable HBM rate (1 GiB device copy): %.0f GB/s" % attainable)
    res = {
        "metric": "lookups/sec fwd and fwd+bwd; achieved HBM GB/s vs peak (1 GPU)",
        "value": L / (ms_step * 1e-3),
        "unit": "lookups/s (fwd+bwd)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",  # the path's arithmetic; the table's storage type is config.table_dtype
        "data": "synthetic (seeded; see workloads.py)",
        "config": {"workload": w.name, "K": list(w.K), "locations": w.N, "m": w.m, "table_dtype": w.dtype,
                   "batch": w.B, "heads": w.H, "lookups": L, "scatter": mode, "ordered": ordered,
                   "parallelism": "none (1 GPU)"},
        "fwd_lookups_per_s": L / (fwd_ms * 1e-3),
        "order_ms": order_ms,
        "fwd_ms": fwd_ms,
        "bwd_ms": bwd_ms,
        "timing": timing,
        "variants": variants,
        "bwd_ms_by_scatter": by_scatter,
        "distinct_rows": U,
        "grad_table_zero_ms": zero_ms,
        "theta": theta,
        "by_k": by_k,
        "roofline": {"kernel": kname, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "attainable": attainable, "frac_attainable": achieved / attainable,
                     "bytes_per_launch": kbytes, "requested_bytes_per_launch": kreq,
                     "requested_GBps": kreq / (kms * 1e-3) / 1e9},
        "fwd_hbm_GBps": fwd_bytes / (fwd_ms * 1e-3) / 1e9,
        "bwd_hbm_GBps": bwd_bytes / (bwd_ms * 1e-3) / 1e9,
        # requested bytes (every lookup reads its 32 rows) over time
        "fwd_requested_GBps": fwd_req / (fwd_ms * 1e-3) / 1e9,
        "bwd_requested_GBps": bwd_req / (bwd_ms * 1e-3) / 1e9,
        # counter-measured HBM bytes of the forward (whole 128-byte lines for
        # 64-byte rows) over its time; null while the counters are stale
        "fwd_traffic_GBps": (fwd_traffic / (fwd_ms * 1e-3) / 1e9) if fwd_traffic else None,
    }
    if not args.no_cpu_baseline:
        import oracle

        log("cpu baseline (oracle) ...")
        res["cpu_baseline"] = cpu_baseline(oracle, W, w, q_np, table, G, args.cpu_seconds, torch)
        log("cpu baseline done")
    del table, gtab, G, out, gq, q
    torch.cuda.empty_cache()
    if not args.no_workloads:
        res["workloads"] = time_workloads(torch, lram, W, log)
    if not args.no_subnetwork:
        res["memory_subnetwork"] = time_subnetwork(torch, lram, log)
    if not args.no_training:
        res["training"] = time_training(torch, lram, W, log)
    if not args.no_graph:
        res["small_batch_graph"] = time_small_graph(torch, lram, W, log)
    print(json.dumps(res), flush=True)


def time_workloads(torch, lram, W, log, reps=10):
    """The other full-size workloads, timed like the headline one (not part of
    `value`): k8-m64-f32-uniform (forward only: 256-byte fp32 rows, whole
    lines) and k12-m64-bf16-proj (forward + backward, 128-byte rows, queries
    from a dense projection), each with its requested bytes (every lookup
    reads its 32 rows) and compulsory bytes (each distinct row once) per
    second, and the requested rate as a fraction of the 8 TB/s peak."""
    dev = torch.device("cuda")
    stream = torch.cuda.current_stream()
    out = {}

    def timed(f):
        f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for name in ("k8-m64-f32-uniform", "k12-m64-bf16-proj"):
        w, fits = pick_workload(W, name, torch)
        if not fits:
            out[name] = None
            continue
        q = torch.from_numpy(W.queries(w)).to(dev)
        table = W.make_table(w, dev)
        o = torch.empty((w.B, w.H, w.m), dtype=table.dtype, device=dev)
        U = unique_rows(lram, q, w.K, torch)
        st = 4 if w.dtype == "f32" else 2
        L = w.L
        fwd_ms = timed(lambda: lram.forward(q, table, w.K, out=o))
        fwd_req = L * (32 + 32 * w.m * st + w.m * st)
        fwd_comp = L * (32 + w.m * st) + U * w.m * st
        rec = {"lookups": L, "locations": w.N, "m": w.m, "table_dtype": w.dtype, "distinct_rows": U,
               "fwd_ms": fwd_ms, "fwd_lookups_per_s": L / (fwd_ms * 1e-3),
               "fwd_requested_GBps": fwd_req / (fwd_ms * 1e-3) / 1e9,
               "fwd_requested_frac": fwd_req / (fwd_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
               "fwd_hbm_GBps": fwd_comp / (fwd_ms * 1e-3) / 1e9}
        if w.backward:
            G = W.grad_out(w, dev)
            gtab = torch.zeros((w.N, w.m), dtype=torch.float32, device=dev)
            gq = torch.empty((w.B, w.H, 8), dtype=torch.float32, device=dev)
            mode = lram.resolved_mode(w.B, w.H, "auto")
            nws = lram.backward_workspace_bytes(w.B, w.H, w.m, mode)
            ws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None
            bwd_ms = timed(lambda: lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=mode,
                                                 workspace=ws))
            bwd_req = L * (32 + w.m * 4 + 32 + 32 * (w.m * st + 2 * w.m * 4))
            bwd_comp = L * (32 + w.m * 4 + 32) + U * (w.m * st + 2 * w.m * 4)
            rec.update({"scatter": mode, "bwd_ms": bwd_ms, "lookups_per_s": L / ((fwd_ms + bwd_ms) * 1e-3),
                        "bwd_requested_GBps": bwd_req / (bwd_ms * 1e-3) / 1e9,
                        "bwd_requested_frac": bwd_req / (bwd_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                        "bwd_hbm_GBps": bwd_comp / (bwd_ms * 1e-3) / 1e9})
            del G, gtab, gq, ws
        out[name] = rec
        log("%s: forward %.3f ms (%.0f GB/s requested)%s" % (
            name, fwd_ms, rec["fwd_requested_GBps"],
            ", backward %.3f ms (%.0f GB/s requested)" % (rec["bwd_ms"], rec["bwd_requested_GBps"])
            if w.backward else ""))
        del q, table, o
        torch.cuda.empty_cache()
    return out


def time_small_graph(torch, lram, W, log, reps=200):
    """The 4,096-lookup configurations are launch-bound: one forward + backward
    step launched eagerly through the binding, and the same step captured once
    into a HIP graph and replayed (microseconds per step, `reps` steps back to
    back; the gradient table accumulates across steps)."""
    out = {}
    for name in ("k4-m32-f32-uniform", "k4-m32-f32-gmm64"):
        w = W.WORKLOADS[name]
        q = torch.from_numpy(W.queries(w)).to("cuda")
        table = W.make_table(w, torch.device("cuda"))
        G = W.grad_out(w, torch.device("cuda"))
        gtab = torch.zeros((w.N, w.m), dtype=torch.float32, device="cuda")
        o = torch.empty((w.B, w.H, w.m), dtype=table.dtype, device="cuda")
        gq = torch.empty((w.B, w.H, 8), dtype=torch.float32, device="cuda")
        mode = lram.resolved_mode(w.B, w.H, "auto")
        nws = lram.backward_workspace_bytes(w.B, w.H, w.m, mode)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None

        nl = lram.new_lists(q)

        def step():
            lram.forward(q, table, w.K, out=o)
            lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=mode, workspace=ws)

        def step_saved():
            lram.forward(q, table, w.K, out=o, lists=nl)
            lram.backward(q, table, w.K, G, grad_table=gtab, grad_q=gq, mode=mode, workspace=ws, lists=nl)

        def timed(f):
            for _ in range(10):
                f()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                f()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps * 1e3

        def captured(f):
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                f()
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                f()
            return graph

        def kernel_us(f):
            """Kernel time of one step: HIP events around each of `reps` steps
            with the host waiting in between (no launch overlap)."""
            ts = []
            for _ in range(20):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                f()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3)
            return float(np.median(ts))

        eager_us = timed(step)
        graph = captured(step)
        graph_us = timed(graph.replay)
        eager_saved_us = timed(step_saved)
        graph_s = captured(step_saved)
        graph_saved_us = timed(graph_s.replay)
        out[name] = {"lookups": w.L, "scatter": mode, "eager_us": eager_us, "graph_us": graph_us,
                     "graph_lookups_per_s": w.L / (graph_us * 1e-6),
                     "saved_lists": {"eager_us": eager_saved_us, "graph_us": graph_saved_us},
                     "isolated_step_us": {"recompute": kernel_us(step), "saved_lists": kernel_us(step_saved)}}
        log("%s: fwd+bwd step %.1f us eager, %.1f us graph replay; with saved lists %.1f / %.1f us" % (
            name, eager_us, graph_us, eager_saved_us, graph_saved_us))
        del graph, graph_s, q, table, G, gtab, o, gq, ws, nl
        torch.cuda.empty_cache()
    return out


def time_training(torch, lram, W, log, batches=16):
    """The utilisation table's analogue and the optimiser step at the paper's
    memory sizes (2^18, 2^20, 2^22 locations of m = 64 fp32) and at 2^26:
    access share and KL over `batches` synthetic batches of 8192 x 32 lookups
    (the queries of the bench workload's Zipf/uniform mix on each torus; one
    batch at 2^26), then one backward + sparse Adam step per batch, twice:
    the full-scan step, and the touched-row step (flags from mark_touched for
    the batch, then the step on the flagged rows) on a copy of the same table,
    moments and gradient.  Adam times and the full step's HBM rate (grad scan +
    the touched rows' moments, values and cleared gradient)."""
    out = {}
    for name, K, nb in (("2^18", (4, 4, 4, 4, 4, 4, 8, 8), batches), ("2^20", (4, 4, 4, 4, 8, 8, 8, 8), batches),
                        ("2^22", (4, 4, 8, 8, 8, 8, 8, 8), batches), ("2^26", (8, 8, 8, 8, 8, 8, 16, 16), 1)):
        N = int(np.prod(K))
        wl = W.Workload("stats", K, 64, "f32", 8192, 32, "zipf_mix", True, gmm_sigma=0.3, zipf_centres=4096,
                        zipf_s=1.1)
        table = torch.randn((N, 64), device="cuda") * 0.02
        table2 = table.clone()
        opt = lram.SparseAdam(table, lr=1e-3)
        opt2 = lram.SparseAdam(table2, lr=1e-3)
        gtab = torch.zeros((N, 64), dtype=torch.float32, device="cuda")
        hist = torch.zeros(N, dtype=torch.float32, device="cuda")
        flags = torch.zeros(N, dtype=torch.uint8, device="cuda")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        adam_ms = touched_ms = mark_ms = 0.0
        touched = 0
        for b in range(nb):
            q = torch.from_numpy(W.queries(wl, seed=100 + b)).to("cuda")
            lram.access_histogram(q, K, hist)
            G = torch.randn((wl.B, wl.H, 64), device="cuda")
            lram.backward(q, table, K, G, grad_table=gtab, want_grad_q=False)
            gtab2 = gtab.clone()
            if b == nb - 1:
                touched = int((gtab != 0).any(1).sum().item())
            torch.cuda.synchronize()
            ev[0].record()
            opt.step(gtab)
            ev[1].record()
            lram.mark_touched(q, K, flags)
            ev[2].record()
            opt2.step(gtab2, flags)
            ev[3].record()
            torch.cuda.synchronize()
            adam_ms += ev[0].elapsed_time(ev[1]) / nb
            mark_ms += ev[1].elapsed_time(ev[2]) / nb
            touched_ms += ev[2].elapsed_time(ev[3]) / nb
            del gtab2
        same = bool(torch.equal(table, table2))
        st = lram.access_stats(hist)
        adam_bytes = N * 64 * 4 + touched * 64 * 4 * 7
        out[name] = {"locations": N, "K": list(K), "lookups": nb * wl.L, "used": st["used"], "kl": st["kl"],
                     "adam_ms": adam_ms, "adam_touched_rows": touched,
                     "adam_GBps": adam_bytes / (adam_ms * 1e-3) / 1e9,
                     "adam_touched_step_ms": touched_ms, "mark_touched_ms": mark_ms, "touched_step_identical": same}
        log("memory %s: used %.4f, KL %.3f over %d lookups; Adam step %.3f ms full scan (%d touched rows, %.0f GB/s), "
            "%.3f ms on the flagged rows (+ %.3f ms marking them), identical %s" % (
                name, st["used"], st["kl"], nb * wl.L, adam_ms, touched, out[name]["adam_GBps"], touched_ms, mark_ms,
                same))
        del table, table2, opt, opt2, gtab, hist, flags
        torch.cuda.empty_cache()
    return out


def time_subnetwork(torch, lram, log, widths=(2048, 3072, 4096, 6144, 8192, 12288), tokens=8192, K=(10,) * 8):
    """Inference time per vector of the memory subnetwork (dense w -> w, batch
    norm, theta with h = w/16 heads of m = 64, dense 4w -> w) at the widths of
    the paper's timing table, bf16 dense layers and table, one shared table of
    prod K = 1e8 locations (12.8 GB), a batch of 8192 vectors (32 x 256 tokens)."""
    from paper_2107_03474_amd.memory_layer import MemorySubnetwork, M_VALUE

    N = int(np.prod(K))
    table = torch.empty((N, M_VALUE), dtype=torch.bfloat16, device="cuda")
    for s in range(0, N, 1 << 22):
        table[s:s + (1 << 22)] = torch.randn((min(1 << 22, N - s), M_VALUE), device="cuda") * 0.02
    out = {"tokens": tokens, "K": list(K), "dtype": "bf16 dense and table, fp32 accumulate", "us_per_vector": {}}
    for wd in widths:
        net = MemorySubnetwork(wd, K, dtype=torch.bfloat16, table=table).eval()
        x = torch.randn((tokens, wd), device="cuda", dtype=torch.bfloat16)
        with torch.no_grad():
            for _ in range(2):
                net(x)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(5):
                net(x)
            e1.record()
            torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / 5 * 1e3 / tokens
        out["us_per_vector"][str(wd)] = us
        log("memory subnetwork w=%d: %.3f us per vector (%d lookups per batch)" % (wd, us, tokens * wd // 16))
        del net, x
        torch.cuda.empty_cache()
    del table
    torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark: one step = the whole hot path on the ResNet-50-shaped workload.

Step = sparsify of the 161-tensor, 25,557,032-element gradient set (x = g + r,
exact global top-k at rho = 0.001, ascending (idx, val), residual written
back), followed by the sparse aggregate + SGD update of P = 128 workers' lists
(this GPU's own 25,558 pairs plus 127 seeded lists of 25,600 pairs) into
ResNet-50-shaped parameters with momentum 0.9, weight decay 5e-5, lr 0.1.

Inputs are synthetic and resident in HBM before timing: ten seeded gradient
steps and three replicas of (residual, parameters, momentum, gathered lists),
rotated so that consecutive steps never reuse a buffer and a step's inputs are
not left in the 256 MB last-level cache by the step before. The residual of
each replica is carried across steps.

Prints one JSON line. `value` = sparsify throughput in Gelem/s (d / mean
sparsify time); the update's rate is reported beside it.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "top-k sparsify Gelem/s at d=25.6M rho=0.001 (% of HBM peak); update GB/s"
HBM_PEAK_GBPS = 8000.0
RHO = 0.001
P_WORKERS = 128
K_LIST = 25_600
LR, MU, WD = 0.1, 0.9, 5e-5
GRAD_STEPS = 10


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--replicas", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the CPU oracle")
    ap.add_argument("--workload", default="resnet50",
                    choices=["resnet50", "c1", "transformer", "bert", "sweep"],
                    help="resnet50: the headline step (default); c1: one 1 M-element tensor, "
                         "rho 0.001, then a one-worker plain update; transformer: the 110 M "
                         "Transformer-shaped set, Laplace(0, 1e-3), rho 0.001 and 0.01, global "
                         "and per tensor; bert: one 340 M-element tie-stressed buffer, rho 0.001 "
                         "(these three print sparsify rates only, no extras); sweep: flat "
                         "N(0,1) vectors of 2^18 .. 2^27 elements, k = ceil(0.001 d)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the variant paths timed after the step (fp16 values, dense "
                         "aggregation, shard-shaped sparsify)")
    ap.add_argument("--kernel-events", type=int, default=1,
                    help="record HIP events around every kernel (1) or only per phase (0)")
    ap.add_argument("--probe-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain elementwise copy of MIB MiB five times (the "
                         "reference kernel for scaling HBM counter readings) and exit")
    ap.add_argument("--probe-add", type=int, default=0, metavar="MIB",
                    help="only run an elementwise add of two MIB MiB arrays into a third "
                         "five times (two reads, one write: the stream's pattern) and exit")
    ap.add_argument("--cpu-procs", type=int, default=0,
                    help="processes of the all-core oracle leg (default: the usable cores, "
                         "at most 16)")
    ap.add_argument("--summarize-stats", metavar="CSV",
                    help="print the tkef kernels of a rocprofv3 --stats kernel_stats.csv and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("CSV", "COUNTER"),
                    help="print per-dispatch averages of COUNTER per tkef kernel from a "
                         "rocprofv3 --pmc counter_collection.csv and exit")
    return ap.parse_args()


def probe_copy(mib: int) -> int:
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"probe_copy_bytes_read": n * 4, "probe_copy_bytes_written": n * 4,
                      "launches": 5}), flush=True)
    return 0


def probe_add(mib: int) -> int:
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, device="cuda:0")
    b = torch.ones(n, device="cuda:0")
    c = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(5):
        torch.add(a, b, out=c)
    torch.cuda.synchronize()
    print(json.dumps({"probe_add_bytes_read": 2 * n * 4, "probe_add_bytes_written": n * 4,
                      "launches": 5}), flush=True)
    return 0


def _short_kernel(name: str) -> str:
    n = name.split("(")[0]
    return n[5:] if n.startswith("void ") else n


def summarize_stats(path: str) -> int:
    """Kernel table (calls, average / min / max duration) of the tkef kernels
    in a rocprofv3 kernel_stats.csv."""
    import csv
    print(f"{'kernel':36s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} "
          f"{'pct':>6s}")
    for r in csv.DictReader(open(path)):
        n = _short_kernel(r["Name"])
        if n.startswith("tkef::"):
            print(f"{n:36s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:9.2f} "
                  f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} "
                  f"{float(r['Percentage']):6.2f}")
    return 0


def summarize_pmc(path: str, counter: str) -> int:
    """Per-dispatch average of one counter (summed over the dispatch's rows)
    for every kernel in a rocprofv3 counter_collection.csv."""
    import collections
    import csv
    per = collections.defaultdict(float)
    names = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        per[r["Dispatch_Id"]] += float(r["Counter_Value"])
        names[r["Dispatch_Id"]] = _short_kernel(r["Kernel_Name"])
    agg = collections.defaultdict(list)
    for dsp, v in per.items():
        agg[names[dsp]].append(v)
    print(f"{'kernel':40s} {'dispatches':>10s} {counter + ' per dispatch':>28s}")
    for n, vs in sorted(agg.items(), key=lambda kv: -max(kv[1])):
        print(f"{n:40s} {len(vs):10d} {sum(vs) / len(vs):28.1f}")
    return 0


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def usable_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def log(msg: str) -> None:
    sys.stderr.write(f"[bench] {msg}\n")
    sys.stderr.flush()


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2010_10458_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel: str, digest: str):
    """HBM traffic per launch measured by rocprofv3 counters, if a summary for
    this kernel exists and was taken on the current kernel sources: the
    scaled bytes, and the raw FETCH_SIZE / WRITE_SIZE readings with their
    scale factors."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_resnet50.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_digest") != digest:
        return None
    try:
        fs, ws = (float(x) for x in vals["scale (fetch, write)"].split(","))
        return {"bytes": float(vals["hbm_bytes_per_launch"]),
                "fetch_kib_raw": float(vals["FETCH_SIZE per launch (raw KiB)"]),
                "write_kib_raw": float(vals["WRITE_SIZE per launch (raw KiB)"]),
                "fetch_scale": fs, "write_scale": ws}
    except (KeyError, ValueError):
        return None


def _oracle_worker(step, barrier, out):
    """One process of the all-core leg: the oracle's sparsify of gradient
    step `step` of the same workload, timed after every process is ready."""
    import numpy as np

    import gen
    import oracle
    orc = oracle.Oracle()
    grads = gen.resnet_grads(step)
    res = [np.zeros(a.size, np.float32) for a in grads]
    barrier.wait()
    t0 = time.perf_counter()
    orc.sparsify(grads, res, rho=RHO)
    out.put((t0, time.perf_counter()))


def cpu_baseline(sizes, d, procs=0):
    """The CPU oracle on bounded samples of the same workload: one sparsify
    step (and one update) on one thread, then one sparsify step per process on
    every usable core at once (the oracle as it is, one process per core)."""
    import multiprocessing as mp

    import numpy as np

    import gen
    import oracle
    orc = oracle.Oracle()
    grads = gen.resnet_grads(0)
    res = [np.zeros(n, np.float32) for n in sizes]
    t0 = time.perf_counter()
    idx, val, _, ks = orc.sparsify(grads, res, rho=RHO)
    t_sp = time.perf_counter() - t0
    del grads, res
    lists_i, lists_v = gen.sparse_lists(d, P_WORKERS, K_LIST, step=0)
    w = gen.concat(gen.params_like(sizes, config=5))
    b = np.zeros(d, np.float32)
    t0 = time.perf_counter()
    orc.update(w, b, lists_i, lists_v, lr=LR, mu=MU, wd=WD)
    t_up = time.perf_counter() - t0
    del lists_i, lists_v, w, b
    upd_bytes = 16 * d + 8 * P_WORKERS * K_LIST
    # all cores: spawned processes (the parent holds a GPU context, so no fork)
    n = procs or min(16, usable_cores())
    ctx = mp.get_context("spawn")
    barrier, out = ctx.Barrier(n), ctx.Queue()
    ps = [ctx.Process(target=_oracle_worker, args=(s % GRAD_STEPS, barrier, out))
          for s in range(n)]
    for p in ps:
        p.start()
    spans = [out.get() for _ in range(n)]
    for p in ps:
        p.join()
    wall = max(e for _, e in spans) - min(b for b, _ in spans)
    all_rate = n * d / wall / 1e9
    return {"value": round(all_rate, 6), "unit": "Gelem/s", "cores": n, "kind": "oracle",
            "sample": f"ResNet-50-shaped sparsify steps (d={d}, k={ks[0]}, full comparison "
                      f"sort): one per process on {n} processes at once (value), and one on "
                      f"a single thread; plus one P={P_WORKERS} x {K_LIST} momentum update "
                      f"on a single thread",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "usable_cores": usable_cores(),
            "all_cores_wall_s": round(wall, 3),
            "single_thread": {"value": round(d / t_sp / 1e9, 6), "sparsify_s": round(t_sp, 3),
                              "update_s": round(t_up, 3),
                              "update_GBps": round(upd_bytes / t_up / 1e9, 3)}}


def time_calls(plan_of, call, n_calls, warmup, make_events):
    """Mean whole-call and per-kernel times (ms) of call(plan_of(i)) over
    n_calls, from events recorded by the plans' own dispatches. plan_of
    rotates over plans with separate buffers, as the step does."""
    import numpy as np
    import torch
    names = plan_of(0).launch_names()
    for i in range(warmup):
        call(plan_of(i))
    evs = [make_events(len(names) + 1) for _ in range(n_calls)]
    torch.cuda.synchronize()
    for t in range(n_calls):
        pl = plan_of(warmup + t)
        pl.set_events(evs[t])
        call(pl)
        pl.set_events(None)
    torch.cuda.synchronize()
    total = float(np.mean([e[0].elapsed_time(e[-1]) for e in evs]))
    kern = {n: round(float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) * 1e3, 2)
            for i, n in enumerate(names)}
    return total, kern


def extras(args, tk, gen, sizes, d, bank, resid, idx_all, val_all, nnz, k_total, make_events):
    """Variant paths on the same resident inputs, each timed like the step
    (rotating buffers): binary16 values out of the sparsify, the dense
    aggregation of the P = 128 lists, and the per-GPU shard of the
    hierarchical scheme (8 contiguous shards of a flat 25.6 M gradient,
    k~ = ceil(rho d / 8))."""
    import torch
    dev = bank[0][0].device
    K, W, R = args.steps, args.warmup, len(resid)
    ex = {}

    log("extras: sparsify with binary16 values")
    p16 = [[tk.SparsifyPlan(sizes, rho=RHO, val_dtype=torch.float16).bind(bank[s], resid[j])
            for j in range(R)] for s in range(len(bank))]
    i16 = torch.empty(k_total, dtype=torch.int32, device=dev)
    v16 = torch.empty(k_total, dtype=torch.float16, device=dev)
    ms, kern = time_calls(lambda i: p16[i % len(bank)][i % R], lambda pl: pl.execute(i16, v16),
                          K, W, make_events)
    ex["sparsify_fp16_us"] = round(ms * 1e3, 2)
    ex["sparsify_fp16_kernels_us"] = kern
    del p16

    log("extras: MSTopK (Alg. 1, N = 30) on the same workload")
    pms = [[tk.SparsifyPlan(sizes, mode=tk.APPROX, rho=RHO, n_search=30).bind(bank[s], resid[j])
            for j in range(R)] for s in range(len(bank))]
    ims = torch.empty(k_total, dtype=torch.int32, device=dev)
    vms = torch.empty(k_total, dtype=torch.float32, device=dev)
    ms, kern = time_calls(lambda i: pms[i % len(bank)][i % R],
                          lambda pl: pl.execute(ims, vms, window_word=0x9E3779B97F4A7C15),
                          K, W, make_events)
    # selection quality against the exact top-k of the same x (fresh residual)
    x_ref = [t.clone() for t in bank[0]]
    r0 = [torch.zeros_like(t) for t in bank[0]]
    pe = tk.SparsifyPlan(sizes, rho=RHO).bind(x_ref, r0)
    ie, _ = pe.execute()
    r1 = [torch.zeros_like(t) for t in bank[0]]
    pa = tk.SparsifyPlan(sizes, mode=tk.APPROX, rho=RHO, n_search=30).bind(x_ref, r1)
    ia, _ = pa.execute(window_word=0x9E3779B97F4A7C15)
    info = pa.approx_result()
    xf = torch.cat(x_ref).abs().double()
    overlap = torch.isin(ia.long(), ie.long()).sum().item() / k_total
    mass = (xf[ia.long()].sum() / xf[ie.long()].sum()).item()
    ex["mstopk"] = {"n_search": 30, "sparsify_us": round(ms * 1e3, 2),
                    "Gelem_per_s": round(d / (ms / 1e3) / 1e9, 2),
                    "kernels_us": kern,
                    "overlap_with_exact": round(overlap, 5),
                    "abs_mass_vs_exact": round(mass, 6),
                    "k1": info["k1"], "band_taken": info["take"], "band": info["k2"] - info["k1"]}
    del pms, pe, pa, x_ref, r0, r1

    log("extras: dense aggregation of the P = 128 lists")
    outs = [[torch.empty(n, device=dev) for n in sizes] for _ in range(R)]
    aplans = [tk.UpdatePlan(sizes, P=P_WORKERS, stride=K_LIST).bind(outs[j]) for j in range(R)]
    ms, kern = time_calls(lambda i: aplans[i % R],
                          lambda pl: pl.aggregate(idx_all[aplans.index(pl)],
                                                  val_all[aplans.index(pl)], nnz=nnz),
                          K, W, make_events)
    pairs = k_total + (P_WORKERS - 1) * K_LIST
    ex["aggregate_us"] = round(ms * 1e3, 2)
    ex["aggregate_GBps"] = round((4 * d + 8 * pairs) / (ms / 1e3) / 1e9, 1)
    ex["aggregate_kernels_us"] = kern
    del outs, aplans

    log("extras: the momentum update with each position summed in worker order")
    dw = [[t.clone() for t in bank[j % len(bank)]] for j in range(R)]   # parameters
    db = [[torch.zeros_like(t) for t in bank[0]] for _ in range(R)]
    dplans = [tk.UpdatePlan(sizes, P=P_WORKERS, stride=K_LIST, deterministic=True)
              .bind(dw[j], db[j]) for j in range(R)]
    ms, kern = time_calls(lambda i: dplans[i % R],
                          lambda pl: pl.execute(idx_all[dplans.index(pl)],
                                                val_all[dplans.index(pl)], lr=LR, mu=MU, wd=WD,
                                                nnz=nnz),
                          K, W, make_events)
    ex["update_deterministic_us"] = round(ms * 1e3, 2)
    ex["update_deterministic_kernels_us"] = kern
    del dw, db, dplans

    log("extras: LARS (Eq. lars) step fused with the P = 128 aggregate; dense rates")
    lw = [[t.clone() for t in bank[j % len(bank)]] for j in range(R)]   # parameters
    lb = [[torch.zeros_like(t) for t in bank[0]] for _ in range(R)]     # momentum
    lplans = [tk.UpdatePlan(sizes, P=P_WORKERS, stride=K_LIST).bind(lw[j], lb[j]) for j in range(R)]
    names = list(tk.LARS_LAUNCHES)

    def lars_run(i, t=None):
        j = i % R
        if t is not None:
            lplans[j].set_events(t)
        lplans[j].lars_execute(idx_all[j], val_all[j], 0.001, LR, WD, mu=MU, nnz=nnz)
        if t is not None:
            lplans[j].set_events(None)

    for i in range(W):
        lars_run(i)
    evs = [make_events(len(names) + 1) for _ in range(K)]
    torch.cuda.synchronize()
    for t in range(K):
        lars_run(W + t, evs[t])
    torch.cuda.synchronize()
    import numpy as np
    ms = float(np.mean([e[0].elapsed_time(e[-1]) for e in evs]))
    kern = {n: round(float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) * 1e3, 2)
            for i, n in enumerate(names)}
    pairs = k_total + (P_WORKERS - 1) * K_LIST
    lbytes = 20 * d + 16 * pairs   # norm pass: w + lists; step: w, b in and out + lists
    ex["lars_update"] = {"us": round(ms * 1e3, 2), "GBps": round(lbytes / (ms / 1e3) / 1e9, 1),
                         "algorithmic_bytes": lbytes, "kernels_us": kern}
    del lplans, lw, lb
    for model, shapes in (("resnet50", gen.resnet50_shapes()), ("transformer", gen.transformer_shapes())):
        szs = gen.numels(shapes)
        dd = sum(szs)
        ws_ = [torch.randn(n, device=dev) * 0.05 for n in szs]
        gs_ = [torch.randn(n, device=dev) * 1e-3 for n in szs]
        rp = tk.UpdatePlan(szs, P=1, stride=0).bind(ws_)
        rp.bind_grads(gs_)
        rates = torch.empty(len(szs), dtype=torch.float64, device=dev)
        dn = list(tk.LARS_DENSE_LAUNCHES)
        for _ in range(W):
            rp.lars_rates(0.001, LR, WD, rates=rates)
        evs = [make_events(len(dn) + 1) for _ in range(K)]
        torch.cuda.synchronize()
        for t in range(K):
            rp.set_events(evs[t])
            rp.lars_rates(0.001, LR, WD, rates=rates)
            rp.set_events(None)
        torch.cuda.synchronize()
        ms = float(np.mean([e[0].elapsed_time(e[-1]) for e in evs]))
        ex[f"lars_rates_{model}"] = {
            "layers": len(szs), "d": dd, "us": round(ms * 1e3, 2),
            "GBps": round(8 * dd / (ms / 1e3) / 1e9, 1),
            "kernels_us": {n: round(float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) * 1e3, 2)
                           for i, n in enumerate(dn)}}
        del rp, ws_, gs_

    log("extras: shard-shaped sparsify (1 of 8 shards)")
    n_sh = 8
    shard = -(-d // n_sh)
    k_sh = -(-d // (n_sh * 1000))          # ceil(rho d / 8) with rho = 1/1000
    flats = [torch.from_numpy(gen.flat_normal(d, config=2, step=s, std=1e-2)).to(dev)
             for s in range(2)]
    rflat = [torch.zeros(d, device=dev) for _ in range(2)]
    # the 7 full shards of two gradients: 14 plans, 360 MB of g and r, rotated
    # so that no call finds its inputs in the last-level cache
    splans = [tk.SparsifyPlan([shard], k=k_sh).bind([flats[s][q * shard:(q + 1) * shard]],
                                                     [rflat[s][q * shard:(q + 1) * shard]])
              for s in range(2) for q in range(n_sh - 1)]
    si = torch.empty(k_sh, dtype=torch.int32, device=dev)
    sv = torch.empty(k_sh, dtype=torch.float32, device=dev)
    ms, kern = time_calls(lambda i: splans[i % len(splans)], lambda pl: pl.execute(si, sv),
                          max(K, 2 * len(splans)), len(splans), make_events)
    ex["shard"] = {"d": shard, "k": k_sh, "shards_rotated": len(splans),
                   "sparsify_us": round(ms * 1e3, 2),
                   "Gelem_per_s": round(shard / (ms / 1e3) / 1e9, 2),
                   "frac_hbm_peak": round((12 * shard + 8 * k_sh) / (ms / 1e3) / 1e9
                                          / HBM_PEAK_GBPS, 4),
                   "kernels_us": kern}
    return ex


def time_sparsify(tk, plans, K, W, make_events, idx_out=None, val_out=None):
    """Mean total and per-kernel times (ms) of plans[i % len(plans)].execute()."""
    import numpy as np
    import torch
    names = plans[0].launch_names()
    for i in range(W):
        plans[i % len(plans)].execute(idx_out, val_out)
    evs = [make_events(len(names) + 1) for _ in range(K)]
    torch.cuda.synchronize()
    for t in range(K):
        pl = plans[(W + t) % len(plans)]
        pl.set_events(evs[t])
        pl.execute(idx_out, val_out)
        pl.set_events(None)
    torch.cuda.synchronize()
    total = float(np.mean([e[0].elapsed_time(e[-1]) for e in evs]))
    kern = {n: round(float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) * 1e3, 2)
            for i, n in enumerate(names)}
    return total, kern


def other_workload(args) -> int:
    """The other configurations: sparsify rates (and, for c1, the one-worker
    plain update), inputs resident, rotating buffers larger than the last-
    level cache."""
    import numpy as np
    import torch

    import gen
    import paper_2010_10458_amd as tk

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    K, W = args.steps, args.warmup

    def make_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    def line(metric_value, d, ms, kern, workload, extra):
        frac = (12 * d) / (ms / 1e3) / 1e9 / HBM_PEAK_GBPS
        out = {"metric": METRIC, "value": round(metric_value, 3), "unit": "Gelem/s", "n_gpus": 1,
               "steps": K, "warmup": W, "ms_per_step": round(ms, 4), "higher_is_better": True,
               "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
               "config": {"workload": workload, "d": d}, "sparsify_us": round(ms * 1e3, 2),
               "sparsify_frac_hbm_peak": round(frac, 4), "kernels_us": kern}
        out.update(extra)
        print(json.dumps(out), flush=True)

    if args.workload == "c1":
        d = gen.C1_D
        R = 64   # 64 x (g, r, w) of 4 MB: more than the 256 MB last-level cache
        gs = [[torch.from_numpy(gen.flat_normal(d, config=1, step=j % 4)).to(dev)] for j in range(R)]
        rs = [[torch.zeros(d, device=dev)] for _ in range(R)]
        ws = [[torch.from_numpy(gen.params_like([d], config=1)[0]).to(dev)] for _ in range(R)]
        sps = [tk.SparsifyPlan([d], rho=RHO).bind(gs[j], rs[j]) for j in range(R)]
        k = sps[0].k_total
        ups = [tk.UpdatePlan([d], P=1, stride=k).bind(ws[j]) for j in range(R)]
        idx = [torch.empty(k, dtype=torch.int32, device=dev) for _ in range(R)]
        val = [torch.empty(k, device=dev) for _ in range(R)]
        n_sp, n_up = len(sps[0].launch_names()), len(ups[0].launch_names())
        for i in range(W):
            sps[i % R].execute(idx[i % R], val[i % R])
            ups[i % R].execute(idx[i % R], val[i % R], lr=0.1)
        e_sp = [make_events(n_sp + 1) for _ in range(K)]
        e_up = [make_events(n_up + 1) for _ in range(K)]
        torch.cuda.synchronize()
        for t in range(K):
            j = (W + t) % R
            sps[j].set_events(e_sp[t])
            sps[j].execute(idx[j], val[j])
            sps[j].set_events(None)
            ups[j].set_events(e_up[t])
            ups[j].execute(idx[j], val[j], lr=0.1)
            ups[j].set_events(None)
        torch.cuda.synchronize()
        sp_ms = float(np.mean([e[0].elapsed_time(e[-1]) for e in e_sp]))
        up_ms = float(np.mean([e[0].elapsed_time(e[-1]) for e in e_up]))
        kern = {n: round(float(np.mean([e[i].elapsed_time(e[i + 1]) for e in e_sp])) * 1e3, 2)
                for i, n in enumerate(sps[0].launch_names())}
        line(d / (sp_ms / 1e3) / 1e9, d, sp_ms, kern,
             "single fp32 tensor d=1048576, N(0,1), residual zero, rho=0.001 (k=1049); then a "
             "one-worker plain SGD update, lr 0.1", {"k": k, "update_us": round(up_ms * 1e3, 2)})
        return 0

    if args.workload == "transformer":
        sizes = gen.numels(gen.transformer_shapes())
        d = sum(sizes)
        bank = [[torch.from_numpy(a).to(dev) for a in gen.laplace_grads(s, sizes)] for s in range(2)]
        res = {}
        for mode, mname in ((tk.GLOBAL, "global"), (tk.PER_TENSOR, "per_tensor")):
            for rho in (0.001, 0.01):
                # fresh residuals per configuration (each carries its own error feedback)
                resid = [[torch.zeros(n, device=dev) for n in sizes] for _ in range(2)]
                plans = [tk.SparsifyPlan(sizes, mode=mode, rho=rho).bind(bank[s], resid[j])
                         for s in range(2) for j in range(2)]
                ms, kern = time_sparsify(tk, plans, K, W, make_events)
                res[f"{mname}_rho{rho}"] = {"k": plans[0].k_total, "sparsify_us": round(ms * 1e3, 2),
                                            "Gelem_per_s": round(d / (ms / 1e3) / 1e9, 2),
                                            "frac_hbm_peak": round((12 * d + 8 * plans[0].k_total) / (ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
                                            "kernels_us": kern}
                del plans, resid
        head = res["global_rho0.001"]
        line(head["Gelem_per_s"], d, head["sparsify_us"] / 1e3, head["kernels_us"],
             "transformer-base-shaped set: 261 fp32 tensors, d=109708544, Laplace(0, 1e-3); rho "
             "0.001 and 0.01, global and per-tensor top-k", {"variants": res})
        return 0

    if args.workload == "sweep":
        # flat N(0, 1) vectors of 2^18 .. 2^27 elements (the 256 K .. 128 M
        # operator range of Sec. 5.2), k = ceil(0.001 d). Gradients are eight
        # slices of one 2^28-element buffer, residuals disjoint slices of
        # another, zeroed for each size; call i takes gradient slice i % 8 and
        # residual i % R, so consecutive calls on one residual see different
        # gradients (as error feedback does), and there are enough residuals
        # (at least 768 MiB of g and r together) that no call finds its
        # inputs in the 256 MB last-level cache.
        total, n_g = 1 << 28, 8
        log("generating the 2^28-element sweep buffer")
        G = torch.from_numpy(gen.flat_normal(total, config=6)).to(dev)
        Rb = torch.zeros(total, device=dev)
        rows = []
        for e in range(18, 28):
            d = 1 << e
            R = max(2, min(total // d, -(-(768 << 20) // (8 * d))))
            gstep = (total - d) // (n_g - 1) // 4096 * 4096
            Rb.zero_()
            plans = [tk.SparsifyPlan([d], rho=RHO).bind(
                [G[(i % n_g) * gstep:(i % n_g) * gstep + d]],
                [Rb[(i % R) * d:(i % R + 1) * d]]) for i in range(max(n_g, R))]
            k = plans[0].k_total
            io = torch.empty(k, dtype=torch.int32, device=dev)
            vo = torch.empty(k, device=dev)
            ms, kern = time_sparsify(tk, plans, K, W, make_events, io, vo)
            rows.append({"d": d, "k": k, "replicas": R, "sparsify_us": round(ms * 1e3, 2),
                         "Gelem_per_s": round(d / (ms / 1e3) / 1e9, 2),
                         "frac_hbm_peak": round((12 * d + 8 * k) / (ms / 1e3) / 1e9
                                                / HBM_PEAK_GBPS, 4),
                         "kernels_us": kern})
            log(f"sweep d=2^{e}: {rows[-1]['sparsify_us']} us")
            del plans
        top = rows[-1]
        line(top["Gelem_per_s"], top["d"], top["sparsify_us"] / 1e3, top["kernels_us"],
             "sweep: flat fp32 N(0,1) vectors, d = 2^18 .. 2^27, residual carried over rotating "
             "gradients, global top-k rho=0.001", {"sweep": rows})
        return 0

    # bert: one 340 M-element buffer with exact-duplicate magnitudes
    d = gen.BERT_LARGE_D
    log("generating the 340 M-element tie-stressed buffer")
    g = [torch.from_numpy(gen.tie_stressed(d)).to(dev)]
    resid = [[torch.zeros(d, device=dev)] for _ in range(2)]
    plans = [tk.SparsifyPlan([d], rho=RHO).bind(g, resid[j]) for j in range(2)]
    ms, kern = time_sparsify(tk, plans, K, W, make_events)
    line(d / (ms / 1e3) / 1e9, d, ms, kern,
         "bert-large-sized flat fp32 buffer d=340000000, N(0,1) with 10% bfloat16-truncated "
         "exact-duplicate magnitudes and a tie class at the rho=0.001 boundary",
         {"k": plans[0].k_total})
    return 0


def main() -> int:
    args = parse_args()
    if args.probe_copy:
        return probe_copy(args.probe_copy)
    if args.probe_add:
        return probe_add(args.probe_add)
    if args.summarize_stats:
        return summarize_stats(args.summarize_stats)
    if args.summarize_pmc:
        return summarize_pmc(*args.summarize_pmc)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the library has no multi-GPU path); "
              f"got --gpus {args.gpus}", file=sys.stderr)
        return 2
    if args.workload != "resnet50":
        return other_workload(args)
    import numpy as np
    import torch

    import gen
    import paper_2010_10458_amd as tk

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    R = args.replicas

    log(f"generating inputs: d={d}, {GRAD_STEPS} gradient steps, {R} replicas")
    bank = []
    for s in range(GRAD_STEPS):
        bank.append([torch.from_numpy(a).to(dev) for a in gen.resnet_grads(s)])
    resid = [[torch.zeros(n, device=dev) for n in sizes] for _ in range(R)]
    w0 = gen.params_like(sizes, config=5)
    params = [[torch.from_numpy(a).to(dev) for a in w0] for _ in range(R)]
    mom = [[torch.zeros(n, device=dev) for n in sizes] for _ in range(R)]
    idx_all, val_all = [], []
    for j in range(R):
        li, lv = gen.sparse_lists(d, P_WORKERS, K_LIST, step=100 + j)
        idx_all.append(torch.from_numpy(li).to(dev))
        val_all.append(torch.from_numpy(lv).to(dev))

    plans = [[tk.SparsifyPlan(sizes, rho=RHO) for _ in range(R)] for _ in range(GRAD_STEPS)]
    for s in range(GRAD_STEPS):
        for j in range(R):
            plans[s][j].bind(bank[s], resid[j])
    k_total = plans[0][0].k_total
    uplans = [tk.UpdatePlan(sizes, P=P_WORKERS, stride=K_LIST).bind(params[j], mom[j])
              for j in range(R)]
    nnz = torch.tensor([k_total] + [K_LIST] * (P_WORKERS - 1), dtype=torch.int32, device=dev)
    sp_names = plans[0][0].launch_names()
    up_names = uplans[0].launch_names()
    n_sp, n_up = len(sp_names) + 1, len(up_names) + 1
    if not args.kernel_events:
        n_sp = n_up = 1

    def make_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    K, W = args.steps, args.warmup
    ev_sp = [make_events(max(n_sp, 2)) for _ in range(K)]
    ev_up = [make_events(max(n_up, 2)) for _ in range(K)]
    torch.cuda.synchronize()

    def step(i, t=None):
        s, j = i % GRAD_STEPS, i % R
        sp, up = plans[s][j], uplans[j]
        if t is not None and args.kernel_events:
            sp.set_events(ev_sp[t])
            up.set_events(ev_up[t])
        elif t is not None:
            ev_sp[t][0].record()
        sp.execute(idx_out=idx_all[j][0], val_out=val_all[j][0])
        if t is not None and not args.kernel_events:
            ev_sp[t][1].record()
            ev_up[t][0].record()
        up.execute(idx_all[j], val_all[j], lr=LR, mu=MU, wd=WD, nnz=nnz)
        if t is not None and not args.kernel_events:
            ev_up[t][1].record()
        if t is not None and args.kernel_events:
            sp.set_events(None)
            up.set_events(None)

    log(f"warmup {W} steps")
    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    log(f"timing {K} steps")
    t0 = time.perf_counter()
    for t in range(K):
        step(W + t, t)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log("timed region done")

    sp_ms = np.array([ev_sp[t][0].elapsed_time(ev_sp[t][-1]) for t in range(K)])
    up_ms = np.array([ev_up[t][0].elapsed_time(ev_up[t][-1]) for t in range(K)])
    kern = {}
    if args.kernel_events:
        for names, evs in ((sp_names, ev_sp), (up_names, ev_up)):
            for i, name in enumerate(names):
                kern[name] = float(np.mean([evs[t][i].elapsed_time(evs[t][i + 1])
                                            for t in range(K)]))

    sp_s = float(sp_ms.mean()) / 1e3
    up_s = float(up_ms.mean()) / 1e3
    sp_bytes = 12 * d + 8 * k_total
    total_pairs = k_total + (P_WORKERS - 1) * K_LIST
    up_bytes = 16 * d + 8 * total_pairs
    algo = {"stream": 12 * d, "update": 16 * d + 8 * total_pairs, "emit": 8 * k_total}

    roofline = None
    if kern:
        dom = max(kern, key=kern.get)
        bytes_per_launch = algo.get(dom, 0)
        achieved = bytes_per_launch / (kern[dom] / 1e3) / 1e9
        digest = kernel_source_digest()
        roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBPS, 4),
                    "traffic": None,
                    "algorithmic_bytes_per_launch": bytes_per_launch,
                    "mean_launch_us": round(kern[dom] * 1e3, 2),
                    "source_digest": digest}
        tr = read_traffic(dom, digest)
        if tr is not None:
            roofline["traffic"] = round(tr["bytes"])
            roofline["traffic_raw"] = {k: v for k, v in tr.items() if k != "bytes"}

    out = {
        "metric": METRIC,
        "value": round(d / sp_s / 1e9, 3),
        "unit": "Gelem/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(wall / K * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "resnet50-shaped gradient set: 161 fp32 tensors, d=25557032, "
                               "N(0,1e-2) with 1% x100 outliers, residual carried; global top-k "
                               "rho=0.001; then P=128 aggregate-update (25,600-pair lists), "
                               "momentum 0.9, wd 5e-5, lr 0.1",
                   "d": d, "k": k_total, "rho": RHO, "P": P_WORKERS, "replicas": R},
        "sparsify_us": round(sp_s * 1e6, 2),
        "sparsify_GBps": round(sp_bytes / sp_s / 1e9, 1),
        "sparsify_frac_hbm_peak": round(sp_bytes / sp_s / 1e9 / HBM_PEAK_GBPS, 4),
        "sparsify_us_p10_p50_p90": [round(float(v) * 1e3, 2)
                                    for v in np.percentile(sp_ms, [10, 50, 90])],
        "update_us": round(up_s * 1e6, 2),
        "update_us_p10_p50_p90": [round(float(v) * 1e3, 2)
                                  for v in np.percentile(up_ms, [10, 50, 90])],
        "update_GBps": round(up_bytes / up_s / 1e9, 1),
        "update_frac_hbm_peak": round(up_bytes / up_s / 1e9 / HBM_PEAK_GBPS, 4),
        "kernels_us": {k: round(v * 1e3, 2) for k, v in kern.items()},
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if not args.no_extras:
        out["extras"] = extras(args, tk, gen, sizes, d, bank, resid, idx_all, val_all, nnz,
                               k_total, make_events)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on one step (bounded sample)")
        out["cpu_baseline"] = cpu_baseline(sizes, d, args.cpu_procs)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

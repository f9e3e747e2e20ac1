#!/usr/bin/env python3
"""Benchmark of the multi-table embedding-bag lookup on one MI355X.

One step = one emb_lookup over one batch of the workload (all tables, all
samples).  Inputs (tables, indices, offsets) are resident in HBM before timing;
R distinct batches are cycled.  Prints ONE JSON line:

  value            lookups/s over the K timed steps (whole job, one GPU), one batch at a time
                   on one stream.  With --streams S > 1 the steps of another timed pass are
                   dealt round-robin to S streams (one plan per stream, each writing its own
                   output), so that one batch's last workers overlap the next batch's first;
                   value and ms_per_step then come from that pass, and single_stream holds
                   the one-stream figures (a kernel trace then also holds the overlapped
                   dispatches, whose begin-to-end times are longer than launch_us)
  queries_per_s    samples/s (the paper's TPS), from the same pass as value
  p99_us           nearest-rank P99 of the per-batch latency (a separate pass of 1000
                   batches, 200 for workload 5, with HIP events around each launch;
                   mean_us is that pass's mean)
  cold_cache       the same latency with L2 and MALL flushed (a 512 MiB write) before
                   each batch, outside the timed region
  launch_us        average launch duration over the K single-stream steps (one HIP event
                   pair on the launch stream around the back-to-back launches); this pass runs
                   last, so that a kernel trace's last K dispatches are these
  useful_hbm_frac  (lookups x row bytes) per launch_us over the 8 TB/s HBM peak: every
                   lookup's row counted, also when L2 or the MALL serves it (can exceed 1)
  roofline         compulsory bytes per launch over launch_us, against the 8 TB/s HBM peak:
                   each distinct row of the batch once (row bytes), 8 B per index (+4 B per
                   weight), 8 B per offset, 4E B per pooled output -- what has to cross HBM
                   at least once, so frac <= 1; traffic = measured bytes per launch beyond L2
                   (profiles/traffic_<workload>.json: FETCH_SIZE and WRITE_SIZE, each scaled by
                   its reading for a 1 GiB device copy) when the committed counters were taken
                   on this kernel source, else null
  launch_floor_us  back-to-back interval of a one-workgroup kernel launched through the same
                   ctypes path and stream (the floor of launch_us)
  cpu_baseline     the CPU oracle timed on a bounded sample of the same workload; beside it
                   (torch_embedding_bag) torch's CPU embedding_bag on the same sample, with
                   the threads it used, for unweighted runs

  python bench.py [--config 5] [--steps 200] [--warmup 20] [--streams 1]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "embedding lookups/s + queries/s, P99 batch latency, % HBM peak (1 MI355X)"
DEFAULT_CONFIG = 5
# what decides a launch's memory traffic: the kernels and the plan (planner + metadata);
# a stored traffic measurement is used only while their hash is unchanged
KERNEL_SOURCES = ["paper_2507_01676_amd/csrc/lookup.hip", "paper_2507_01676_amd/csrc/gather.hip",
                  "paper_2507_01676_amd/csrc/device_types.hpp",
                  "paper_2507_01676_amd/csrc/planner.cpp", "paper_2507_01676_amd/csrc/planner.hpp",
                  "paper_2507_01676_amd/csrc/api.cpp"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def p99(xs):
    s = sorted(xs)
    return s[max(0, math.ceil(0.99 * len(s)) - 1)]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(c: W.Config, batches, budget_s: float, pooling: str = "sum", psw=None):
    """The CPU oracle (plain NumPy, float64 accumulation) on a bounded sample of the workload
    (with the run's pooling and, for weighted runs, the same per-lookup weights)."""
    from oracle import pool as OP
    t0 = time.time()
    if c.cfg_id == 5:
        # the full table set (~130 GB) does not fit a host budget: the sample is the
        # tables of at most 500k rows (61 of 100, 2.8 GB), over a 4096-query sub-batch
        keep = [t for t, m in enumerate(c.rows) if m <= 500_000]
        Bs = 4096
    else:
        keep = list(range(c.T))
        Bs = c.batch
    weights = [W.materialize_table(t, c.rows[t], c.E, c.dtype, seed=c.value_seeds[t], lo=c.lo, hi=c.hi)
               for t in keep]
    log(f"cpu baseline: materialized {len(keep)} tables in {time.time() - t0:.1f}s")
    subs = []
    for bt in batches:
        B = bt.B
        Bs = min(Bs, B)
        parts, lens, wparts = [], [], []
        for t in keep:
            lo, hi = bt.offsets[t * B], bt.offsets[t * B + Bs]
            parts.append(bt.indices[lo:hi])
            lens.append(np.diff(bt.offsets[t * B: t * B + Bs + 1]))
            if psw is not None:
                wparts.append(psw[len(subs)][lo:hi])
        off = np.zeros(len(keep) * Bs + 1, np.int64)
        np.cumsum(np.concatenate(lens), out=off[1:])
        subs.append((np.concatenate(parts), off, np.concatenate(wparts) if psw is not None else None))
    lat = []
    n_look = 0
    start = time.perf_counter()
    i = 0
    while True:
        idx, off, wk = subs[i % len(subs)]
        t1 = time.perf_counter()
        OP.pool_reference(weights, idx, off, Bs, pooling=pooling, psw=wk)
        lat.append(time.perf_counter() - t1)
        n_look += int(off[-1])
        i += 1
        if (time.perf_counter() - start >= budget_s and i >= 3) or i >= 1000:
            break
    tot = sum(lat)
    sample = (f"{'all' if len(keep) == c.T else len(keep)} of {c.T} tables, {Bs}-query batches, "
              f"{i} batches cycled over {len(subs)} distinct")
    res = {"value": n_look / tot, "unit": "lookups/s", "cores": 1, "kind": "oracle", "sample": sample,
           "queries_per_s": Bs * i / tot, "p99_us": p99(lat) * 1e6, "cpu_model": cpu_model(),
           "cpu_count": os.cpu_count()}
    if psw is None:
        res["torch_embedding_bag"] = torch_cpu_reference(weights, subs, Bs, budget_s / 2, pooling)
    return res


def torch_cpu_reference(weights, subs, Bs: int, budget_s: float, pooling: str):
    """A second CPU reference on the same sample: torch.nn.functional.embedding_bag per
    table (fp32, torch's own thread pool), timed like the oracle."""
    import torch
    import torch.nn.functional as F
    tw = [torch.from_numpy(np.ascontiguousarray(w, dtype=np.float32)) for w in weights]
    T = len(tw)
    prepared = []
    for idx, off, _ in subs:
        ti = torch.from_numpy(idx)
        starts = [torch.from_numpy(off[t * Bs:(t + 1) * Bs] - off[t * Bs]) for t in range(T)]
        prepared.append((ti, [(int(off[t * Bs]), int(off[(t + 1) * Bs])) for t in range(T)], starts, int(off[-1])))
    lat, n_look, i = [], 0, 0
    start = time.perf_counter()
    while True:
        ti, spans, starts, n = prepared[i % len(prepared)]
        t1 = time.perf_counter()
        out = torch.stack([F.embedding_bag(ti[a:b], tw[t], starts[t], mode=pooling)
                           for t, (a, b) in enumerate(spans)], dim=1)
        lat.append(time.perf_counter() - t1)
        del out
        n_look += n
        i += 1
        if (time.perf_counter() - start >= budget_s and i >= 3) or i >= 1000:
            break
    tot = sum(lat)
    return {"value": n_look / tot, "unit": "lookups/s", "threads": torch.get_num_threads(),
            "queries_per_s": Bs * i / tot, "p99_us": p99(lat) * 1e6, "batches": i}


def copy_bandwidth_gbps() -> float:
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 10
    del a, b
    return 2 * n / (ms * 1e-3) / 1e9


def launch_floor_us(stream) -> float:
    """Back-to-back interval of a near-empty kernel (the library's table filler on one
    row of 4 floats: one workgroup) launched through the same ctypes path and stream as
    the timed lookups: the per-launch cost that no launch of this loop goes below."""
    import torch
    import paper_2507_01676_amd as embx
    x = torch.empty((1, 4), device="cuda")
    ptr, sp = x.data_ptr(), stream.cuda_stream

    def launch():
        embx.fill_table_ptr(ptr, 0, 1, 4, embx.DTYPE_F32, 0, 1, 0.0, 1.0, 0, sp)
    for _ in range(20):
        launch()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(500):
        launch()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / 500


def load_traffic(workload: str, src_hash: str):
    """HBM bytes per launch from the committed counter summary, if it matches this kernel."""
    p = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        d = json.load(f)
    if d.get("kernel_source_hash") != src_hash:
        return None
    return d.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=DEFAULT_CONFIG, help="workload 1..5")
    ap.add_argument("--batches", type=int, default=0, help="distinct resident batches (default 8, 4 for workload 5)")
    ap.add_argument("--p99-batches", type=int, default=0, help="latency pass length (default 1000; 200 for workload 5)")
    ap.add_argument("--cold-batches", type=int, default=20, help="batches timed after a cache-flushing write (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-copy", action="store_true")
    ap.add_argument("--lds-budget", type=int, default=0)
    ap.add_argument("--force", type=str, default="", help="force one strategy for all tables (lds|hot|dedup|gather|stream)")
    ap.add_argument("--pooling", choices=["sum", "mean"], default="sum", help="reduction of every table's bags")
    ap.add_argument("--weighted", action="store_true", help="per-lookup weights (emb_lookup_weighted)")
    ap.add_argument("--dist", choices=list(W.DISTRIBUTIONS), default="config",
                    help="query distribution of every table: the workload's own, uniform, or fixed "
                         "(every lookup of a table on one row)")
    ap.add_argument("--lif-milli", type=int, default=0,
                    help="load-imbalance threshold x 1000 of the symmetric fallback (0: the library default)")
    ap.add_argument("--sym-max", type=int, default=0,
                    help="gather tables split over all workers while at most this many (0: the library default)")
    ap.add_argument("--order-mode", type=int, default=0, choices=[0, 1],
                    help="slice order of the placement: 0 longest first, 1 the paper's (s desc, m asc)")
    ap.add_argument("--no-replication", action="store_true",
                    help="no batch splits (replication 1); with --order-mode 1 the paper's solver as printed")
    ap.add_argument("--table-costs", type=int, default=0,
                    help="rounds of per-table lookup-cost calibration before timing: traced launches of "
                         "the plan over the resident batches, a fit of each table's cost of a lookup "
                         "served from memory, and a re-plan with those costs (0: the vector's G1 for all)")
    ap.add_argument("--streams", type=int, default=1, choices=[1, 2, 3, 4],
                    help="streams a second throughput pass deals its steps to (1: none, one batch at a time)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the lookup runs on a single MI355X "
              "(multi-GPU sharding is a design note here, not implemented); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2507_01676_amd as embx
    assert torch.cuda.is_available(), "no GPU"
    torch.cuda.set_device(0)

    c = W.with_distribution(W.make_config(args.config), args.dist)
    R = args.batches or (4 if args.config == 5 else 8)
    t0 = time.time()
    log(f"workload {c.cfg_id}: {c.name}; generating {R} batches + statistics")
    batches = []
    for i in range(R):
        batches.append(W.gen_batch(c, i))
        log(f"batch {i}: {batches[-1].n_lookups} lookups ({time.time() - t0:.1f}s)")
    stats = W.history_stats(c)
    log(f"inputs generated in {time.time() - t0:.1f}s; filling {sum(c.rows) * c.row_bytes / 1e9:.2f} GB of tables")
    dt = torch.float16 if c.dtype == "f16" else torch.float32
    weights = []
    for t, m in enumerate(c.rows):
        w = torch.empty((m, c.E), dtype=dt, device="cuda")
        embx.fill_table(w, t, c.value_seeds[t], c.lo, c.hi)
        weights.append(w)
    d_idx = [torch.from_numpy(b.indices).cuda() for b in batches]
    d_off = [torch.from_numpy(b.offsets).cuda() for b in batches]
    # weighted runs: seeded per-lookup weights, uniform in [0.5, 1.5)
    psw = [np.random.default_rng(1000 + i).uniform(0.5, 1.5, size=b.indices.size).astype(np.float32)
           for i, b in enumerate(batches)] if args.weighted else None
    d_w = [torch.from_numpy(x).cuda() for x in psw] if psw is not None else None
    out = torch.empty((c.batch, c.T, c.E), dtype=torch.float32, device="cuda")
    opts = {}
    if args.lds_budget:
        opts["lds_budget"] = args.lds_budget
    if args.force:
        opts["force"] = [{"lds": 0, "hot": 1, "dedup": 2, "gather": 3, "stream": 4}[args.force]] * c.T
    if args.pooling != "sum":
        opts["pooling"] = args.pooling
    if args.sym_max:
        opts["sym_max"] = args.sym_max
    if args.lif_milli:
        opts["lif_milli"] = args.lif_milli
    if args.order_mode:
        opts["order_mode"] = args.order_mode
    if args.no_replication:
        opts["no_replication"] = True
    tp = time.time()
    plan = embx.Plan(c.rows, c.E, c.dtype, stats, c.batch, **opts).bind(weights)
    plan_ms = (time.time() - tp) * 1e3
    info = plan.info()
    torch.cuda.synchronize()
    log(f"plan: {info['n_strategy']} items={info['num_items']} lif={info['lif_milli']} ({plan_ms:.1f} ms)")

    table_costs = None
    if args.table_costs > 0:
        # closed loop per table: the plan's traced launches over the resident batches, one
        # fit of every table's cost per lookup on all of them, a re-plan with those costs
        from paper_2507_01676_amd import calibrate as CAL
        g0 = (opts.get("beta") or embx.default_beta(c.row_bytes))[0]
        for rnd in range(args.table_costs):
            ps, ns, lams = [], [], []
            for i in range(R):
                # the batch before it first, as in the timed loop: its rows are not the
                # ones left in the caches
                plan.lookup(d_idx[(i - 1) % R], d_off[(i - 1) % R], c.batch, out)
                tr = CAL.traced_launch(plan, d_idx[i], d_off[i], c.batch, out, warm=0)
                a, n, lm = CAL.worker_gather_samples(plan, tr, c.batch, batches[i].offsets, c.T)
                ps.append(a)
                ns.append(n)
                lams.append(lm)
            table_costs = CAL.fit_table_lookup_costs(np.concatenate(ps), np.concatenate(ns), np.concatenate(lams), g0)
            opts["gather_lookup_ps"] = table_costs
            plan.close()
            tp = time.time()
            plan = embx.Plan(c.rows, c.E, c.dtype, stats, c.batch, **opts).bind(weights)
            plan_ms = (time.time() - tp) * 1e3
            info = plan.info()
            log(f"table costs round {rnd + 1}: " + " ".join(f"{x / 1e3:.1f}" for x in table_costs)
                + f" ns; plan items={info['num_items']} lif={info['lif_milli']}")
        torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    ptrs = [(d_idx[i].data_ptr(), d_off[i].data_ptr()) for i in range(R)]
    wptr = [d_w[i].data_ptr() if d_w is not None else 0 for i in range(R)]
    n_look = [b.n_lookups for b in batches]
    outp = out.data_ptr()
    B = c.batch

    for i in range(args.warmup):
        ip, op = ptrs[i % R]
        plan.lookup_ptr(ip, op, B, outp, sp, wptr[i % R])
    torch.cuda.synchronize()
    assert plan.check_errors() == 0

    K = args.steps
    # per-batch latency (P99): an event pair around each launch, over N batches
    N = args.p99_batches or (200 if args.config == 5 else 1000)
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(N)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(N)]
    torch.cuda.synchronize()
    for i in range(N):
        ip, op = ptrs[i % R]
        ev0[i].record(stream)
        plan.lookup_ptr(ip, op, B, outp, sp, wptr[i % R])
        ev1[i].record(stream)
    torch.cuda.synchronize()
    lat_ms = [ev0[i].elapsed_time(ev1[i]) for i in range(N)]

    # cold caches: before each of these batches a 512 MiB buffer is written (outside the
    # timed region), which evicts the tables' rows from L2 and the MALL
    cold = None
    if args.cold_batches > 0:
        flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        c0 = [torch.cuda.Event(enable_timing=True) for _ in range(args.cold_batches)]
        c1 = [torch.cuda.Event(enable_timing=True) for _ in range(args.cold_batches)]
        for i in range(args.cold_batches):
            flush.fill_(i & 0xFF)
            ip, op = ptrs[i % R]
            c0[i].record(stream)
            plan.lookup_ptr(ip, op, B, outp, sp, wptr[i % R])
            c1[i].record(stream)
        torch.cuda.synchronize()
        cl = [c0[i].elapsed_time(c1[i]) for i in range(args.cold_batches)]
        cmean = sum(cl) / len(cl)
        cuse = sum(n_look[i % R] for i in range(args.cold_batches)) * c.row_bytes / len(cl)
        cold = {"batches": len(cl), "mean_us": cmean * 1e3, "p99_us": p99(cl) * 1e3,
                "useful_gbps": cuse / (cmean * 1e-3) / 1e9}
        del flush

    total_lookups = sum(n_look[i % R] for i in range(K))
    # throughput: the K steps dealt round-robin to S streams, each with its own plan (the
    # same tables) and output, synchronized on both sides of the timed region
    S = args.streams
    pipe = None
    if S > 1:
        plans = [plan] + [embx.Plan(c.rows, c.E, c.dtype, stats, c.batch, **opts).bind(weights) for _ in range(S - 1)]
        side = [torch.cuda.Stream() for _ in range(S)]
        outs = [out] + [torch.empty_like(out) for _ in range(S - 1)]
        sps, ops = [x.cuda_stream for x in side], [x.data_ptr() for x in outs]

        def dealt(n):
            for x in side:
                x.wait_stream(stream)
            for i in range(n):
                ip, op = ptrs[i % R]
                plans[i % S].lookup_ptr(ip, op, B, ops[i % S], sps[i % S], wptr[i % R])
            for x in side:
                stream.wait_stream(x)
        dealt(max(args.warmup, S))
        torch.cuda.synchronize()
        wallp0 = time.perf_counter()
        dealt(K)
        torch.cuda.synchronize()
        pipe = time.perf_counter() - wallp0
        for x in plans[1:]:
            assert x.check_errors() == 0
            x.close()
        del outs, plans
    # one batch at a time: the K steps back to back on one stream; one event pair on the
    # launch stream gives the average launch duration
    e_start, e_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e_start.record(stream)
    for i in range(K):
        ip, op = ptrs[i % R]
        plan.lookup_ptr(ip, op, B, outp, sp, wptr[i % R])
    e_stop.record(stream)
    torch.cuda.synchronize()
    wall1 = time.perf_counter() - wall0
    launch_ms = e_start.elapsed_time(e_stop) / K
    wall = pipe if pipe is not None else wall1
    mean_ms = sum(lat_ms) / len(lat_ms)

    R_b = c.row_bytes
    # weighted runs also read 4 bytes of weight per lookup
    alg = [W.algorithmic_bytes(c, n_look[i % R])["total"] + (4 * n_look[i % R] if args.weighted else 0)
           for i in range(K)]
    alg_mean = sum(alg) / K
    comp_batch = [W.compulsory_bytes(c, b, args.weighted) for b in batches]
    comp_mean = sum(comp_batch[i % R]["total"] for i in range(K)) / K
    useful_mean = sum(n_look[i % R] for i in range(K)) * R_b / K
    achieved = comp_mean / (launch_ms * 1e-3) / 1e9
    src_hash = kernel_source_hash()
    workload = f"workload{c.cfg_id}"
    variant = (("" if args.dist == "config" else f"-{args.dist}") + ("" if args.pooling == "sum" else f"-{args.pooling}")
               + ("-weighted" if args.weighted else ""))
    traffic = load_traffic(workload + variant, src_hash)

    copy_gbps = None if args.no_copy else copy_bandwidth_gbps()
    floor_us = launch_floor_us(stream)
    cpu = None
    if not args.no_cpu:
        log("timing the CPU oracle")
        cpu = cpu_baseline(c, batches, args.cpu_seconds, args.pooling, psw)

    res = {
        "metric": METRIC,
        "value": total_lookups / wall,
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{workload}{variant}: {c.name}", "tables": c.T, "E": c.E, "table_dtype": c.dtype,
                   "batch": c.batch, "lookups_per_batch": int(sum(n_look) / R), "resident_batches": R,
                   "table_bytes": sum(c.rows) * R_b, "pooling": args.pooling, "weighted": bool(args.weighted),
                   "queries": args.dist},
        "queries_per_s": B * K / wall,
        "streams": S,
        "single_stream": {"value": total_lookups / wall1, "ms_per_step": wall1 * 1e3 / K,
                          "queries_per_s": B * K / wall1},
        "p99_us": p99(lat_ms) * 1e3,
        "mean_us": mean_ms * 1e3,
        "launch_us": launch_ms * 1e3,
        "useful_gbps": useful_mean / (launch_ms * 1e-3) / 1e9,
        "useful_hbm_frac": useful_mean / (launch_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": traffic,
                     "traffic_over_compulsory": None if traffic is None else traffic / comp_mean,
                     "traffic_gbps": None if traffic is None else traffic / (launch_ms * 1e-3) / 1e9,
                     "compulsory_bytes_per_launch": comp_mean,
                     "compulsory_rows_bytes_per_launch": sum(comp_batch[i % R]["rows"] for i in range(K)) / K,
                     "per_lookup_bytes_per_launch": alg_mean,
                     "per_lookup_frac": alg_mean / (launch_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                     "kernel": info["kernel"]},
        "p99_batches": len(lat_ms),
        "cold_cache": cold,
        "copy_gbps": copy_gbps,
        "launch_floor_us": floor_us,
        "plan": {"kernel": info["kernel"], "strategies": info["n_strategy"], "items": info["num_items"],
                 "lif_milli": info["lif_milli"], "predicted_us": info["max_load_ps"] / 1e6,
                 "gather_steps": info["gather_steps"],
                 "workers": info["num_workers"], "lds_bytes": info["lds_bytes"], "build_ms": plan_ms,
                 "options": {k: opts[k] for k in ("lif_milli", "sym_max", "order_mode", "no_replication")
                             if k in opts},
                 "table_lookup_ps": None if table_costs is None else [round(x, 1) for x in table_costs],
                 "table_cost_rounds": args.table_costs},
        "kernel_source_hash": src_hash,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

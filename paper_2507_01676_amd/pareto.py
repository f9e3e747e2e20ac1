"""Batch-size sweep: throughput against P99 batch latency, re-planning per batch size.

The paper evaluates its mappings by sweeping the batch size and plotting average
throughput against P99 latency, keeping the Pareto front (Sec. IV, Fig. 4).  This
module does the same on the current device for the synthetic workloads: for each
batch size it builds a plan for that maximum batch (same tables and statistics),
times an event pair around each of ``n_p99`` launches (P99, nearest rank) and one
event pair around ``steps`` back-to-back launches (throughput), and marks the
points that no other point beats on both axes.  With ``streams`` above 1 a batch
size also gets a point with that many batches in flight: launches dealt round-robin
to as many streams, each with its own plan over the same tables and its own output;
its P99 is each launch's event pair on its own stream, so it includes the time the
launch waits for CUs that the other streams' batches still hold.

    python -m paper_2507_01676_amd.pareto --configs 2 3 4 --streams 1 2 --out profiles/pareto.md
"""
from __future__ import annotations

import json
import math
import sys
from typing import Dict, List, Sequence


def p99(xs: Sequence[float]) -> float:
    s = sorted(xs)
    return s[max(0, math.ceil(0.99 * len(s)) - 1)]


def pareto_front(points: List[Dict]) -> List[Dict]:
    """Points not dominated by another (throughput at least as high and P99 at most as
    low, one of them strictly)."""
    front = []
    for p in points:
        dominated = any((q["lookups_per_s"] >= p["lookups_per_s"] and q["p99_us"] <= p["p99_us"]) and
                        (q["lookups_per_s"] > p["lookups_per_s"] or q["p99_us"] < p["p99_us"]) for q in points)
        if not dominated:
            front.append(p)
    return front


def sweep(cfg: int, fractions: Sequence[float] = (1 / 16, 1 / 8, 1 / 4, 1 / 2, 1.0), steps: int = 100,
          warmup: int = 10, n_p99: int = 500, n_batches: int = 0, log=print, verify=None,
          streams: Sequence[int] = (1,)) -> List[Dict]:
    """One point per batch size (a fraction of the workload's batch) and number of batches
    in flight (``streams``): plans made for that batch, the time per batch back to back,
    the P99 of the launches, and whether the point is on the Pareto front.
    ``verify(config, batch, out)``, when given, is called once per batch size with the
    workload at that batch, resident batch 0 and its pooled output (a device tensor) from
    the first plan that is timed."""
    import torch
    import workloads as W
    from . import Plan, fill_table
    c = W.make_config(cfg)
    # distinct resident batches cycled, as bench.py does (fewer let a workload's rows stay
    # in the MALL from one batch to the next)
    n_batches = n_batches or (4 if cfg == 5 else 8)
    stats = W.history_stats(c)
    dt = torch.float16 if c.dtype == "f16" else torch.float32
    weights = []
    for t, m in enumerate(c.rows):
        w = torch.empty((m, c.E), dtype=dt, device="cuda")
        fill_table(w, t, c.value_seeds[t], c.lo, c.hi)
        weights.append(w)
    full = c.batch
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    out_pts = []
    for fr in fractions:
        B = max(1, int(round(full * fr)))
        c.batch = B
        batches = [W.gen_batch(c, i) for i in range(n_batches)]
        smax = max(streams)
        plans = [Plan(c.rows, c.E, c.dtype, stats, B).bind(weights) for _ in range(smax)]
        idx = [torch.from_numpy(b.indices).cuda() for b in batches]
        off = [torch.from_numpy(b.offsets).cuda() for b in batches]
        outs = [torch.empty((B, c.T, c.E), dtype=torch.float32, device="cuda") for _ in range(smax)]
        # batches in flight go to streams of their own: the default stream would order
        # itself against the others
        pool = [torch.cuda.Stream() for _ in range(smax if smax > 1 else 0)]
        ptrs = [(idx[i].data_ptr(), off[i].data_ptr()) for i in range(n_batches)]
        look = [b.n_lookups for b in batches]
        for i in range(warmup):
            plans[0].lookup_ptr(*ptrs[i % n_batches], B, outs[0].data_ptr(), sp)
        torch.cuda.synchronize()
        if verify is not None:
            plans[0].lookup_ptr(*ptrs[0], B, outs[0].data_ptr(), sp)
            torch.cuda.synchronize()
            verify(c, batches[0], outs[0])

        for S in streams:
            side = [stream] if S == 1 else pool[:S]
            others = pool[:S] if S > 1 else []

            ops, sps = [x.data_ptr() for x in outs[:S]], [x.cuda_stream for x in side]

            def launch(i):   # launch i of the pass
                j = i % S
                ip, op = ptrs[i % n_batches]
                plans[j].lookup_ptr(ip, op, B, ops[j], sps[j])

            for x in others:
                x.wait_stream(stream)
            for i in range(warmup if S > 1 else 0):
                launch(i)
            e0 = [torch.cuda.Event(enable_timing=True) for _ in range(n_p99)]
            e1 = [torch.cuda.Event(enable_timing=True) for _ in range(n_p99)]
            for i in range(n_p99):
                e0[i].record(side[i % S])
                launch(i)
                e1[i].record(side[i % S])
            for x in others:
                stream.wait_stream(x)
            torch.cuda.synchronize()
            lat = [e0[i].elapsed_time(e1[i]) * 1e3 for i in range(n_p99)]
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for x in others:
                x.wait_stream(stream)
            for i in range(steps):
                launch(i)
            for x in others:
                stream.wait_stream(x)
            b.record(stream)
            torch.cuda.synchronize()
            us = a.elapsed_time(b) * 1e3 / steps
            nl = sum(look[i % n_batches] for i in range(steps)) / steps
            pt = dict(workload=cfg, batch=B, streams=S, launch_us=us, p99_us=p99(lat), mean_us=sum(lat) / len(lat),
                      lookups_per_s=nl / (us * 1e-6), queries_per_s=B / (us * 1e-6),
                      useful_gbps=nl * c.row_bytes / (us * 1e-6) / 1e9)
            log(f"workload {cfg} batch {B}, {S} in flight: {us:.1f} us per batch, P99 {pt['p99_us']:.1f} us, "
                f"{pt['lookups_per_s']:.3g} lookups/s")
            out_pts.append(pt)
        for x in plans:
            assert x.check_errors() == 0
            x.close()
        del idx, off, outs, batches, plans, pool
    c.batch = full
    del weights
    torch.cuda.empty_cache()
    front = {id(p) for p in pareto_front(out_pts)}
    for p in out_pts:
        p["pareto"] = id(p) in front
    return out_pts


def to_markdown(points: List[Dict], command: str) -> str:
    lines = ["# Batch-size sweep: throughput against P99 (re-planned per batch size)", "",
             "Command:", "", "```", command, "```", "",
             "`us per batch`: event pair around back-to-back launches / launches (with batches in flight, "
             "dealt to that many streams); P99: event pair per launch on its stream (nearest rank); "
             "* = on the Pareto front of its workload.", "",
             "| workload | batch | in flight | us per batch | P99 us | lookups/s | queries/s | useful GB/s | front |",
             "|---|---|---|---|---|---|---|---|---|"]
    for p in points:
        lines.append(f"| {p['workload']} | {p['batch']} | {p.get('streams', 1)} | {p['launch_us']:.1f} | "
                     f"{p['p99_us']:.1f} | {p['lookups_per_s']:.3g} | {p['queries_per_s']:.3g} | "
                     f"{p['useful_gbps']:.0f} | {'*' if p['pareto'] else ''} |")
    return "\n".join(lines) + "\n"


def main(argv=None) -> int:
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--configs", type=int, nargs="+", default=[2, 3, 4])
    ap.add_argument("--fractions", type=float, nargs="+", default=[1 / 16, 1 / 8, 1 / 4, 1 / 2, 1.0])
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--p99", type=int, default=500)
    ap.add_argument("--out", default=None, help="markdown summary")
    ap.add_argument("--json", default=None)
    ap.add_argument("--batches", type=int, default=0, help="distinct resident batches (default 8, 4 for workload 5)")
    ap.add_argument("--streams", type=int, nargs="+", default=[1], choices=[1, 2, 3, 4],
                    help="batches in flight, one point each per batch size (a plan and a stream each)")
    a = ap.parse_args(argv)
    pts = []
    for cfg in a.configs:
        pts += sweep(cfg, a.fractions, a.steps, n_p99=a.p99, n_batches=a.batches,
                     log=lambda m: print(m, file=sys.stderr, flush=True), streams=sorted(set(a.streams)))
    cmd = "python -m paper_2507_01676_amd.pareto " + " ".join(argv if argv is not None else sys.argv[1:])
    md = to_markdown(pts, cmd)
    print(md)
    if a.out:
        with open(a.out, "w") as f:
            f.write(md)
    if a.json:
        with open(a.json, "w") as f:
            json.dump(pts, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())

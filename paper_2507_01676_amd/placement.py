"""Symmetric against asymmetric placement of gather tables, on many-table workloads.

The paper maps tables onto cores asymmetrically (whole tables, or row chunks, on
the least-loaded core, Sec. III-B) instead of splitting every table over every core
(symmetric partitioning, Sec. III-A).  With few tables the planner here splits
every gather table over all workers; past ``sym_max`` gather tables it does so only
for tables whose slices would hold at least 64 lookups, and places the rest by cost.  This study times both plans on synthetic workloads of T tables with
log-uniform row counts and Zipf-distributed ids, s lookups per bag:

    python -m paper_2507_01676_amd.placement --tables 26 64 100 300 1000
    python -m paper_2507_01676_amd.placement --tables 100 300 --batch 4096 --pooling 4
"""
from __future__ import annotations

import sys
from typing import Dict, List, Sequence


def study(tables: Sequence[int] = (26, 100, 1000), batch: int = 1024, E: int = 64, launches: int = 100,
          log=print, pooling: int = 1) -> List[Dict]:
    import numpy as np
    import torch
    import workloads as W
    from . import EmbxError, Plan, fill_table
    out = []
    for T in tables:
        g = np.random.default_rng(T)
        rows = [int(x) for x in np.exp(g.uniform(np.log(100), np.log(1e6), size=T))]
        tabs = [W.TableSpec(m, "fixed", float(pooling), pooling, pooling, "zipf", 1.05) for m in rows]
        c = W.Config(600 + T % 1000, f"{T} tables", E, "f32", -0.05, 0.05, batch, tabs)
        c.value_seeds = [W.value_seed(c.cfg_id, t) for t in range(c.T)]
        bt = W.gen_batch(c, 0)
        stats = W.history_stats(c)
        ws = []
        for t, m in enumerate(c.rows):
            w = torch.empty((m, c.E), device="cuda")
            fill_table(w, t, c.value_seeds[t], c.lo, c.hi)
            ws.append(w)
        idx = torch.from_numpy(bt.indices).cuda()
        off = torch.from_numpy(bt.offsets).cuda()
        res = torch.empty((c.batch, c.T, c.E), device="cuda")
        for name, sym_max in (("default", 0), ("by cost", -1), ("all symmetric", 1 << 30)):
            try:
                plan = Plan(c.rows, c.E, c.dtype, stats, c.batch, sym_max=sym_max).bind(ws)
            except EmbxError as e:
                log(f"{T} tables, {name}: refused ({e})")
                out.append(dict(tables=T, placement=name, refused=str(e)))
                continue
            for _ in range(30):
                plan.lookup(idx, off, c.batch, res)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            # raw-pointer launches, as bench.py times them (no per-call argument checks)
            ip, op, rp, sp = idx.data_ptr(), off.data_ptr(), res.data_ptr(), torch.cuda.current_stream().cuda_stream
            a.record()
            for _ in range(launches):
                plan.lookup_ptr(ip, op, c.batch, rp, sp)
            b.record()
            torch.cuda.synchronize()
            info = plan.info()
            ks = [int(ln.split()[8]) for ln in plan.serialize().splitlines() if ln.startswith("item ")]
            us = a.elapsed_time(b) * 1e3 / launches
            r = dict(tables=T, batch=batch, pooling=pooling, share=batch * pooling / 256,
                     placement=name, slices=info["num_items"], whole_tables=ks.count(1),
                     lif_milli=info["lif_milli"], launch_us=us, lookups_per_s=bt.n_lookups / (us * 1e-6))
            log(f"{T} tables, {name}: {r['slices']} slices ({r['whole_tables']} whole tables), "
                f"LIF {r['lif_milli'] / 1000:.3f}, {us:.1f} us per batch")
            out.append(r)
            plan.close()
        del ws
        torch.cuda.empty_cache()
    return out


def main(argv=None) -> int:
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--tables", type=int, nargs="+", default=[26, 64, 100, 300, 1000])
    ap.add_argument("--batch", type=int, nargs="+", default=[1024])
    ap.add_argument("--pooling", type=int, nargs="+", default=[1])
    a = ap.parse_args(argv)
    rs = []
    for bsz in a.batch:
        for s in a.pooling:
            rs += study(a.tables, bsz, log=lambda m: print(m, file=sys.stderr, flush=True), pooling=s)
    print("| tables | batch | pooling | lookups per table per worker | placement | slices | whole tables | LIF | "
          "us per batch | lookups/s |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    for r in rs:
        if "refused" in r:
            print(f"| {r['tables']} | | | | {r['placement']} | refused | | | | |")
        else:
            print(f"| {r['tables']} | {r['batch']} | {r['pooling']} | {r['share']:.0f} | {r['placement']} | "
                  f"{r['slices']} | {r['whole_tables']} | {r['lif_milli'] / 1000:.3f} | {r['launch_us']:.1f} | "
                  f"{r['lookups_per_s']:.3g} |")
    return 0


if __name__ == "__main__":
    sys.exit(main())

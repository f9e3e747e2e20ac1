"""Per-strategy timing on a grid of table sizes and pooling factors.

The paper picks one data flow per table from a cost model (Sec. III-A, Eq. (2)) and
compares its flows across table sizes and sequence lengths.  This study times every
strategy, forced in turn, on T identical tables of m rows each (Zipf-skewed ids, a
fixed pooling factor s), for a grid of m and s, and reports which one is fastest on
this device and which one the planner picks on its own:

    python -m paper_2507_01676_amd.strategies --rows 512 4096 32768 262144 --pooling 1 8 64 256
"""
from __future__ import annotations

import sys
from typing import Dict, List, Sequence

NAMES = {"auto": -1, "lds": 0, "hot": 1, "dedup": 2, "gather": 3, "stream": 4}


def study(rows: Sequence[int], pooling: Sequence[int], T: int = 8, batch: int = 4096, E: int = 64,
          launches: int = 30, log=print) -> List[Dict]:
    import torch
    import workloads as W
    from . import EmbxError, Plan, fill_table
    out = []
    for m in rows:
        tabs0 = [W.TableSpec(m, "fixed", 1.0, 1, 1, "zipf", 1.05) for _ in range(T)]
        c0 = W.Config(700, f"{T} x {m} rows", E, "f32", -0.05, 0.05, batch, tabs0)
        c0.value_seeds = [W.value_seed(700, t) for t in range(T)]
        ws = []
        for t in range(T):
            w = torch.empty((m, E), device="cuda")
            fill_table(w, t, c0.value_seeds[t], c0.lo, c0.hi)
            ws.append(w)
        for s in pooling:
            tabs = [W.TableSpec(m, "fixed", float(s), s, s, "zipf", 1.05) for _ in range(T)]
            c = W.Config(700 + s, f"{T} x {m} rows, s={s}", E, "f32", -0.05, 0.05, batch, tabs)
            c.value_seeds = c0.value_seeds
            bt = W.gen_batch(c, 0)
            stats = W.history_stats(c)
            idx = torch.from_numpy(bt.indices).cuda()
            off = torch.from_numpy(bt.offsets).cuda()
            res = torch.empty((batch, T, E), device="cuda")
            row = dict(rows=m, pooling=s, table_bytes=m * E * 4, lookups=int(bt.n_lookups))
            for name, code in NAMES.items():
                opts = {} if code < 0 else {"force": [code] * T}
                try:
                    plan = Plan(c.rows, E, "f32", stats, batch, **opts).bind(ws)
                except EmbxError as e:
                    row[name] = None
                    log(f"m={m} s={s} {name}: not applicable ({e})")
                    continue
                for _ in range(5):
                    plan.lookup(idx, off, batch, res)
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                # raw-pointer launches, as bench.py times them (no per-call argument checks)
                ip, op, rp, sp = idx.data_ptr(), off.data_ptr(), res.data_ptr(), torch.cuda.current_stream().cuda_stream
                a.record()
                for _ in range(launches):
                    plan.lookup_ptr(ip, op, batch, rp, sp)
                b.record()
                torch.cuda.synchronize()
                us = a.elapsed_time(b) * 1e3 / launches
                row[name] = us
                if code < 0:
                    row["auto_pick"] = "+".join(k for k, v in plan.info()["n_strategy"].items() if v)
                plan.close()
                log(f"m={m} s={s} {name}: {us:.1f} us")
            forced = {k: v for k, v in row.items() if k in NAMES and k != "auto" and v is not None}
            row["fastest"] = min(forced, key=forced.get)
            out.append(row)
            del idx, off, res
        del ws
        torch.cuda.empty_cache()
    return out


def to_markdown(rs: List[Dict], command: str) -> str:
    cols = [k for k in NAMES if k != "auto"]
    lines = ["# Per-strategy launch time on a grid of table sizes and pooling factors", "",
             "Command:", "", "```", command, "```", "",
             "8 identical fp32 tables (E = 64, 256-byte rows), Zipf(1.05) ids, a fixed pooling factor, "
             "batch 4096; each strategy forced on every table in turn (the planner still chooses splits "
             "and placement), µs per launch (event pair around 30 launches). `auto` is the planner's "
             "own choice; `-` = not applicable (HOT needs hot rows).", "",
             "| rows (table MB) | pooling | " + " | ".join(cols) + " | fastest | auto | auto picks |",
             "|---|---|" + "---|" * (len(cols) + 3)]
    for r in rs:
        cells = [("-" if r.get(k) is None else f"{r[k]:.1f}") for k in cols]
        lines.append(f"| {r['rows']} ({r['table_bytes'] / 2**20:.2f}) | {r['pooling']} | " + " | ".join(cells) +
                     f" | {r['fastest']} | {r['auto']:.1f} | {r.get('auto_pick', '')} |")
    return "\n".join(lines) + "\n"


def main(argv=None) -> int:
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--rows", type=int, nargs="+", default=[512, 4096, 32768, 262144])
    ap.add_argument("--pooling", type=int, nargs="+", default=[1, 8, 64, 256])
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    rs = study(a.rows, a.pooling, log=lambda m: print(m, file=sys.stderr, flush=True))
    cmd = "python -m paper_2507_01676_amd.strategies " + " ".join(argv if argv is not None else sys.argv[1:])
    md = to_markdown(rs, cmd)
    print(md)
    if a.out:
        with open(a.out, "w") as f:
            f.write(md)
    return 0


if __name__ == "__main__":
    sys.exit(main())

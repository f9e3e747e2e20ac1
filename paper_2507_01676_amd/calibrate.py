"""Calibration of the planner's cost model on the device it runs on (Eq. (2)).

The paper prices each table-to-core assignment with a cost linear in the
table's parameters and fits the coefficients by ordinary least squares on
measured runs (Sec. III-A).  Here the measured runs are lookups on synthetic
workloads with every table forced to one strategy and the per-slice timers of
``emb_plan_set_trace`` switched on; the coefficients are the planner's beta
vector (picoseconds), in the layout of ``include/embx.h``:

    G0 G1 L0 L1 S I H0 P D0 D1 SH

and each strategy's cost of one slice with lambda lookups is

    GATHER   G0 + G1 lambda
    LDS      L0 + S mu R + L1 lambda                 (mu rows staged)
    chunk    L0 + S mu R + I lambda + L1 lambda / c  (one of c row chunks)
    HOT      H0 + SH C R + lambda (P + h L1 + (1 - h) G1)   (C hot rows staged)
    DEDUP    D0 + D1 lambda + G1 u lambda

Shared coefficients are fitted once and then held fixed: GATHER first (G0,
G1 from each worker's gather-phase time against its gather slices and
lookups), LDS next (L0, S, L1 from whole-table slices, then I from what they
leave of the row-chunk slices' times, so that I also carries the chunk
combine), then HOT (H0, SH, P) and DEDUP (D0, D1) on what their costs leave
after the shared terms.  HOT has its own per-byte staging term: its rows are
fetched by id, one row per sub-wavefront, where an LDS slice copies a block, and
the paper's coefficients differ per strategy in the same way (Sec. III-A).
Every fit is ``numpy.linalg.lstsq``, reweighted once so that residuals count
relative to each sample's predicted time, and constrained to non-negative coefficients
(an active-set NNLS) when the unconstrained solution has a negative one: the
coefficients are times, and the planner refuses negative ones.

``fit_beta`` is plain host arithmetic; ``collect`` runs lookups on the current
device and needs the extension.  ``python -m paper_2507_01676_amd.calibrate``
runs both on the synthetic workloads and prints the fitted vector; with
``--report`` it re-plans the workloads with that vector and sets each plan's
predicted makespan beside the measured one, and with ``--loop N`` it closes the
loop: plan, run the plan with its timers on, add the plan's own timings to the
samples, fit again and re-plan, for up to N rounds or until the plans stop
changing (``loop``).
"""
from __future__ import annotations

import json
import sys
from dataclasses import dataclass, field
from types import SimpleNamespace
from typing import Dict, List, Optional, Sequence

import numpy as np

G0, G1, L0, L1, S, I, H0, P, D0, D1, SH = range(11)
NBETA = 11
BETA_NAMES = ["G0", "G1", "L0", "L1", "S", "I", "H0", "P", "D0", "D1", "SH"]
LDS, HOT, DEDUP, GATHER = 0, 1, 2, 3
TICK_PS = 10_000.0          # the kernel timers count a 100 MHz clock


@dataclass
class SliceSample:
    """One staged slice (LDS, HOT or DEDUP) and its measured time."""
    strat: int
    lam: float              # lookups of the slice in the measured batch
    mu: float = 0.0         # LDS: rows staged;  HOT: hot rows staged (C)
    R: int = 0              # row bytes
    c: int = 1              # LDS: number of row chunks of the table
    h: float = 0.0          # HOT: fraction of the table's lookups on the staged rows
    u: float = 1.0          # DEDUP: distinct rows per lookup
    ps: float = 0.0         # measured time


@dataclass
class WorkerSample:
    """One worker's gather phase: its gather slices, their lookups and its time."""
    n_slices: int
    lam: float
    ps: float


@dataclass
class Samples:
    slices: List[SliceSample] = field(default_factory=list)
    workers: List[WorkerSample] = field(default_factory=list)


def _lstsq(A: np.ndarray, y: np.ndarray, offset: Optional[np.ndarray] = None) -> np.ndarray:
    """Least squares with non-negative coefficients (the planner refuses negative ones):
    the unconstrained solution when it is non-negative, else the best fit over the
    columns that stay free (scipy's active-set NNLS), columns scaled to unit norm.

    With ``offset`` (the part of each sample's time already accounted for, so that the
    sample's time is A x + offset) the fit is reweighted once: residuals are divided by
    each sample's time as predicted by a first plain fit (at least 1 us).  Timing noise
    grows with the time (contention), so unweighted, the long slices' scatter sets the
    intercept -- it then came out negative for strategies whose short slices are
    nearly all fixed cost.  The predicted rather than the measured time keeps the
    weights free of the noise they correct for."""
    if offset is not None:
        x0, *_ = np.linalg.lstsq(A, y, rcond=None)
        w = 1.0 / np.maximum(A @ x0 + np.asarray(offset, dtype=np.float64), 1e6)
        A = A * w[:, None]
        y = y * w
    x, *_ = np.linalg.lstsq(A, y, rcond=None)
    if np.all(x >= 0.0):
        return x
    from scipy.optimize import nnls
    norm = np.linalg.norm(A, axis=0)
    norm[norm == 0.0] = 1.0
    z, _ = nnls(A / norm, y)
    return z / norm


def fit_beta(s: Samples, base: Optional[Sequence[float]] = None) -> List[float]:
    """Least-squares fit of the beta vector, residuals relative to each sample's predicted
    time (one reweighting step); coefficients with no samples keep ``base``'s value."""
    b = list(base) if base is not None else [0.0] * NBETA
    if s.workers:
        A = np.array([[w.n_slices, w.lam] for w in s.workers], dtype=np.float64)
        y = np.array([w.ps for w in s.workers], dtype=np.float64)
        b[G0], b[G1] = (float(v) for v in _lstsq(A, y, np.zeros(len(y))))
    whole = [x for x in s.slices if x.strat == LDS and x.c == 1]
    if whole:
        A = np.array([[1.0, x.mu * x.R, x.lam] for x in whole])
        y = np.array([x.ps for x in whole])
        b[L0], b[S], b[L1] = (float(v) for v in _lstsq(A, y, np.zeros(len(y))))
    chunks = [x for x in s.slices if x.strat == LDS and x.c > 1]
    if chunks:
        # I on what the whole-table terms leave; it absorbs the chunk combine as well
        A = np.array([[x.lam] for x in chunks])
        off = np.array([b[L0] + b[S] * x.mu * x.R + b[L1] * x.lam / x.c for x in chunks])
        y = np.array([x.ps for x in chunks]) - off
        b[I] = float(_lstsq(A, y, off)[0])
    hot = [x for x in s.slices if x.strat == HOT]
    if hot:
        A = np.array([[1.0, x.mu * x.R, x.lam] for x in hot])
        off = np.array([x.lam * (x.h * b[L1] + (1.0 - x.h) * b[G1]) for x in hot])
        y = np.array([x.ps for x in hot]) - off
        b[H0], b[SH], b[P] = (float(v) for v in _lstsq(A, y, off))
    dd = [x for x in s.slices if x.strat == DEDUP]
    if dd:
        A = np.array([[1.0, x.lam] for x in dd])
        off = np.array([b[G1] * x.u * x.lam for x in dd])
        y = np.array([x.ps for x in dd]) - off
        b[D0], b[D1] = (float(v) for v in _lstsq(A, y, off))
    return b


def predict(b: Sequence[float], x) -> float:
    """The cost model's time for one sample (the same formulas the fit inverts)."""
    if isinstance(x, WorkerSample):
        return b[G0] * x.n_slices + b[G1] * x.lam
    if x.strat == LDS:
        extra = b[I] * x.lam if x.c > 1 else 0.0
        return b[L0] + b[S] * x.mu * x.R + extra + b[L1] * x.lam / x.c
    if x.strat == HOT:
        return b[H0] + b[SH] * x.mu * x.R + x.lam * (b[P] + x.h * b[L1] + (1.0 - x.h) * b[G1])
    if x.strat == DEDUP:
        return b[D0] + b[D1] * x.lam + b[G1] * x.u * x.lam
    raise ValueError(x.strat)


# ---------------------------------------------------------------- measurement

def _plan_items(text: str):
    out = []
    for ln in text.splitlines():
        if ln.startswith("item "):
            f = ln.split()
            out.append(dict(wg=int(f[1]), t=int(f[2]), strat=int(f[3]), chunk=int(f[4]), nchunks=int(f[5]),
                            r0=int(f[6]), r1=int(f[7]), k=int(f[8]), j=int(f[9]), C=int(f[10])))
    return out


def traced_launch(plan, indices, offsets, batch: int, out, warm: int = 3) -> np.ndarray:
    """``warm`` untimed launches, then one with the kernel timers on; returns the timers."""
    import torch
    for _ in range(warm):
        plan.lookup(indices, offsets, batch, out)
    n = plan.trace_size()
    buf = torch.zeros(n, dtype=torch.int64, device=indices.device)
    plan.set_trace(buf)
    plan.lookup(indices, offsets, batch, out)
    torch.cuda.synchronize()
    plan.set_trace(None)
    return buf.cpu().numpy()


def samples_of(plan, tr: np.ndarray, batch: int, host_offsets: np.ndarray, stats, R: int) -> Samples:
    """The samples one traced launch gives: each staged slice's time, and each worker's
    gather phase (its gather slices run merged).  ``host_offsets`` is the batch's CSR
    offsets on the host (to count each slice's lookups); ``stats`` the per-table
    statistics the plan was made from."""
    info = plan.info()
    K = info["num_workers"]
    per = 2 + 1024 // 64
    tw = tr[:K * per].reshape(K, per)
    ti = tr[K * per:].reshape(-1, 2)
    items = _plan_items(plan.serialize())
    s = Samples()
    gcount = np.zeros(K, dtype=np.int64)
    glam = np.zeros(K, dtype=np.float64)
    for i, it in enumerate(items):
        bs, be = it["j"] * batch // it["k"], (it["j"] + 1) * batch // it["k"]
        t = it["t"]
        lam = float(host_offsets[t * batch + be] - host_offsets[t * batch + bs])
        if it["strat"] == GATHER:
            gcount[it["wg"]] += 1
            glam[it["wg"]] += lam
            continue
        if be <= bs:
            continue
        ps = float(ti[i, 1] - ti[i, 0]) * TICK_PS
        st = stats[t]
        hot_f = getattr(st, "hot_freq", None)
        h = float(np.sum(hot_f[:it["C"]])) if (hot_f is not None and it["C"] > 0) else 0.0
        u = float(getattr(st, "unique_frac", 1.0))
        mu = float(it["r1"] - it["r0"]) if it["strat"] == LDS else float(it["C"])
        s.slices.append(SliceSample(it["strat"], lam, mu, R, it["nchunks"], h, u if 0 < u <= 1 else 1.0, ps))
    gat = (tw[:, 2:].max(axis=1) - tw[:, 1]).astype(np.float64) * TICK_PS
    for w in range(K):
        if gcount[w]:
            s.workers.append(WorkerSample(int(gcount[w]), float(glam[w]), float(gat[w])))
    return s


def worker_gather_samples(plan, tr: np.ndarray, batch: int, host_offsets: np.ndarray, T: int):
    """From one traced launch: for each worker with gather slices, its gather-phase time
    (ps), its number of gather slices and its lookups from each table at this batch
    (rows of a K' x T matrix)."""
    info = plan.info()
    K = info["num_workers"]
    per = 2 + 1024 // 64
    tw = tr[:K * per].reshape(K, per)
    lam = np.zeros((K, T), dtype=np.float64)
    n = np.zeros(K, dtype=np.int64)
    for it in _plan_items(plan.serialize()):
        if it["strat"] != GATHER:
            continue
        bs, be = it["j"] * batch // it["k"], (it["j"] + 1) * batch // it["k"]
        t = it["t"]
        lam[it["wg"], t] += float(host_offsets[t * batch + be] - host_offsets[t * batch + bs])
        n[it["wg"]] += 1
    gat = (tw[:, 2:].max(axis=1) - tw[:, 1]).astype(np.float64) * TICK_PS
    keep = n > 0
    return gat[keep], n[keep], lam[keep]


def fit_table_lookup_costs(ps: np.ndarray, n_slices: np.ndarray, lam: np.ndarray, g0: float) -> List[float]:
    """Each table's cost of one lookup served from memory (ps), from workers' gather
    phases: time = c + G0 x slices + sum over tables of G1_t x lookups_t, with one shared
    c (the latency chain every worker pays once: launch skew, run header, first loads)
    and G0 from the cost vector, fitted with non-negative coefficients and residuals
    relative to each worker's predicted time.  Eq. (2) prices a lookup alike in every
    table; on this device one that misses the caches costs a CU several times one that
    hits, and Sec. III-A fits the coefficients per configuration.  A table with no
    lookups in the samples gets 0 (the planner then uses the vector's G1)."""
    ps = np.asarray(ps, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    used = np.flatnonzero(lam.sum(axis=0) > 0)
    if used.size == 0 or len(ps) <= used.size:   # nothing to fit, or fewer workers than unknowns
        return [0.0] * lam.shape[1]
    A = np.column_stack([np.ones(len(ps)), lam[:, used]])
    y = ps - g0 * np.asarray(n_slices, dtype=np.float64)
    x = _lstsq(A, y, np.zeros(len(y)))
    out = [0.0] * lam.shape[1]
    for i, t in enumerate(used):
        out[int(t)] = float(x[1 + i])
    return out


def measure(plan, indices, offsets, batch: int, out, host_offsets: np.ndarray, stats, R: int,
            warm: int = 3) -> Samples:
    """Runs one traced launch of ``plan`` and turns its timers into samples."""
    return samples_of(plan, traced_launch(plan, indices, offsets, batch, out, warm), batch, host_offsets, stats, R)


def collect(configs: Sequence[int] = (2, 3, 4), strategies: Sequence[str] = ("gather", "lds", "hot", "dedup"),
            lds_max_bytes: int = 32 << 20, log=print, dists: Sequence[str] = ("config",),
            hot_sizes: Sequence[int] = (1, 8, 64, 512)) -> Samples:
    """Measures the synthetic workloads with each strategy forced on every table, under
    each query distribution of ``dists`` (the workload's own, 'uniform', 'fixed').

    HOT runs once per size in ``hot_sizes``: each table's statistics list only its C
    hottest rows, and the plan is made with a vector that prices staging and LDS reads at
    nothing (SH = L1 = 0), so that every listed row is staged and the samples span C."""
    import dataclasses

    import torch
    import workloads as W
    from . import Plan, default_beta, fill_table
    code = {"lds": LDS, "hot": HOT, "dedup": DEDUP, "gather": GATHER}
    stage_all = list(default_beta(256))
    stage_all[SH] = 0.0
    stage_all[L1] = 0.0
    allS = Samples()
    for cfg, dist in [(cfg, d) for cfg in configs for d in dists]:
        c = W.with_distribution(W.make_config(cfg), dist)
        bt = W.gen_batch(c, 0)
        stats = W.history_stats(c)
        dt = torch.float16 if c.dtype == "f16" else torch.float32
        ws = []
        for t, m in enumerate(c.rows):
            w = torch.empty((m, c.E), dtype=dt, device="cuda")
            fill_table(w, t, c.value_seeds[t], c.lo, c.hi)
            ws.append(w)
        idx = torch.from_numpy(bt.indices).cuda()
        off = torch.from_numpy(bt.offsets).cuda()
        out = torch.empty((c.batch, c.T, c.E), device="cuda")
        runs = []
        for name in strategies:
            force = [code[name]] * c.T
            if name == "lds":
                # LDS (row chunks) only on the tables of at most lds_max_bytes; the rest
                # gather, and those gather workers are not samples (their time follows
                # the staged slices on the same workers)
                force = [LDS if m * c.row_bytes <= lds_max_bytes else GATHER for m in c.rows]
            if name == "hot":
                for C in hot_sizes:
                    st_c = [dataclasses.replace(x, hot_rows=x.hot_rows[:C], hot_freq=x.hot_freq[:C]) for x in stats]
                    runs.append((f"hot C<={C}", force, st_c, stage_all))
            else:
                runs.append((name, force, stats, None))
        for name, force, st_r, plan_beta in runs:
            extra = {} if plan_beta is None else {"beta": plan_beta}
            plan = Plan(c.rows, c.E, c.dtype, st_r, c.batch, force=force, **extra).bind(ws)
            s = measure(plan, idx, off, c.batch, out, bt.offsets, st_r, c.row_bytes)
            plan.close()
            if name == "lds":
                s.workers = []
            log(f"workload {cfg} ({dist} queries) {name}: {len(s.slices)} slices, {len(s.workers)} gather workers")
            allS.slices += s.slices
            allS.workers += s.workers
        del ws
        torch.cuda.empty_cache()
    return allS


def collect_staging(sizes: Sequence[int] = (16, 64, 128, 256, 512), E: int = 64, K: int = 256, B: int = 256,
                    log=print) -> Samples:
    """Whole-table LDS slices that differ only in the bytes they stage: K tables of m rows
    (E fp32), one slice per worker (no batch splits, K workers), B bags of one lookup each,
    for each m in ``sizes`` -- the workloads' few small tables alone leave the per-byte
    staging term S undetermined."""
    import torch
    from . import Plan
    s_all = Samples()
    g = np.random.default_rng(7)
    for m in sizes:
        ws = [torch.empty((m, E), device="cuda").uniform_(-1.0, 1.0) for _ in range(K)]
        st = [dict(mean_pooling=1.0, max_pooling=1) for _ in range(K)]
        plan = Plan([m] * K, E, "f32", st, B, force=[LDS] * K, num_workers=K, no_replication=True).bind(ws)
        ids = g.integers(0, m, size=K * B).astype(np.int64)
        off = np.arange(K * B + 1, dtype=np.int64)
        out = torch.empty((B, K, E), device="cuda")
        s = measure(plan, torch.from_numpy(ids).cuda(), torch.from_numpy(off).cuda(), B, out, off,
                    [SimpleNamespace(unique_frac=1.0, hot_freq=None)] * K, E * 4)
        plan.close()
        log(f"staging sweep, {m} rows a table: {len(s.slices)} slices")
        s_all.slices += s.slices
        del ws
        torch.cuda.empty_cache()
    return s_all


def report(beta: Sequence[float], configs: Sequence[int] = (1, 2, 3, 4), log=print,
           samples: Optional[Samples] = None) -> List[Dict]:
    """Re-plans each workload with ``beta`` and sets the plan's predicted makespan (the
    most loaded worker, in the cost model's units) beside the measured one: the slowest
    worker's span from the kernel timers and the mean launch time of back-to-back
    launches.  With ``samples``, the traced launch's own slices and workers are added to it."""
    import hashlib

    import torch
    import workloads as W
    from . import Plan, fill_table
    rows_out = []
    for cfg in configs:
        c = W.make_config(cfg)
        bt = W.gen_batch(c, 0)
        stats = W.history_stats(c)
        dt = torch.float16 if c.dtype == "f16" else torch.float32
        ws = []
        for t, m in enumerate(c.rows):
            w = torch.empty((m, c.E), dtype=dt, device="cuda")
            fill_table(w, t, c.value_seeds[t], c.lo, c.hi)
            ws.append(w)
        plan = Plan(c.rows, c.E, c.dtype, stats, c.batch, beta=list(beta)).bind(ws)
        idx = torch.from_numpy(bt.indices).cuda()
        off = torch.from_numpy(bt.offsets).cuda()
        out = torch.empty((c.batch, c.T, c.E), device="cuda")
        for _ in range(5):
            plan.lookup(idx, off, c.batch, out)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        # raw-pointer launches, as bench.py times them (no per-call argument checks)
        ip, op, rp, sp = idx.data_ptr(), off.data_ptr(), out.data_ptr(), torch.cuda.current_stream().cuda_stream
        n_launch = 50 if cfg != 5 else 10
        a.record()
        for _ in range(n_launch):
            plan.lookup_ptr(ip, op, c.batch, rp, sp)
        b.record()
        torch.cuda.synchronize()
        launch_us = a.elapsed_time(b) * 1e3 / n_launch
        tr = traced_launch(plan, idx, off, c.batch, out, warm=0)
        info = plan.info()
        K = info["num_workers"]
        per = 2 + 1024 // 64
        tw = tr[:K * per].reshape(K, per)
        span_us = float((tw[:, 2:].max() - tw[:, 0].min()) * TICK_PS / 1e6)
        # each worker's busy time (start to its last wavefront's end), and the skew of starts
        busy = (tw[:, 2:].max(axis=1) - tw[:, 0]).astype(np.float64) * TICK_PS / 1e6
        skew_us = float((tw[:, 0].max() - tw[:, 0].min()) * TICK_PS / 1e6)
        if samples is not None:
            s = samples_of(plan, tr, c.batch, bt.offsets, stats, c.row_bytes)
            samples.slices += s.slices
            samples.workers += s.workers
        # the plan's structure: every slice's placement and shape, without its cost
        text = "\n".join(" ".join(ln.split()[:-1]) for ln in plan.serialize().splitlines() if ln.startswith("item "))
        r = dict(workload=cfg, strategies=info["n_strategy"], kernel=info["kernel"], lif_milli=info["lif_milli"],
                 predicted_us=info["max_load_ps"] / 1e6, measured_span_us=span_us, launch_us=launch_us,
                 busy_mean_us=float(busy.mean()), busy_max_us=float(busy.max()), start_skew_us=skew_us,
                 plan_sha=hashlib.sha256(text.encode()).hexdigest()[:16])
        log(f"workload {cfg}: plan {r['strategies']} ({r['kernel']}) lif {r['lif_milli']}; predicted makespan "
            f"{r['predicted_us']:.1f} us, measured worker span {span_us:.1f} us (start skew {skew_us:.2f}, busy "
            f"mean {busy.mean():.2f} max {busy.max():.2f}), launch {launch_us:.1f} us")
        rows_out.append(r)
        plan.close()
        del ws
        torch.cuda.empty_cache()
    return rows_out


def loop(beta: Sequence[float], samples: Samples, configs: Sequence[int] = (1, 2, 3, 4), rounds: int = 3,
         base: Optional[Sequence[float]] = None, log=print) -> Dict:
    """The calibration loop closed (Sec. III-A): plan every workload with the current
    coefficients, run each plan with its timers on, add the plan's own slice and worker
    times to the samples, fit again and re-plan; stops after ``rounds`` rounds or as soon
    as a fit leaves every plan as it was.  Returns the final vector and each round's
    predicted and measured makespans."""
    beta = list(beta)
    history = []
    prev = None
    for r in range(rounds):
        rows = report(beta, configs, log=log, samples=samples)
        history.append(dict(round=r, beta=dict(zip(BETA_NAMES, beta)), workloads=rows))
        shas = [x["plan_sha"] for x in rows]
        beta = fit_beta(samples, base)
        log(f"round {r}: refit on {len(samples.slices)} slices and {len(samples.workers)} workers: "
            + " ".join(f"{n}={v:.4g}" for n, v in zip(BETA_NAMES, beta)))
        if shas == prev:
            break
        prev = shas
    return dict(beta=dict(zip(BETA_NAMES, beta)), rounds=history)


def write_samples_csv(s: Samples, path: str, max_rows: int = 250, seed: int = 0) -> None:
    """The samples as CSV (one header line of column names; kind = worker or slice), at
    most ``max_rows`` of each group (gather workers; whole-table LDS; LDS row chunks; HOT;
    DEDUP), picked at random with ``seed`` when there are more."""
    g = np.random.default_rng(seed)

    def pick(xs):
        if len(xs) <= max_rows:
            return list(xs)
        keep = np.sort(g.choice(len(xs), size=max_rows, replace=False))
        return [xs[i] for i in keep]

    with open(path, "w") as f:
        f.write("kind,strat,lam,mu,R,c,h,u,n_slices,ps\n")
        for w in pick(s.workers):
            f.write(f"worker,{GATHER},{w.lam:.8g},0,0,1,0,1,{w.n_slices},{w.ps:.8g}\n")
        groups = [[x for x in s.slices if x.strat == LDS and x.c == 1], [x for x in s.slices if x.strat == LDS and x.c > 1],
                  [x for x in s.slices if x.strat == HOT], [x for x in s.slices if x.strat == DEDUP]]
        for grp in groups:
            for x in pick(grp):
                f.write(f"slice,{x.strat},{x.lam:.8g},{x.mu:.8g},{x.R},{x.c},{x.h:.8g},{x.u:.8g},0,{x.ps:.8g}\n")


def read_samples_csv(path: str) -> Samples:
    s = Samples()
    with open(path) as f:
        head = None
        for ln in f:
            if ln.startswith("#") or not ln.strip():
                continue
            v = ln.strip().split(",")
            if head is None:
                head = v
                continue
            d = dict(zip(head, v))
            if d["kind"] == "worker":
                s.workers.append(WorkerSample(int(d["n_slices"]), float(d["lam"]), float(d["ps"])))
            else:
                s.slices.append(SliceSample(int(d["strat"]), float(d["lam"]), float(d["mu"]), int(d["R"]),
                                            int(d["c"]), float(d["h"]), float(d["u"]), float(d["ps"])))
    return s


def _residuals(b, s: Samples, log):
    for st, nm in ((LDS, "LDS"), (HOT, "HOT"), (DEDUP, "DEDUP")):
        xs = [x for x in s.slices if x.strat == st]
        if xs:
            err = np.array([predict(b, x) - x.ps for x in xs])
            rel = np.abs(err) / np.maximum(np.array([x.ps for x in xs]), 1e6)
            log(f"{nm}: {len(xs)} slices, rms residual {np.sqrt(np.mean(err ** 2)) / 1e6:.2f} us, "
                f"median relative {np.median(rel):.2f}")
    if s.workers:
        err = np.array([predict(b, x) - x.ps for x in s.workers])
        log(f"GATHER: {len(s.workers)} workers, rms residual {np.sqrt(np.mean(err ** 2)) / 1e6:.2f} us")


def main(argv=None) -> int:
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--configs", type=int, nargs="+", default=[2, 3, 4])
    ap.add_argument("--strategies", nargs="+", default=["gather", "lds", "hot", "dedup"])
    ap.add_argument("--dists", nargs="+", default=["config"],
                    help="query distributions to measure under (config, uniform, fixed)")
    ap.add_argument("--hot-sizes", type=int, nargs="+", default=[1, 8, 64, 512],
                    help="hot rows listed per table in the HOT runs (one run per size)")
    ap.add_argument("--base", default=None,
                    help="coefficients kept where no sample fits them: 'builtin' (the library's own), "
                         "or a JSON file of {name: value}")
    ap.add_argument("--samples-in", default=None, help="start from these samples (CSV) instead of measuring")
    ap.add_argument("--samples-csv", default=None, help="write the forced-strategy samples as CSV")
    ap.add_argument("--out", default=None, help="write the samples and the fit as JSON")
    ap.add_argument("--report", type=int, nargs="*", default=None,
                    help="re-plan these workloads with the fitted beta and compare predicted and measured makespans")
    ap.add_argument("--loop", type=int, default=0,
                    help="rounds of plan -> traced run -> refit -> re-plan over the --report workloads")
    a = ap.parse_args(argv)
    log = lambda m: print(m, file=sys.stderr, flush=True)   # noqa: E731
    if a.samples_in:
        s = read_samples_csv(a.samples_in)
    else:
        s = collect(a.configs, a.strategies, log=log, dists=a.dists, hot_sizes=a.hot_sizes)
        if "lds" in a.strategies:
            st = collect_staging(log=log)
            s.slices += st.slices
    if a.samples_csv:
        write_samples_csv(s, a.samples_csv)
    base = None
    if a.base == "builtin":
        from . import default_beta
        base = default_beta(256)
    elif a.base:
        with open(a.base) as f:
            given = json.load(f)
        base = [float(given.get(n, 0.0)) for n in BETA_NAMES]
    b = fit_beta(s, base)
    _residuals(b, s, log)
    print(json.dumps(dict(zip(BETA_NAMES, b))))
    rep = lp = None
    configs = a.report if a.report else (1, 2, 3, 4)
    if a.loop > 0:
        lp = loop(b, s, configs, rounds=a.loop, base=base, log=log)
        print(json.dumps(lp["beta"]))
    elif a.report is not None:
        rep = report(b, configs, log=log)
    if a.out:
        with open(a.out, "w") as f:
            json.dump(dict(beta=dict(zip(BETA_NAMES, b)), report=rep, loop=lp,
                           n_slices=len(s.slices), n_workers=len(s.workers)), f)
    return 0


if __name__ == "__main__":
    sys.exit(main())

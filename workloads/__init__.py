"""Seeded synthetic inputs for the multi-table embedding-bag lookup.

This module only *produces inputs*: table shapes, table values, query batches
(indices + CSR offsets) and the per-table index statistics that the planner
takes.  It holds none of the lookup's arithmetic (no gathering, no pooling, no
cost model), so both the CPU oracle tests and the GPU path can consume it
without sharing any of the method's code.

The paper's workloads (tables extracted from public CTR datasets plus a
proprietary model, Sec. IV-A) are not available; the five synthetic
configurations below stand in for them.  They keep the structure the paper
describes: tables from a few rows to GB scale (Sec. IV-A, Fig. 2), uniform and
skewed query distributions (Sec. IV-A), sum pooling with fixed or variable
sequence length (Sec. II-B, Sec. IV-A).

Randomness
----------
Every stream is ``numpy.random.Generator(PCG64(SeedSequence([MASTER, cfg,
purpose, table, batch_id])))`` so any (table, batch) can be regenerated alone.

Table values are a pure function of (table, row, column) built on the
SplitMix64 finalizer (Steele, Lea, Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014).  The GPU-side table filler implements the same
published generator independently.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

MASTER = 250701676

# purposes of the seeded streams
P_SIZES, P_ALPHA, P_PERM, P_PF, P_INDICES, P_VALUE, P_FIXED = 0, 1, 2, 3, 4, 5, 6

GOLDEN = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
M64 = (1 << 64) - 1

HISTORY_BATCH = 1000          # batch_id of the batch the statistics come from
N_HOT_STATS = 4096            # hot rows reported per table


def rng(cfg: int, purpose: int, t: int = 0, batch_id: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([MASTER, cfg, purpose, t, batch_id]))


# ----------------------------------------------------------------------------
# SplitMix64 value generator
# ----------------------------------------------------------------------------

def splitmix64_mix_scalar(z: int) -> int:
    """SplitMix64 output function on a python int (mod 2**64)."""
    z &= M64
    z = ((z ^ (z >> 30)) * MIX1) & M64
    z = ((z ^ (z >> 27)) * MIX2) & M64
    return z ^ (z >> 31)


def _mix_inplace(z: np.ndarray) -> np.ndarray:
    z ^= z >> np.uint64(30)
    z *= np.uint64(MIX1)
    z ^= z >> np.uint64(27)
    z *= np.uint64(MIX2)
    z ^= z >> np.uint64(31)
    return z


def value_seed(cfg: int, t: int) -> int:
    """Per-table seed of the value generator (a uint64)."""
    return int(rng(cfg, P_VALUE, t).integers(0, 1 << 63, dtype=np.uint64))


# value modes
VAL_UNIFORM = 0     # uniform in [lo, hi)
VAL_INTEGER = 1     # small integers that make every pooled sum exact


def table_rows_at(t: int, rows: np.ndarray, E: int, dtype: str, *, seed: int,
                  lo: float = -0.05, hi: float = 0.05, mode: int = VAL_UNIFORM) -> np.ndarray:
    """Rows ``rows`` (any row ids) of table t as an array [len(rows), E] of ``dtype`` ('f32'|'f16').

    key = (t << 40) | (r << 8) | c;  x = mix(key + seed * GOLDEN mod 2**64)

    VAL_UNIFORM: u = x >> 40 (24 bits); v = fp32(lo + (hi - lo) * ((u + 0.5) * 2**-24))
                 evaluated in binary64 then rounded to nearest-even fp32 (and to fp16
                 for 'f16' tables, again nearest-even).
    VAL_INTEGER: column 0 -> 1; columns 1..3 -> base-2048 digits of r (low first);
                 column 4 -> t + 1; other columns -> x >> 53 (11 bits).  Every value
                 is an integer in [0, 2047], exact in fp16, and any sum of up to
                 8192 of them is exact in fp32.
    """
    assert E <= 256 and t < (1 << 23)
    rr = np.asarray(rows, dtype=np.int64).reshape(-1)
    r = rr.astype(np.uint64)[:, None]
    c = np.arange(E, dtype=np.uint64)[None, :]
    key = (np.uint64(t) << np.uint64(40)) | (r << np.uint64(8)) | c
    key = key + np.uint64((seed * GOLDEN) & M64)
    x = _mix_inplace(key)
    if mode == VAL_UNIFORM:
        u = (x >> np.uint64(40)).astype(np.float64)
        u += 0.5
        u *= 2.0 ** -24
        u *= (hi - lo)
        u += lo
        v = u.astype(np.float32)
    elif mode == VAL_INTEGER:
        v = (x >> np.uint64(53)).astype(np.float32)
        v[:, 0] = 1.0
        if E > 1:
            v[:, 1] = (rr & 2047).astype(np.float32)
        if E > 2:
            v[:, 2] = ((rr >> 11) & 2047).astype(np.float32)
        if E > 3:
            v[:, 3] = ((rr >> 22) & 2047).astype(np.float32)
        if E > 4:
            v[:, 4] = float(t + 1)
    else:
        raise ValueError(mode)
    if dtype == "f16":
        return v.astype(np.float16)
    assert dtype == "f32"
    return v


def table_rows_block(t: int, r0: int, r1: int, E: int, dtype: str, *, seed: int,
                     lo: float = -0.05, hi: float = 0.05, mode: int = VAL_UNIFORM) -> np.ndarray:
    """Rows [r0, r1) of table t (see ``table_rows_at``)."""
    assert 0 <= r0 <= r1
    return table_rows_at(t, np.arange(r0, r1, dtype=np.int64), E, dtype, seed=seed, lo=lo, hi=hi, mode=mode)


def materialize_table(t: int, rows: int, E: int, dtype: str, *, seed: int, lo: float = -0.05,
                      hi: float = 0.05, mode: int = VAL_UNIFORM, threads: Optional[int] = None) -> np.ndarray:
    """Whole table t as a host array (chunked and threaded; numpy releases the GIL)."""
    out = np.empty((rows, E), dtype=np.float16 if dtype == "f16" else np.float32)
    step = max(1, (1 << 18) // max(E, 1))
    blocks = [(s, min(rows, s + step)) for s in range(0, rows, step)]

    def work(b):
        s, e = b
        out[s:e] = table_rows_block(t, s, e, E, dtype, seed=seed, lo=lo, hi=hi, mode=mode)

    nthr = threads or min(16, os.cpu_count() or 1)
    if len(blocks) == 1 or nthr == 1:
        for b in blocks:
            work(b)
    else:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(work, blocks))
    return out


# ----------------------------------------------------------------------------
# Configurations
# ----------------------------------------------------------------------------

@dataclass
class TableSpec:
    rows: int
    pf_kind: str            # 'fixed' or 'poisson'
    pf_value: float         # fixed PF, or Poisson mean
    pf_lo: int              # clip bounds (poisson) / both = value (fixed)
    pf_hi: int
    dist: str               # 'uniform', 'zipf', or 'fixed' (every lookup on one row)
    alpha: float = 0.0


@dataclass
class Config:
    cfg_id: int
    name: str
    E: int
    dtype: str              # 'f32' | 'f16'
    lo: float
    hi: float
    batch: int
    tables: List[TableSpec]
    note: str = ""
    value_seeds: List[int] = field(default_factory=list)

    @property
    def T(self) -> int:
        return len(self.tables)

    @property
    def rows(self) -> List[int]:
        return [tb.rows for tb in self.tables]

    @property
    def row_bytes(self) -> int:
        return self.E * (2 if self.dtype == "f16" else 4)

    def max_pooling(self, t: int) -> int:
        return self.tables[t].pf_hi


DISTRIBUTIONS = ("config", "uniform", "fixed")


def with_distribution(c: Config, dist: str) -> Config:
    """``c`` with every table's query distribution replaced: 'uniform' (ids uniform over
    the table's rows) or 'fixed' (every lookup of a table on one row), the
    distributions besides the skewed one that the paper runs its workloads under
    (Sec. IV-A).  Shapes, pooling factors and values are unchanged; 'config' returns
    ``c`` itself."""
    if dist == "config":
        return c
    if dist not in DISTRIBUTIONS:
        raise ValueError(f"unknown query distribution {dist!r}")
    tabs = [TableSpec(tb.rows, tb.pf_kind, tb.pf_value, tb.pf_lo, tb.pf_hi, dist, tb.alpha) for tb in c.tables]
    return Config(c.cfg_id, f"{c.name}; {dist} queries", c.E, c.dtype, c.lo, c.hi, c.batch, tabs, c.note,
                  list(c.value_seeds))


def cfg2_sizes() -> List[int]:
    """26 row counts geometrically spaced from 10 to 4,000,000."""
    return [int(round(10.0 * (4.0e5 ** (t / 25.0)))) for t in range(26)]


def make_config(i: int) -> Config:
    """The five synthetic workloads, 1-based ``i``."""
    if i == 1:
        tabs = [TableSpec(m, "fixed", 1, 1, 1, "uniform") for m in (100, 1000, 10000, 100000)]
        c = Config(1, "4 tables {1e2..1e5} rows, E32 fp32, B128, PF1, uniform", 32, "f32", -1.0, 1.0, 128, tabs)
    elif i == 2:
        tabs = [TableSpec(m, "fixed", 1, 1, 1, "zipf", 1.05) for m in cfg2_sizes()]
        c = Config(2, "26 tables 10..4M rows, E64 fp32, B2048, PF1, Zipf 1.05", 64, "f32", -0.05, 0.05, 2048, tabs)
    elif i == 3:
        al = rng(3, P_ALPHA).uniform(0.8, 1.2, size=26)
        tabs = [TableSpec(m, "poisson", 8.0, 1, 20, "zipf", float(a)) for m, a in zip(cfg2_sizes(), al)]
        c = Config(3, "26 tables 10..4M rows, E128 fp16, B16384, PF Poisson(8) in [1,20], Zipf U[0.8,1.2]",
                   128, "f16", -0.05, 0.05, 16384, tabs)
    elif i == 4:
        ls = rng(4, P_SIZES).uniform(math.log(1e3), math.log(1e6), size=25)
        tabs = [TableSpec(10_000_000, "fixed", 50, 50, 50, "zipf", 1.5)]
        tabs += [TableSpec(int(math.floor(math.exp(x))), "fixed", 1, 1, 1, "uniform") for x in ls]
        c = Config(4, "1x10M rows PF50 Zipf 1.5 + 25 tables 1e3..1e6 rows PF1 uniform, E64 fp32, B4096",
                   64, "f32", -0.05, 0.05, 4096, tabs)
    elif i == 5:
        ls = rng(5, P_SIZES).uniform(math.log(1e3), math.log(2e7), size=100)
        rows = [int(math.floor(math.exp(x))) for x in ls]
        cap = 150 * 10 ** 9
        tot = sum(rows) * 128 * 4
        note = ""
        if tot > cap:
            rows = [max(1000, int(math.floor(m * cap / tot))) for m in rows]
            note = "rows scaled to the 150 GB cap"
        tabs = [TableSpec(m, "poisson", 20.0, 1, 100, "zipf", 1.1) for m in rows]
        c = Config(5, "100 tables 1e3..2e7 rows (<=150 GB), E128 fp32, B65536, PF Poisson(20) in [1,100], Zipf 1.1",
                   128, "f32", -0.05, 0.05, 65536, tabs, note=note)
    else:
        raise ValueError(f"config {i} does not exist (1..5)")
    c.value_seeds = [value_seed(i, t) for t in range(c.T)]
    return c


# ----------------------------------------------------------------------------
# Query batches
# ----------------------------------------------------------------------------

_CDF_CACHE: dict = {}


def zipf_cdf(m: int, alpha: float) -> np.ndarray:
    """Unnormalised CDF of the bounded Zipf law P(k) ~ k**-alpha, k = 1..m (float64)."""
    key = (m, alpha)
    c = _CDF_CACHE.get(key)
    if c is None:
        k = np.arange(1, m + 1, dtype=np.float64)
        c = np.cumsum(np.power(k, -alpha))
        if m >= 1 << 20:
            _CDF_CACHE.clear()
        _CDF_CACHE[key] = c
    return c


def zipf_ranks(g: np.random.Generator, m: int, alpha: float, n: int) -> np.ndarray:
    """n bounded-Zipf ranks in [0, m) by inverse CDF (numpy's zipf is unbounded, alpha>1 only)."""
    cdf = zipf_cdf(m, alpha)
    u = g.random(n) * cdf[-1]
    r = np.searchsorted(cdf, u, side="right")
    return np.minimum(r, m - 1).astype(np.int64)


def rank_permutation(cfg: int, t: int, m: int) -> np.ndarray:
    """Seeded random permutation rank -> row of table t."""
    p = rng(cfg, P_PERM, t).permutation(m)
    return p.astype(np.int32 if m < (1 << 31) else np.int64)


def pooling_factors(c: Config, t: int, batch_id: int, B: Optional[int] = None) -> np.ndarray:
    B = c.batch if B is None else B
    tb = c.tables[t]
    if tb.pf_kind == "fixed":
        return np.full(B, int(tb.pf_value), dtype=np.int64)
    g = rng(c.cfg_id, P_PF, t, batch_id)
    return np.clip(g.poisson(tb.pf_value, size=B), tb.pf_lo, tb.pf_hi).astype(np.int64)


def fixed_row(cfg: int, t: int, m: int) -> int:
    """The one row every lookup of table t reads under the 'fixed' distribution: a
    seeded row, the same in every batch (history batch included)."""
    return int(rng(cfg, P_FIXED, t).integers(0, m))


def table_indices(c: Config, t: int, n: int, batch_id: int, perm: Optional[np.ndarray] = None) -> np.ndarray:
    """n row ids of table t for batch ``batch_id``."""
    tb = c.tables[t]
    if tb.dist == "fixed":
        return np.full(n, fixed_row(c.cfg_id, t, tb.rows), dtype=np.int64)
    g = rng(c.cfg_id, P_INDICES, t, batch_id)
    if tb.dist == "uniform":
        return g.integers(0, tb.rows, size=n, dtype=np.int64)
    ranks = zipf_ranks(g, tb.rows, tb.alpha, n)
    if perm is None:
        perm = rank_permutation(c.cfg_id, t, tb.rows)
    return perm[ranks].astype(np.int64)


@dataclass
class Batch:
    B: int
    T: int
    indices: np.ndarray     # int64 [L], table-major concatenation of bags
    offsets: np.ndarray     # int64 [T*B + 1], bag (t, b) = indices[offsets[t*B+b] : offsets[t*B+b+1]]

    @property
    def n_lookups(self) -> int:
        return int(self.offsets[-1])


def gen_table_batch(c: Config, t: int, batch_id: int, B: Optional[int] = None,
                    perm: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """(pooling factors [B], indices [sum pf]) of table t."""
    pf = pooling_factors(c, t, batch_id, B)
    idx = table_indices(c, t, int(pf.sum()), batch_id, perm)
    return pf, idx


def gen_batch(c: Config, batch_id: int, B: Optional[int] = None, threads: Optional[int] = None) -> Batch:
    B = c.batch if B is None else B
    nthr = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(nthr) as ex:
        parts = list(ex.map(lambda t: gen_table_batch(c, t, batch_id, B), range(c.T)))
    pf = np.concatenate([p for p, _ in parts])
    offsets = np.zeros(c.T * B + 1, dtype=np.int64)
    np.cumsum(pf, out=offsets[1:])
    indices = np.concatenate([i for _, i in parts]) if parts else np.zeros(0, np.int64)
    return Batch(B, c.T, indices, offsets)


def batch_from_bags(T: int, B: int, bags: Sequence[Sequence[int]]) -> Batch:
    """Batch from an explicit table-major list of T*B bags (tests)."""
    assert len(bags) == T * B
    lens = np.array([len(x) for x in bags], dtype=np.int64)
    off = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    idx = np.array([v for x in bags for v in x], dtype=np.int64)
    return Batch(B, T, idx, off)


# ----------------------------------------------------------------------------
# Planner statistics (the paper's S and I: sequence lengths and query distribution)
# ----------------------------------------------------------------------------

@dataclass
class TableStats:
    mean_pooling: float
    max_pooling: int
    hot_rows: np.ndarray        # int64, hottest first (count desc, row asc)
    hot_freq: np.ndarray        # float64, fraction of the table's lookups on each hot row
    unique_frac: float


def stats_from_indices(idx: np.ndarray, pf: np.ndarray, max_pooling: int, n_hot: int = N_HOT_STATS) -> TableStats:
    n = int(idx.size)
    if n == 0:
        return TableStats(float(pf.mean()) if pf.size else 0.0, max_pooling,
                          np.zeros(0, np.int64), np.zeros(0, np.float64), 1.0)
    rows, counts = np.unique(idx, return_counts=True)
    order = np.lexsort((rows, -counts))[:n_hot]          # count desc, row asc
    return TableStats(float(pf.mean()), int(max_pooling), rows[order].astype(np.int64),
                      counts[order].astype(np.float64) / float(n), float(rows.size) / float(n))


def history_stats(c: Config, B: Optional[int] = None, threads: Optional[int] = None) -> List[TableStats]:
    """Statistics of each table measured on the history batch (batch_id 1000)."""
    nthr = threads or min(16, os.cpu_count() or 1)

    def one(t):
        pf, idx = gen_table_batch(c, t, HISTORY_BATCH, B)
        return stats_from_indices(idx, pf, c.max_pooling(t))

    with ThreadPoolExecutor(nthr) as ex:
        return list(ex.map(one, range(c.T)))


def algorithmic_bytes(c: Config, n_lookups: int, B: Optional[int] = None) -> dict:
    """Bytes one batch names: every lookup's row + indices + offsets + output (a row read
    twice counts twice; see ``compulsory_bytes`` for what must cross HBM)."""
    B = c.batch if B is None else B
    R = c.row_bytes
    rows = n_lookups * R
    idx = n_lookups * 8
    offs = (c.T * B + 1) * 8
    out = c.T * B * c.E * 4
    return {"rows": rows, "indices": idx, "offsets": offs, "out": out, "total": rows + idx + offs + out}


def distinct_rows(c: Config, batch: "Batch") -> List[int]:
    """Distinct valid row ids each table's lookups of ``batch`` name."""
    B = batch.B
    out = []
    for t, m in enumerate(c.rows):
        ids = batch.indices[batch.offsets[t * B]: batch.offsets[(t + 1) * B]]
        ids = ids[(ids >= 0) & (ids < m)]
        seen = np.zeros(m, dtype=np.bool_)
        seen[ids] = True
        out.append(int(np.count_nonzero(seen)))
    return out


def compulsory_bytes(c: Config, batch: "Batch", weighted: bool = False) -> dict:
    """Bytes one batch must move between HBM and the chip at the least: each distinct row
    once, every index (and weight), every offset and the output once."""
    B = batch.B
    L = batch.n_lookups
    rows = sum(distinct_rows(c, batch)) * c.row_bytes
    idx = L * 8 + (L * 4 if weighted else 0)
    offs = (c.T * B + 1) * 8
    out = c.T * B * c.E * 4
    return {"rows": rows, "indices": idx, "offsets": offs, "out": out, "total": rows + idx + offs + out}

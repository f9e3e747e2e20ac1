"""Planner oracle (test infrastructure only): cost model + greedy asymmetric mapping.

The paper (Sec. III) chooses one data-flow strategy per table with a linear
cost model (Eq. (2)), then maps tables, or row chunks of them, onto the K
cores of the SoC with a greedy algorithm (Sec. III-B, "Sharding and Load
Balancing", steps 1-4) and falls back to symmetric (batch-split) partitioning
when the load imbalance factor LIF = t_max / t_avg crosses a threshold.

This module restates that algorithm for the GPU strategies (LDS-resident
table/chunk, hot-row LDS cache, tile sort/dedup, direct HBM gather) in a form
with every tie-break pinned, so that the C++ planner can be checked against it
byte for byte.  It uses binary64 ``+ - * /`` and ``floor`` only; every cost is
floored to integer picoseconds right after it is computed, and every decision
compares integers.

Steps (names follow the paper's notation: m_t rows, s_t sequence length /
pooling factor, B batch, K cores = GPU workers, L persistent-buffer size = LDS
budget for rows):

  P1  strategy choice per table at split k: minimum cost among the feasible
      strategies in the fixed order LDS, HOT, DEDUP, GATHER, STREAM (ties ->
      earlier).  LDS is feasible iff m_t R <= L; HOT iff C_t >= 1 with C_t =
      min(hot rows listed, floor(L / R), 2048) the most hot rows one slice may
      stage.  HOT stages the first C listed rows, C taken among 1, 2, 4, ...
      below C_t and C_t itself, the one of least cost at the slice's lookups
      (ties -> the smaller C); h(C) is the fraction of lookups those rows catch
      (summed in list order).  u_t = unique fraction (1 if unknown).  STREAM (the GM-UB flow of Sec. II-B: the table
      moves through the buffer in chunks, each chunk serving the lookups that
      fall in it) takes c_t = ceil(m_t / floor(L / R)) chunks on one worker; it
      is a candidate when forced, or when c_t <= 64 and its cost stays below the
      cost cap (a larger one is left out, not an error).
  P2  (paper step 1) a table larger than L is split into the fewest chunks of
      at most floor(min(chunk_max, L) / R) rows, but only if its best unsplit
      cost exceeds the sum of the chunk costs (the speed-up exceeds the number
      of chunks); chunks use the LDS strategy.
  P3  tau = ceil(sum of item costs / K), the ideal per-worker load.
  P4  (skipped with no_replication: the paper's solver fixes the replication
      factor to 1, so with order_mode 1 the plan is Sec. III-B steps 1-4 as
      printed)
      an unchunked GATHER item whose k = min(K, B) slices would each hold at
      least 64 expected lookups (Lam_t / k >= 64) is split k ways (symmetric
      partitioning, Sec. III-A: a gather slice stages nothing, so every worker
      takes 1/k of every such table and the mix of cache-resident and
      HBM-bound tables is the same on every worker); smaller ones are split
      like the others (T x K tiny slices would swamp the launch), which leaves
      small tables whole and places them asymmetrically (Sec. III-B).  With
      sym_max > 0 every GATHER item is split k ways while the plan has at most
      sym_max of them; sym_max < 0 turns symmetric splitting off.  Any other item
      costing more than tau is batch-split k ways (the paper's optional
      replication): the smallest k in [2, min(K, B)] whose best cost is at most
      max(tau, 2 x its fixed cost); all chunks of one table share one k.  A
      split item keeps the strategy that is best at its k.
  P5  (paper step 2) slices sorted by (cost desc, s desc, m asc, t, chunk, j)
      -- longest-processing-time first with the paper's keys as tie-breaks --
      or, with order_mode 1, by the paper's literal key (s desc, m asc, t,
      chunk, j).
  P6  (paper step 2) each slice goes to the least-loaded worker (ties -> lowest
      index).  (Paper step 3, "L1 if available", is per item here: LDS does not
      persist across launches, so every item re-stages its own rows.)
  P7  (paper step 4) if LIF (in thousandths) exceeds the threshold, the last r
      tables of the paper's order (s desc, m asc, t) become symmetric -- split
      min(K, B) ways with slice j on worker j, placed first -- for r = 1, 2, ...
      until LIF is within the threshold; if no r gets there, the r (0
      included) with the smallest maximum load.
  P8  canonical text: one line per slice in worker order then placement order.

A table may carry its own G1, the cost of one lookup served from memory (its
gathers, HOT misses and DEDUP's distinct rows), fitted on the device for that
table's size and query distribution: Sec. III-A fits the model's coefficients per
configuration.  Every other coefficient is shared.
"""
from __future__ import annotations

import heapq
import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

# strategies (same numbering as the C header)
LDS, HOT, DEDUP, GATHER, STREAM = 0, 1, 2, 3, 4
AUTO = -1
STRAT_ORDER = (LDS, HOT, DEDUP, GATHER, STREAM)

# beta layout (picoseconds; per item, per lookup, per staged byte)
G0, G1, L0, L1, S, I, H0, P, D0, D1, SH = range(11)
NBETA = 11

MAX_HOT = 4096          # hot rows a table's statistics may list
MAX_HOT_SLOTS = 2048    # hot rows one HOT item stages at most
MAX_CHUNKS = 65536
STREAM_MAX_CHUNKS = 64  # STREAM is an automatic candidate up to this many chunks
SYM_SHARE_MIN = 64.0    # GATHER tables split over all workers when each slice would hold this many lookups


class PlanError(ValueError):
    pass


def default_beta(R: int) -> List[float]:
    """Built-in coefficients (picoseconds): the least-squares fit (Eq. (2), Sec. III-A) of the
    MI355X calibration samples in tests/golden/calibration_samples.csv, each rounded to three
    significant digits.

    The fit is sequential, each stage on what the earlier ones leave, and every stage is
    reweighted once so that residuals count relative to each sample's predicted time:
    GATHER (G0 per slice, G1 per lookup) on the workers' gather phases; LDS (L0, S per staged
    byte, L1 per lookup) on whole-table slices; I on the row-chunk slices; HOT (H0, SH per
    staged byte, P per lookup) and DEDUP (D0, D1 per lookup).  The samples use R = 256 B
    rows; the per-lookup terms serve unchanged for other row sizes.
    """
    del R
    b = [0.0] * NBETA
    b[G0] = 480000.0
    b[G1] = 6370.0
    b[L0] = 997000.0
    b[L1] = 11100.0
    b[S] = 41.1
    b[I] = 38500.0
    b[H0] = 4110000.0
    b[P] = 5790.0
    b[D0] = 8190000.0
    b[D1] = 24600.0
    b[SH] = 35.5
    return b


@dataclass
class Stat:
    mean_pooling: float
    max_pooling: int = 0
    hot_freq: Sequence[float] = ()
    unique_frac: float = -1.0

    @property
    def n_hot(self) -> int:
        return len(self.hot_freq)


@dataclass
class Options:
    lds_budget: int = 131072
    lif_milli: int = 1500
    chunk_max_bytes: int = 0          # <= 0 -> lds_budget
    order_mode: int = 0
    beta: Optional[Sequence[float]] = None
    force: Optional[Sequence[int]] = None
    sym_max: int = 0                  # > 0: GATHER items split symmetrically while at most this many; < 0: never
    no_replication: bool = False      # True: no batch splits (P4 off), replication factor 1
    gather_lookup_ps: Optional[Sequence[float]] = None   # per table G1 (0: beta's), or None


@dataclass
class Slice:
    wg: int
    t: int
    strat: int
    chunk: int
    nchunks: int
    r0: int
    r1: int
    k: int
    j: int
    C: int
    cost: int
    seq: int = 0          # placement sequence number


@dataclass
class Plan:
    T: int
    E: int
    dtype: str
    R: int
    K: int
    L: int
    B: int
    theta: int
    order_mode: int
    slices: List[Slice] = field(default_factory=list)
    max_ps: int = 0
    sum_ps: int = 0
    lif_milli: int = 0
    r_sym: int = 0
    sym_max: int = 0
    no_replication: bool = False

    def text(self) -> str:
        lines = ["embx-plan v1",
                 f"T {self.T} E {self.E} dtype {self.dtype} R {self.R} K {self.K} L {self.L} B {self.B} "
                 f"theta {self.theta} order {self.order_mode} symmax {self.sym_max}"
                 + (" norepl 1" if self.no_replication else "")]
        for s in sorted(self.slices, key=lambda x: (x.wg, x.seq)):
            lines.append(f"item {s.wg} {s.t} {s.strat} {s.chunk} {s.nchunks} {s.r0} {s.r1} {s.k} {s.j} {s.C} {s.cost}")
        lines.append(f"end max {self.max_ps} sum {self.sum_ps} lif {self.lif_milli} sym {self.r_sym}")
        return "\n".join(lines) + "\n"


COST_CAP = 2.0 ** 40          # a slice costing more (about 1.1 s) is rejected
MAX_SLICES = 1 << 20


def _fl(x: float) -> int:
    """floor to integer picoseconds, never negative."""
    if not math.isfinite(x) or x >= COST_CAP:
        raise PlanError("cost model out of range")
    v = math.floor(x)
    return v if v > 0 else 0


# --- Eq. (2), one worker's cost for one slice; lam = expected lookups of the slice -------------

def cost_gather(b, lam):
    return _fl(b[G0] + b[G1] * lam), _fl(b[G0])


def cost_lds(b, mu, R, lam):
    return _fl(b[L0] + b[S] * float(mu * R) + b[L1] * lam), _fl(b[L0] + b[S] * float(mu * R))


def cost_chunk(b, mu, R, lam, c):
    return (_fl(b[L0] + b[S] * float(mu * R) + b[I] * lam + b[L1] * (lam / float(c))),
            _fl(b[L0] + b[S] * float(mu * R)))


def cost_hot(b, C, R, h, lam):
    return (_fl(b[H0] + b[SH] * float(C * R) + lam * (b[P] + h * b[L1] + (1.0 - h) * b[G1])),
            _fl(b[H0] + b[SH] * float(C * R)))


def cost_dedup(b, u, lam):
    return _fl(b[D0] + b[D1] * lam + (b[G1] * u) * lam), _fl(b[D0])


def cost_stream(b, m, R, lam, c):
    """The whole table through LDS in c chunks on one worker: each chunk scans the
    slice's lookups (I), each lookup is read from LDS once (L1)."""
    return (_fl(b[L0] + b[S] * float(m * R) + b[I] * lam * float(c) + b[L1] * lam),
            _fl(b[L0] + b[S] * float(m * R)))


class _Table:
    def __init__(self, t, m, st: Stat, R, L, B, force, g1=None):
        self.t, self.m, self.R = t, m, R
        self.g1 = float(g1) if g1 else None   # this table's G1, None: beta's
        self.s = float(st.mean_pooling)
        self.Lam = float(B) * self.s
        self.C = min(st.n_hot, L // R, MAX_HOT_SLOTS)
        # HOT candidates (C, h(C)): C = 1, 2, 4, ... below the cap, and the cap
        self.hot_sizes = []
        h = 0.0
        for k in range(self.C):
            h = h + float(st.hot_freq[k])
            n = k + 1
            if (n & (n - 1)) == 0 or n == self.C:
                self.hot_sizes.append((n, h))
        u = float(st.unique_frac)
        self.u = u if (u > 0.0 and u <= 1.0) else 1.0
        self.fits = m * R <= L
        self.sc = (m + L // R - 1) // (L // R)   # STREAM chunks
        self.force = force

    def allowed(self, b, k):
        out = []
        for s in STRAT_ORDER:
            if self.force != AUTO and s != self.force:
                continue
            if s == LDS and not self.fits:
                continue
            if s == HOT and self.C < 1:
                continue
            if s == STREAM and self.force == AUTO and not self.stream_ok(b, k):
                continue
            out.append(s)
        return out

    def stream_ok(self, b, k):
        if self.sc > STREAM_MAX_CHUNKS:
            return False
        lam = self.Lam / float(k)
        x = b[L0] + b[S] * float(self.m * self.R) + b[I] * lam * float(self.sc) + b[L1] * lam
        return math.isfinite(x) and x < COST_CAP

    def cost(self, b, strat, k):
        """(cost, fixed cost, hot rows staged) of one slice at split k."""
        if self.g1 is not None:
            b = list(b[:G1]) + [self.g1] + list(b[G1 + 1:])
        lam = self.Lam / float(k)
        if strat == LDS:
            return cost_lds(b, self.m, self.R, lam) + (0,)
        if strat == HOT:
            best = None
            for C, h in self.hot_sizes:
                c, f = cost_hot(b, C, self.R, h, lam)
                if best is None or c < best[0]:
                    best = (c, f, C)
            return best
        if strat == DEDUP:
            return cost_dedup(b, self.u, lam) + (0,)
        if strat == STREAM:
            return cost_stream(b, self.m, self.R, lam, self.sc) + (0,)
        return cost_gather(b, lam) + (0,)

    def best(self, b, k):
        """(strategy, cost, fixed cost, hot rows staged) -- P1, ties to the earlier strategy."""
        best = None
        for s in self.allowed(b, k):
            c, f, C = self.cost(b, s, k)
            if best is None or c < best[1]:
                best = (s, c, f, C)
        return best


@dataclass
class _Item:
    t: int
    chunk: int
    nchunks: int
    r0: int
    r1: int
    strat: int = GATHER
    k: int = 1
    cost: int = 0          # cost of one slice at split k
    C: int = 0             # HOT: hot rows staged


def _validate(rows, E, dtype, stats, B, K, opts: Options):
    T = len(rows)
    if T < 1 or len(stats) != T:
        raise PlanError("need T >= 1 tables with stats")
    if dtype not in ("f32", "f16"):
        raise PlanError("dtype")
    esz = 4 if dtype == "f32" else 2
    if E < 1 or E > 256 or (E * esz) % 16 != 0:
        raise PlanError("E must make 16-byte multiple rows, E <= 256")
    if B < 1 or K < 1:
        raise PlanError("B and K must be >= 1")
    R = E * esz
    L = int(opts.lds_budget)
    if L < R:
        raise PlanError("LDS budget below one row")
    for m in rows:
        if m < 1 or m >= (1 << 31):
            raise PlanError("rows must be in [1, 2^31)")
    for st in stats:
        if not (math.isfinite(st.mean_pooling) and st.mean_pooling >= 0.0):
            raise PlanError("mean_pooling")
        if st.n_hot > MAX_HOT:
            raise PlanError("n_hot")
        for f in st.hot_freq:
            if not (math.isfinite(f) and f >= 0.0):
                raise PlanError("hot_freq")
        if not math.isfinite(st.unique_frac):
            raise PlanError("unique_frac")
    if opts.order_mode not in (0, 1):
        raise PlanError("order_mode")
    beta = list(opts.beta) if opts.beta is not None else default_beta(R)
    # the coefficients price times: a negative one can make a slice cost less than
    # nothing, and least-loaded placement would then pile such slices onto one worker
    if len(beta) != NBETA or not all(math.isfinite(x) and x >= 0.0 for x in beta):
        raise PlanError("beta")
    g1 = list(opts.gather_lookup_ps) if opts.gather_lookup_ps is not None else None
    if g1 is not None and (len(g1) != T or not all(math.isfinite(x) and x >= 0.0 for x in g1)):
        raise PlanError("gather_lookup_ps")
    force = list(opts.force) if opts.force is not None else [AUTO] * T
    if len(force) != T or any(f not in (AUTO, LDS, HOT, DEDUP, GATHER, STREAM) for f in force):
        raise PlanError("force_strategy")
    return T, R, L, beta, force, g1


def plan_reference(rows: Sequence[int], E: int, dtype: str, stats: Sequence[Stat], B: int, K: int,
                   opts: Optional[Options] = None) -> Plan:
    opts = opts or Options()
    T, R, L, b, force, g1 = _validate(rows, E, dtype, stats, B, K, opts)
    cm = opts.chunk_max_bytes if opts.chunk_max_bytes > 0 else L
    crow = min(cm, L) // R
    if crow < 1:
        raise PlanError("chunk_max_bytes below one row")
    tabs = [_Table(t, int(rows[t]), stats[t], R, L, B, force[t], g1[t] if g1 is not None else None)
            for t in range(T)]
    for tb in tabs:
        if tb.force == HOT and tb.C < 1:
            raise PlanError("HOT forced on a table without hot rows")

    # P1 + P2: strategy per table, chunking of tables larger than L
    items: List[_Item] = []
    groups: List[List[_Item]] = []
    for tb in tabs:
        chunked = False
        c = 1
        if not tb.fits and tb.force in (AUTO, LDS):
            c = (tb.m + crow - 1) // crow
            if tb.force == LDS:
                if c > MAX_CHUNKS:
                    raise PlanError("too many chunks")
                chunked = True
            elif 2 <= c <= K:
                csum = 0
                for i in range(c):
                    r0, r1 = (i * tb.m) // c, ((i + 1) * tb.m) // c
                    csum += cost_chunk(b, r1 - r0, R, tb.Lam, c)[0]
                chunked = tb.best(b, 1)[1] > csum
        g = []
        if chunked:
            for i in range(c):
                r0, r1 = (i * tb.m) // c, ((i + 1) * tb.m) // c
                it = _Item(tb.t, i, c, r0, r1, LDS, 1, cost_chunk(b, r1 - r0, R, tb.Lam, c)[0])
                g.append(it)
        else:
            s, cst, _, C = tb.best(b, 1)
            g.append(_Item(tb.t, 0, 1, 0, tb.m, s, 1, cst, C))
        groups.append(g)
        items.extend(g)

    # P3
    total1 = sum(it.cost for it in items)
    tau = (total1 + K - 1) // K
    kmax = min(K, B)

    # P4
    def split_k(it: _Item):
        """smallest k in [2, kmax] with cost_k <= max(tau, 2 fixed_k), else kmax."""
        tb = tabs[it.t]
        for k in range(2, kmax + 1):
            s, cst, fx, _ = _item_best(tb, it, k)
            if cst <= max(tau, 2 * fx):
                return k
        return kmax

    def _item_best(tb, it, k):
        if it.nchunks > 1:
            lam = tb.Lam / float(k)
            c, f = cost_chunk(b, it.r1 - it.r0, R, lam, it.nchunks)
            return LDS, c, f, 0
        return tb.best(b, k)

    sym_max = opts.sym_max
    n_gather = sum(1 for g in groups if g[0].nchunks == 1 and g[0].strat == GATHER)
    few_gather = sym_max > 0 and n_gather <= sym_max
    for g in groups:
        if opts.no_replication:
            break
        sym = (sym_max >= 0 and g[0].nchunks == 1 and g[0].strat == GATHER and
               (few_gather or tabs[g[0].t].Lam / float(kmax) >= SYM_SHARE_MIN))
        if sym:
            ks = [kmax]
        else:
            ks = [1 if it.cost <= tau else split_k(it) for it in g]
        k = max(ks)
        for it in g:
            s, cst, _, C = _item_best(tabs[it.t], it, k)
            it.strat, it.k, it.cost, it.C = s, k, cst, C

    def slices_of(it: _Item) -> List[Slice]:
        C = it.C if it.strat == HOT else 0
        return [Slice(-1, it.t, it.strat, it.chunk, it.nchunks, it.r0, it.r1, it.k, j, C, it.cost)
                for j in range(it.k)]

    def key(sl: Slice):
        tb = tabs[sl.t]
        if opts.order_mode == 0:
            return (-sl.cost, -tb.s, tb.m, sl.t, sl.chunk, sl.j)
        return (-tb.s, tb.m, sl.t, sl.chunk, sl.j)

    paper_order = sorted(range(T), key=lambda t: (-tabs[t].s, tabs[t].m, t))

    def place(demoted: List[int]):
        """P5 + P6 (+ symmetric tables of P7 first). Returns (slices, loads)."""
        loads = [0] * K
        seq = 0
        out: List[Slice] = []
        dem = set(demoted)
        for t in [x for x in paper_order if x in dem]:
            for it in groups[t]:
                tb = tabs[t]
                s, cst, _, C = _item_best(tb, it, kmax)
                sym = _Item(it.t, it.chunk, it.nchunks, it.r0, it.r1, s, kmax, cst, C)
                for sl in slices_of(sym):
                    sl.wg = sl.j
                    sl.seq = seq
                    seq += 1
                    loads[sl.wg] += sl.cost
                    out.append(sl)
        rest = [sl for g in groups if g[0].t not in dem for it in g for sl in slices_of(it)]
        if len(rest) + len(out) > MAX_SLICES:
            raise PlanError("too many slices")
        rest.sort(key=key)
        heap = [(loads[w], w) for w in range(K)]
        heapq.heapify(heap)
        for sl in rest:
            ld, w = heapq.heappop(heap)
            sl.wg = w
            sl.seq = seq
            seq += 1
            loads[w] = ld + sl.cost
            heapq.heappush(heap, (loads[w], w))
            out.append(sl)
        return out, loads

    def lif_of(loads):
        tot = sum(loads)
        return (1000 * K * max(loads)) // tot if tot > 0 else 1000

    best_r, best_slices, best_loads = 0, *place([])
    lif = lif_of(best_loads)
    if lif > opts.lif_milli:
        found = False
        cand = (max(best_loads), 0, best_slices, best_loads)
        for r in range(1, T + 1):
            sl_r, ld_r = place(paper_order[T - r:])
            if lif_of(ld_r) <= opts.lif_milli:
                best_r, best_slices, best_loads = r, sl_r, ld_r
                found = True
                break
            if max(ld_r) < cand[0]:
                cand = (max(ld_r), r, sl_r, ld_r)
        if not found:
            _, best_r, best_slices, best_loads = cand

    plan = Plan(T, E, dtype, R, K, L, B, opts.lif_milli, opts.order_mode)
    plan.sym_max = sym_max
    plan.no_replication = bool(opts.no_replication)
    plan.slices = best_slices
    plan.max_ps = max(best_loads)
    plan.sum_ps = sum(best_loads)
    plan.lif_milli = lif_of(best_loads)
    plan.r_sym = best_r
    return plan


def stats_from_workload(ts) -> Stat:
    """Adapter from ``workloads.TableStats`` (host lists only)."""
    return Stat(float(ts.mean_pooling), int(ts.max_pooling), [float(x) for x in ts.hot_freq], float(ts.unique_frac))

"""Pins of the planner oracle.

The paper prints no worked plan, so the plan is pinned by properties that any
correct reading must satisfy: the cost formulas agree with each other in the
cases where two strategies coincide, every bag of every table (or row chunk)
is covered exactly once, LDS capacity holds per item, the reported loads and
LIF recompute from the slices, special cases have known answers, and the
greedy placement obeys the classical list-scheduling bounds against a
brute-force optimum (Graham 1969: LPT <= (4/3 - 1/(3K)) OPT, any list order
<= (2 - 1/K) OPT).
"""
import itertools
import math

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import plan as OPL


def _b(R=256):
    return OPL.default_beta(R)


def _roofline_beta(R=256):
    """Coefficients from bandwidths alone (a row at one CU's share of HBM, LDS at
    128 B/clk), for special cases whose premise is that LDS beats HBM per lookup."""
    b = [0.0] * OPL.NBETA
    b[OPL.G0], b[OPL.G1] = 200000.0, R * 32.0 / 0.7
    b[OPL.L0], b[OPL.L1], b[OPL.S], b[OPL.I] = 200000.0, R / 0.3072, 32.0, 256.0
    b[OPL.H0], b[OPL.P], b[OPL.D0], b[OPL.D1] = 200000.0, 100.0, 200000.0, 4000.0
    b[OPL.SH] = 32.0
    return b


# ---------------------------------------------------------------- cost model cross-checks

def test_cost_formulas_coincide_where_strategies_do():
    b = _b()
    R, lam = 256, 12345.0
    # gather is affine in lam: the slope is the per-lookup coefficient
    g1, _ = OPL.cost_gather(b, lam)
    g2, _ = OPL.cost_gather(b, 2 * lam)
    assert abs((g2 - g1) - b[OPL.G1] * lam) <= 1
    # a hot set that catches nothing with a free probe is a gather plus staging
    bz = list(b)
    bz[OPL.P] = 0.0
    bz[OPL.H0] = bz[OPL.G0]
    hot0, fx = OPL.cost_hot(bz, 100, R, 0.0, lam)
    assert abs(hot0 - (g1 + b[OPL.SH] * 100 * R)) <= 1 and fx == math.floor(bz[OPL.G0] + b[OPL.SH] * 100 * R)
    # a hot set that catches everything with a free probe, staged at the LDS byte
    # cost, is an LDS table of C rows
    bl = list(bz)
    bl[OPL.H0] = bl[OPL.L0]
    bl[OPL.SH] = bl[OPL.S]
    hot1, _ = OPL.cost_hot(bl, 100, R, 1.0, lam)
    lds, _ = OPL.cost_lds(bl, 100, R, lam)
    assert abs(hot1 - lds) <= 1
    # one chunk with a free index scan is the whole-table LDS cost
    bi = list(b)
    bi[OPL.I] = 0.0
    assert OPL.cost_chunk(bi, 77, R, lam, 1) == OPL.cost_lds(bi, 77, R, lam)
    # dedup with every lookup unique and free sorting is a gather
    bd = list(b)
    bd[OPL.D1] = 0.0
    bd[OPL.D0] = bd[OPL.G0]
    assert OPL.cost_dedup(bd, 1.0, lam) == OPL.cost_gather(bd, lam)
    # all costs grow with lam and never go negative
    for f in (lambda l: OPL.cost_gather(b, l), lambda l: OPL.cost_lds(b, 50, R, l),
              lambda l: OPL.cost_hot(b, 50, R, 0.5, l), lambda l: OPL.cost_dedup(b, 0.3, l),
              lambda l: OPL.cost_chunk(b, 50, R, l, 3)):
        assert 0 <= f(0.0)[0] <= f(10.0)[0] <= f(1e6)[0]
    neg = [-1e9] * OPL.NBETA
    assert OPL.cost_gather(neg, 5.0) == (0, 0)


# ---------------------------------------------------------------- invariants on random instances

def _random_instance(seed, T=None, K=None):
    g = np.random.default_rng(seed)
    T = T or int(g.integers(1, 14))
    K = K or int(g.integers(1, 24))
    B = int(g.integers(1, 3000))
    rows = [int(math.floor(math.exp(g.uniform(0, math.log(3e6))))) + 1 for _ in range(T)]
    stats = []
    for _ in range(T):
        nh = int(g.integers(0, 40))
        f = np.sort(g.random(nh))[::-1]
        f = f / (f.sum() * g.uniform(1.0, 3.0)) if nh else f
        stats.append(OPL.Stat(float(g.choice([0.0, 1.0, 3.5, 8.0, 50.0])), 20, [float(x) for x in f],
                              float(g.choice([-1.0, 0.05, 0.5, 1.0]))))
    E = int(g.choice([32, 64, 128]))
    dtype = str(g.choice(["f32", "f16"]))
    opts = OPL.Options(lds_budget=int(g.choice([16384, 65536, 131072])), lif_milli=int(g.choice([1000, 1250, 2000])),
                       order_mode=int(g.integers(0, 2)), no_replication=bool(g.integers(0, 4) == 0))
    return rows, E, dtype, stats, B, K, opts


def check_plan_invariants(p: OPL.Plan, rows, stats, B):
    R, L, K = p.R, p.L, p.K
    by_item = {}
    for s in p.slices:
        assert 0 <= s.wg < K
        by_item.setdefault((s.t, s.chunk), []).append(s)
        if s.strat == OPL.LDS:
            assert (s.r1 - s.r0) * R <= L
        if s.strat == OPL.HOT:
            assert 1 <= s.C and s.C * R <= L and s.C <= len(stats[s.t].hot_freq)
        else:
            assert s.C == 0
        if s.nchunks > 1:
            assert s.strat == OPL.LDS
    for t in range(p.T):
        chunks = sorted(c for (tt, c) in by_item if tt == t)
        assert chunks == list(range(len(chunks))) and len(chunks) >= 1
        bounds = []
        ks = set()
        for c in chunks:
            sl = by_item[(t, c)]
            k = sl[0].k
            ks.add(k)
            assert sorted(x.j for x in sl) == list(range(k))       # every slice once
            assert all(x.k == k and x.nchunks == len(chunks) for x in sl)
            assert len({(x.r0, x.r1) for x in sl}) == 1
            bounds.append((sl[0].r0, sl[0].r1))
            assert 1 <= k <= max(1, min(K, B))
        assert len(ks) == 1                                        # one split per table
        pos = 0
        for r0, r1 in bounds:                                      # chunks tile [0, m)
            assert r0 == pos and r1 > r0
            pos = r1
        assert pos == rows[t]
        # the batch slices of a split cover every bag exactly once
        k = ks.pop()
        cover = np.zeros(B, np.int64)
        for j in range(k):
            cover[(j * B) // k: ((j + 1) * B) // k] += 1
        assert np.all(cover == 1)
    loads = [0] * K
    for s in p.slices:
        loads[s.wg] += s.cost
    assert p.max_ps == max(loads) and p.sum_ps == sum(loads)
    tot = sum(loads)
    assert p.lif_milli == ((1000 * K * max(loads)) // tot if tot else 1000)


@pytest.mark.parametrize("seed", range(40))
def test_plan_invariants_random(seed):
    rows, E, dtype, stats, B, K, opts = _random_instance(seed)
    p = OPL.plan_reference(rows, E, dtype, stats, B, K, opts)
    check_plan_invariants(p, rows, stats, B)
    assert p.text().startswith("embx-plan v1\n") and p.text().endswith(f"sym {p.r_sym}\n")


@settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(st.integers(0, 10 ** 6))
def test_plan_invariants_hypothesis(seed):
    rows, E, dtype, stats, B, K, opts = _random_instance(seed)
    check_plan_invariants(OPL.plan_reference(rows, E, dtype, stats, B, K, opts), rows, stats, B)


# ---------------------------------------------------------------- special cases

def test_K_identical_tables_one_per_worker():
    # staged tables (DEDUP forced) that each cost about tau stay whole: one per worker
    K = 8
    rows = [5_000_000] * K
    stats = [OPL.Stat(1.0)] * K
    p = OPL.plan_reference(rows, 64, "f32", stats, 2048, K, OPL.Options(force=[OPL.DEDUP] * K))
    assert sorted(s.wg for s in p.slices) == list(range(K))
    assert all(s.k == 1 and s.strat == OPL.DEDUP for s in p.slices)
    assert p.lif_milli == 1000


def test_gather_tables_are_partitioned_symmetrically():
    # gather tables are split over all workers: every worker gets one slice of each
    K, B = 8, 2048
    rows = [10, 5_000_000, 300_000]
    stats = [OPL.Stat(1.0), OPL.Stat(8.0), OPL.Stat(2.0)]
    p = OPL.plan_reference(rows, 64, "f32", stats, B, K, OPL.Options(force=[OPL.GATHER] * 3))
    assert len(p.slices) == 3 * K
    for t in range(3):
        assert sorted(s.wg for s in p.slices if s.t == t) == list(range(K))
        assert all(s.k == K for s in p.slices if s.t == t)
    assert p.lif_milli == 1000
    # fewer samples than workers: k = B (with sym_max > 0 every gather table is split)
    p = OPL.plan_reference(rows, 64, "f32", stats, 5, K, OPL.Options(force=[OPL.GATHER] * 3, sym_max=10))
    assert all(s.k == 5 for s in p.slices)
    # by default slices of 1..8 lookups are too small to split a table into symmetrically
    # (the LIF fallback, which may still do so, is held off here)
    p = OPL.plan_reference(rows, 64, "f32", stats, 5, K,
                           OPL.Options(force=[OPL.GATHER] * 3, lif_milli=1_000_000))
    assert not any(s.k == 5 for s in p.slices if s.t == 0)


def test_one_huge_table_is_split_over_all_workers():
    K, B = 16, 1000
    p = OPL.plan_reference([10_000_000], 64, "f32", [OPL.Stat(50.0)], B, K)
    assert len(p.slices) == K and sorted(s.wg for s in p.slices) == list(range(K))
    sizes = [((s.j + 1) * B) // K - (s.j * B) // K for s in p.slices]
    assert max(sizes) - min(sizes) <= 1
    assert p.lif_milli == 1000


def test_tiny_tables_with_many_lookups_stay_in_lds():
    rows = [10, 40, 100, 300]
    stats = [OPL.Stat(20.0)] * 4
    p = OPL.plan_reference(rows, 64, "f32", stats, 4096, 64, OPL.Options(beta=_roofline_beta()))
    assert all(s.strat == OPL.LDS for s in p.slices)


def test_chunking_decision_follows_the_speedup_rule():
    # LDS nearly free, HBM gather very expensive: a 4-chunk table is split (speed-up > 4)
    b = [0.0] * OPL.NBETA
    b[OPL.G1] = 1e6
    b[OPL.L1] = 1.0
    b[OPL.S] = 1e-3
    b[OPL.I] = 1.0
    b[OPL.D1] = 1e6
    b[OPL.P] = 1e6
    R, L = 256, 65536
    m = 4 * (L // R)
    p = OPL.plan_reference([m], 64, "f32", [OPL.Stat(10.0)], 100, 8, OPL.Options(lds_budget=L, beta=b))
    assert {s.nchunks for s in p.slices} == {4} and all(s.strat == OPL.LDS for s in p.slices)
    # scanning indices costs as much as gathering: the chunks cannot win
    b2 = list(b)
    b2[OPL.I] = 1e6
    p2 = OPL.plan_reference([m], 64, "f32", [OPL.Stat(10.0)], 100, 8, OPL.Options(lds_budget=L, beta=b2))
    assert {s.nchunks for s in p2.slices} == {1} and p2.slices[0].strat == OPL.GATHER
    # forcing LDS on a table larger than L chunks it regardless of cost
    p3 = OPL.plan_reference([m + 1], 64, "f32", [OPL.Stat(10.0)], 100, 2,
                            OPL.Options(lds_budget=L, force=[OPL.LDS]))
    assert {s.nchunks for s in p3.slices} == {5}


def test_force_strategy_and_errors():
    stats = [OPL.Stat(2.0, 4, [0.3, 0.2], 0.5), OPL.Stat(2.0)]
    for f in (OPL.HOT, OPL.DEDUP, OPL.GATHER):
        p = OPL.plan_reference([1000, 2000], 64, "f32", stats, 64, 4, OPL.Options(force=[f, OPL.GATHER]))
        assert {s.strat for s in p.slices if s.t == 0} == {f}
    with pytest.raises(OPL.PlanError):
        OPL.plan_reference([1000, 2000], 64, "f32", stats, 64, 4, OPL.Options(force=[OPL.AUTO, OPL.HOT]))
    with pytest.raises(OPL.PlanError):
        OPL.plan_reference([1000], 6, "f32", [OPL.Stat(1.0)], 64, 4)            # 24-byte rows
    with pytest.raises(OPL.PlanError):
        OPL.plan_reference([0], 64, "f32", [OPL.Stat(1.0)], 64, 4)
    with pytest.raises(OPL.PlanError):
        OPL.plan_reference([10], 64, "f32", [OPL.Stat(float("nan"))], 64, 4)


def test_order_mode_one_is_paper_order():
    rows = [100000, 200000, 300000, 400000]
    stats = [OPL.Stat(1.0), OPL.Stat(4.0), OPL.Stat(4.0), OPL.Stat(2.0)]
    p = OPL.plan_reference(rows, 64, "f32", stats, 1, 4, OPL.Options(order_mode=1, lif_milli=10 ** 9))
    first = [s.t for s in sorted(p.slices, key=lambda s: s.seq)]
    assert first == [1, 2, 3, 0]                  # s desc, then m asc


def test_lif_fallback_never_worsens_the_makespan():
    # one table that cannot be split (B = 1) dominates: LIF stays high
    rows = [5_000_000, 1000, 2000, 3000]
    stats = [OPL.Stat(100.0), OPL.Stat(1.0), OPL.Stat(1.0), OPL.Stat(1.0)]
    p0 = OPL.plan_reference(rows, 64, "f32", stats, 1, 8, OPL.Options(lif_milli=10 ** 9))
    p1 = OPL.plan_reference(rows, 64, "f32", stats, 1, 8, OPL.Options(lif_milli=1000))
    assert p1.max_ps <= p0.max_ps


def test_lif_fallback_makes_trailing_tables_symmetric():
    # two huge equal tables on three workers: LPT leaves one worker idle (LIF 1.5);
    # making the last table of the paper order symmetric spreads it over all workers
    rows = [1_000_000, 1_000_001]
    stats = [OPL.Stat(1.0), OPL.Stat(1.0)]
    b = OPL.default_beta(256)
    b[OPL.D0] = 1e9            # a big fixed cost keeps P4 from splitting
    p = OPL.plan_reference(rows, 64, "f32", stats, 3, 3,
                           OPL.Options(beta=b, lif_milli=1200, force=[OPL.DEDUP, OPL.DEDUP]))
    assert p.r_sym >= 1
    sym = [s for s in p.slices if s.t == 1]
    assert sorted(s.wg for s in sym) == [0, 1, 2] and all(s.k == 3 for s in sym)


# ---------------------------------------------------------------- scheduling bounds vs brute force

def _opt_makespan(costs, K):
    best = float("inf")
    for assign in itertools.product(range(K), repeat=len(costs)):
        loads = [0] * K
        for c, w in zip(costs, assign):
            loads[w] += c
        best = min(best, max(loads))
    return best


@pytest.mark.parametrize("seed", range(30))
def test_greedy_within_list_scheduling_bounds(seed):
    g = np.random.default_rng(1000 + seed)
    T = int(g.integers(2, 8))
    K = int(g.integers(2, 4))
    rows = [int(g.integers(100000, 3_000_000)) for _ in range(T)]
    stats = [OPL.Stat(float(g.integers(1, 30))) for _ in range(T)]
    for mode in (0, 1):
        p = OPL.plan_reference(rows, 64, "f32", stats, 1, K, OPL.Options(order_mode=mode, lif_milli=10 ** 9))
        assert all(s.k == 1 for s in p.slices)        # B = 1: nothing can be split
        opt = _opt_makespan([s.cost for s in p.slices], K)
        bound = (4.0 / 3.0 - 1.0 / (3 * K)) if mode == 0 else (2.0 - 1.0 / K)
        assert p.max_ps <= bound * opt + 1e-9, (mode, p.max_ps, opt)


def test_lpt_bound_is_tight_on_the_classic_instance():
    # Graham's tight example for K = 2: jobs 3,3,2,2,2 -> LPT 7, OPT 6
    b = [0.0] * OPL.NBETA
    b[OPL.G1] = 1.0
    stats = [OPL.Stat(float(x)) for x in (3, 3, 2, 2, 2)]
    rows = [10 ** 6 + i for i in range(5)]
    p = OPL.plan_reference(rows, 64, "f32", stats, 1, 2, OPL.Options(beta=b, lif_milli=10 ** 9))
    assert sorted(s.cost for s in p.slices) == [2, 2, 2, 3, 3]
    assert p.max_ps == 7 and _opt_makespan([2, 2, 2, 3, 3], 2) == 6


def test_many_gather_tables_are_placed_whole_not_split_over_all_workers():
    # 200 small gather tables on 64 workers (8 lookups per worker share): T x K tiny slices
    # would swamp a launch, so they are priced and split like any item; small ones stay
    # whole and are spread over the workers by least-loaded placement (the asymmetric mapping)
    g = np.random.default_rng(11)
    rows = [int(x) for x in g.integers(1000, 100000, size=200)]
    stats = [OPL.Stat(1.0) for _ in rows]
    b = OPL.default_beta(256)
    b[OPL.L0] = b[OPL.H0] = b[OPL.D0] = 1e12      # only GATHER is affordable
    p = OPL.plan_reference(rows, 64, "f32", stats, 512, 64, OPL.Options(beta=b))
    assert all(s.strat == OPL.GATHER for s in p.slices)
    assert p.sym_max == 0
    assert len(p.slices) < 200 * 64 // 4
    whole = [s for s in p.slices if s.k == 1]
    assert len(whole) >= 150
    assert len({s.wg for s in whole}) == 64          # every worker gets whole tables
    # each table is covered exactly once per bag
    for t in range(200):
        ks = {s.k for s in p.slices if s.t == t}
        assert len(ks) == 1
        assert sorted(s.j for s in p.slices if s.t == t) == list(range(ks.pop()))
    # at or below sym_max every gather table is split over all workers
    p2 = OPL.plan_reference(rows, 64, "f32", stats, 512, 64, OPL.Options(beta=b, sym_max=200))
    assert all(s.k == 64 for s in p2.slices)
    # a negative sym_max leaves every split to P4's cost rule (the LIF fallback, P7, could
    # still make trailing tables symmetric: switched off here)
    p3 = OPL.plan_reference(rows[:10], 64, "f32", stats[:10], 512, 64,
                            OPL.Options(beta=b, sym_max=-1, lif_milli=10 ** 9))
    assert all(s.k < 64 for s in p3.slices)



# ---- STREAM (the GM-UB flow: the table through LDS in chunks on one worker)

@pytest.mark.parametrize("m,R,lam", [(10000, 256, 5000.0), (3000, 512, 12.5), (70001, 128, 1e5)])
def test_stream_cost_is_the_chunk_costs_without_their_extra_item_costs(m, R, lam):
    """One worker scanning c chunks costs what c chunk items cost together, less the
    (c - 1) per-item costs the single item does not pay (up to 1 ps of flooring per term)."""
    b = OPL.default_beta(R)
    L = 131072
    crow = L // R
    c = (m + crow - 1) // crow
    chunks = sum(OPL.cost_chunk(b, ((i + 1) * m) // c - (i * m) // c, R, lam, c)[0] for i in range(c))
    stream, fixed = OPL.cost_stream(b, m, R, lam, c)
    assert abs(stream - (chunks - (c - 1) * b[OPL.L0])) <= c + 1
    assert fixed == math.floor(b[OPL.L0] + b[OPL.S] * float(m * R))


def _stream_beta():
    beta = list(OPL.default_beta(256))
    beta[OPL.S], beta[OPL.I], beta[OPL.L0] = 0.01, 1.0, 1000.0
    beta[OPL.G1] = beta[OPL.D1] = beta[OPL.P] = 1e6
    return beta


def test_stream_is_chosen_when_it_is_cheapest_and_never_past_64_chunks():
    R = 256
    crow = 131072 // R
    rows = [3 * crow, 64 * crow, 64 * crow + 1, 100]
    stats = [OPL.Stat(20.0)] * 4
    p = OPL.plan_reference(rows, 64, "f32", stats, 512, 64, OPL.Options(beta=_stream_beta()))
    strat = {}
    for ln in p.text().splitlines():
        if ln.startswith("item "):
            f = ln.split()
            strat.setdefault(int(f[2]), set()).add(int(f[3]))
    assert strat[0] == {OPL.STREAM} and strat[1] == {OPL.STREAM}
    assert OPL.STREAM not in strat[2]          # 65 chunks: not an automatic candidate
    assert strat[3] == {OPL.LDS}               # fits LDS: staging once beats scanning
    # forcing STREAM is allowed at any size; the plan then has no row chunks
    q = OPL.plan_reference(rows, 64, "f32", stats, 512, 64,
                           OPL.Options(beta=_stream_beta(), force=[OPL.STREAM] * 4))
    for ln in q.text().splitlines():
        if ln.startswith("item "):
            f = ln.split()
            assert int(f[3]) == OPL.STREAM and int(f[5]) == 1


def test_stream_cost_overflow_leaves_stream_out_instead_of_failing():
    # 6.5e6 lookups on a 60-chunk table: scanning them 60 times passes the cost cap while
    # gathering them does not; the plan still builds, without STREAM
    R = 256
    crow = 131072 // R
    b = OPL.default_beta(R)
    lam = 65536 * 100.0
    assert b[OPL.I] * lam * 60 > OPL.COST_CAP > b[OPL.G1] * lam
    p = OPL.plan_reference([60 * crow], 64, "f32", [OPL.Stat(100.0)], 65536, 256)
    assert all(int(ln.split()[3]) != OPL.STREAM for ln in p.text().splitlines() if ln.startswith("item "))


def test_many_gather_tables_split_over_all_workers_only_when_their_slices_are_large():
    """Past sym_max gather tables, a table is split over all workers only if each slice
    would hold at least 64 expected lookups; the small ones are placed by cost."""
    g = np.random.default_rng(4)
    T, B, K = 100, 4096, 256
    rows = [int(x) for x in np.exp(g.uniform(np.log(1e3), np.log(1e6), size=T))]
    pools = [8.0 if t % 2 == 0 else 1.0 for t in range(T)]   # shares 128 and 16 lookups
    stats = [OPL.Stat(s) for s in pools]
    p = OPL.plan_reference(rows, 64, "f32", stats, B, K)
    ks = {}
    for ln in p.text().splitlines():
        if ln.startswith("item "):
            f = ln.split()
            ks.setdefault(int(f[2]), set()).add(int(f[8]))
    for t in range(T):
        if t % 2 == 0:
            assert ks[t] == {K}, (t, ks[t])
        else:
            assert max(ks[t]) < K, (t, ks[t])
    # sym_max < 0 turns both rules off (a table may still reach K slices by its cost or
    # the LIF fallback, but fewer do); a large sym_max splits every table
    def n_full(plan):
        return len({int(ln.split()[2]) for ln in plan.text().splitlines()
                    if ln.startswith("item ") and int(ln.split()[8]) == K})
    q = OPL.plan_reference(rows, 64, "f32", stats, B, K, OPL.Options(sym_max=-1))
    assert n_full(q) < n_full(p) == T // 2
    r = OPL.plan_reference(rows, 64, "f32", stats, B, K, OPL.Options(sym_max=1000))
    assert all(int(ln.split()[8]) == K for ln in r.text().splitlines() if ln.startswith("item "))


# ---------------------------------------------------------------- pins by hand-worked plans

# A cost vector of exact binary values (ps): gather 1000 + 100 lam; LDS 2000 + S mu R + 10 lam
# with S = 1/8 ps per byte; chunk adds I = 50 per lookup scanned; HOT and DEDUP priced out.
WORKED_BETA = [0.0] * OPL.NBETA
WORKED_BETA[OPL.G0], WORKED_BETA[OPL.G1] = 1000.0, 100.0
WORKED_BETA[OPL.L0], WORKED_BETA[OPL.L1], WORKED_BETA[OPL.S], WORKED_BETA[OPL.I] = 2000.0, 10.0, 0.125, 50.0
WORKED_BETA[OPL.H0], WORKED_BETA[OPL.D0] = 1e9, 1e9
WORKED_ROWS = [100, 1000, 50, 10, 300, 20000]
WORKED_S = [2.0, 5.0, 8.0, 1.0, 8.0, 100.0]


def _worked(no_replication, lif_milli):
    stats = [OPL.Stat(s_, 1, [], 1.0) for s_ in WORKED_S]
    opts = OPL.Options(beta=WORKED_BETA, order_mode=1, lif_milli=lif_milli, no_replication=no_replication)
    return WORKED_ROWS, 64, "f32", stats, 10, 2, opts


def _items(text):
    return [ln for ln in text.splitlines() if ln.startswith("item ") or ln.startswith("end ")]


def test_literal_solver_worked_by_hand():
    """The paper's solver (Sec. III-B steps 1-4: no replication, order (s desc, m asc)) on six
    tables, K = 2 workers, B = 10, E = 64 fp32 (R = 256 B, L = 131072 B = 512 rows), with
    WORKED_BETA.  Worked by hand:

    Step 3 / P1, cost of each table at k = 1 (Lam = B s):
      t0 m 100  s 2   Lam 20:   gather 1000 + 2000 = 3000;  LDS 2000 + 3200 + 200 = 5400   -> GATHER 3000
      t1 m 1000 s 5   Lam 50:   gather 6000; does not fit L; step 1 would cut 2 chunks of 500
                                 rows at 2000 + 16000 + 2500 + 250 = 20750 each, 41500 > 6000 -> GATHER 6000
      t2 m 50   s 8   Lam 80:   gather 9000;  LDS 2000 + 1600 + 800 = 4400                  -> LDS 4400
      t3 m 10   s 1   Lam 10:   gather 2000;  LDS 2000 + 320 + 100 = 2420                   -> GATHER 2000
      t4 m 300  s 8   Lam 80:   gather 9000;  LDS 2000 + 9600 + 800 = 12400                 -> GATHER 9000
      t5 m 20000 s 100 Lam 1000: gather 101000; 40 chunks > K, STREAM 2,652,000             -> GATHER 101000
    Step 2, order (s desc, m asc, t): t5, t2, t4, t1, t0, t3; each to the least-loaded worker
    (ties to worker 0): t5 -> 0 (101000), then t2, t4, t1, t0, t3 -> 1 (24400).
    Step 4: LIF = floor(1000 * 2 * 101000 / 125400) = 1610: kept with threshold 2000.  With
    replication (P4) t5 would be split over both workers (Lam / 2 = 500 >= 64 lookups), and with
    the default threshold 1500 the fallback makes every table symmetric: last r tables of the
    order for r = 1..5 give LIF 1621, 1640, 1682, 1746, 1759; r = 6 gives 67000 per worker, 1000.
    """
    cases = {
        (True, 2000): ["item 0 5 3 0 1 0 20000 1 0 0 101000",
                       "item 1 2 0 0 1 0 50 1 0 0 4400",
                       "item 1 4 3 0 1 0 300 1 0 0 9000",
                       "item 1 1 3 0 1 0 1000 1 0 0 6000",
                       "item 1 0 3 0 1 0 100 1 0 0 3000",
                       "item 1 3 3 0 1 0 10 1 0 0 2000",
                       "end max 101000 sum 125400 lif 1610 sym 0"],
        (False, 2000): ["item 0 5 3 0 1 0 20000 2 0 0 51000",
                        "item 0 2 0 0 1 0 50 1 0 0 4400",
                        "item 0 1 3 0 1 0 1000 1 0 0 6000",
                        "item 0 3 3 0 1 0 10 1 0 0 2000",
                        "item 1 5 3 0 1 0 20000 2 1 0 51000",
                        "item 1 4 3 0 1 0 300 1 0 0 9000",
                        "item 1 0 3 0 1 0 100 1 0 0 3000",
                        "end max 63400 sum 126400 lif 1003 sym 0"],
        (True, 1500): ["item 0 5 3 0 1 0 20000 2 0 0 51000",
                       "item 0 2 0 0 1 0 50 2 0 0 4000",
                       "item 0 4 3 0 1 0 300 2 0 0 5000",
                       "item 0 1 3 0 1 0 1000 2 0 0 3500",
                       "item 0 0 3 0 1 0 100 2 0 0 2000",
                       "item 0 3 3 0 1 0 10 2 0 0 1500",
                       "item 1 5 3 0 1 0 20000 2 1 0 51000",
                       "item 1 2 0 0 1 0 50 2 1 0 4000",
                       "item 1 4 3 0 1 0 300 2 1 0 5000",
                       "item 1 1 3 0 1 0 1000 2 1 0 3500",
                       "item 1 0 3 0 1 0 100 2 1 0 2000",
                       "item 1 3 3 0 1 0 10 2 1 0 1500",
                       "end max 67000 sum 134000 lif 1000 sym 6"],
    }
    for (norepl, lif), want in cases.items():
        rows, E, dtype, stats, B, K, opts = _worked(norepl, lif)
        text = OPL.plan_reference(rows, E, dtype, stats, B, K, opts).text()
        assert _items(text) == want, (norepl, lif)
        assert ("norepl 1" in text.splitlines()[1]) == norepl
    # the built-in threshold is 1.5
    assert OPL.Options().lif_milli == 1500


@pytest.mark.parametrize("s,sym", [(63.0, False), (64.0, True), (65.0, True)])
def test_symmetric_split_needs_64_expected_lookups_per_slice(s, sym):
    """P4: an unchunked GATHER table is split over all min(K, B) workers exactly when each
    slice would hold at least 64 expected lookups.  Eight identical 1M-row tables (GATHER is
    their cheapest flow), K = B = 4, pooling s: Lam / 4 = s lookups per slice.  Every table
    costs at most tau = 2 x its cost, so without the rule nothing is split."""
    stats = [OPL.Stat(s, 100, [], 1.0)] * 8
    p = OPL.plan_reference([1_000_000] * 8, 64, "f32", stats, 4, 4)
    assert {sl.strat for sl in p.slices} == {OPL.GATHER}
    ks = {sl.k for sl in p.slices}
    assert ks == ({4} if sym else {1})
    assert len(p.slices) == (32 if sym else 8)


@pytest.mark.parametrize("m,stream", [(32768, True), (32769, False)])
def test_stream_is_a_candidate_up_to_64_chunks(m, stream):
    """P1: STREAM enters the automatic choice for tables of at most 64 chunks of floor(L / R)
    rows.  L = 131072, R = 256: 512 rows a chunk, so 32768 rows are 64 chunks and 32769 are
    65.  The cost vector makes STREAM far cheaper than a gather whenever it is allowed."""
    beta = [0.0] * OPL.NBETA
    beta[OPL.G1], beta[OPL.L1], beta[OPL.I], beta[OPL.D0] = 1e6, 1.0, 1.0, 1e10
    opts = OPL.Options(beta=beta, no_replication=True)
    p = OPL.plan_reference([m], 64, "f32", [OPL.Stat(1.0, 1, [], 1.0)], 16, 4, opts)
    strats = {sl.strat for sl in p.slices}
    assert strats == ({OPL.STREAM} if stream else {OPL.GATHER})


def _hot_worked(hot_freq, SH):
    """One table of 10^6 rows (beyond L: no LDS; 123 STREAM chunks: no STREAM), E = 4 fp32
    (R = 16 B), B = 64, pooling 1 (lam = 64 lookups), K = 1; gather 100 ps a lookup, LDS and
    DEDUP priced out, HOT = SH x C x R + lam (1 - h(C)) G1."""
    beta = [0.0] * OPL.NBETA
    beta[OPL.G1], beta[OPL.SH] = 100.0, SH
    beta[OPL.L0], beta[OPL.D0] = 1e9, 1e9
    stats = [OPL.Stat(1.0, 1, list(hot_freq), 1.0)]
    return [1_000_000], 4, "f32", stats, 64, 1, OPL.Options(beta=beta)


HOT_WORKED = {
    # hot_freq 2^-1 .. 2^-10: cap 10, candidates C = 1, 2, 4, 8, 10; cost 16 C + 6400 (1 - h(C)):
    #   3216, 1632, 464, 128 + 25 = 153, 160 + 6.25 = 166.25 -> C = 8, cost 153 (gather: 6400)
    "ten": ([2.0 ** -(i + 1) for i in range(10)], 1.0, 8, 153),
    # the first six of them: candidates 1, 2, 4, 6 -> 3216, 1632, 464, 96 + 100 = 196 -> C = 6 (the cap)
    "six": ([2.0 ** -(i + 1) for i in range(6)], 1.0, 6, 196),
    # nothing past the second row and no staging cost: h(2) = h(4) = h(5) = 0.75, cost 1600 for
    # each, against 3200 at C = 1 -> the tie goes to the smaller size, C = 2
    "tie": ([0.5, 0.25, 0.0, 0.0, 0.0], 0.0, 2, 1600),
}


@pytest.mark.parametrize("case", sorted(HOT_WORKED))
def test_hot_stages_the_cheapest_hot_set_worked_by_hand(case):
    """P1 prices HOT at each hot-set size C = 1, 2, 4, ... below the cap and at the cap, and
    stages the cheapest (ties to the smaller C), with h(C) the share of the first C listed
    rows; values worked by hand in HOT_WORKED."""
    freq, SH, C, cost = HOT_WORKED[case]
    p = OPL.plan_reference(*_hot_worked(freq, SH))
    assert [(sl.strat, sl.C, sl.cost) for sl in p.slices] == [(OPL.HOT, C, cost)]


def test_per_table_lookup_cost_worked_by_hand():
    """Two GATHER tables alike but for their fitted cost of a lookup served from memory:
    table 0 keeps beta's G1 (6,370 ps; given as 0), table 1 costs 4x (25,480 ps).
    E 64 fp32 (R 256), 1,000,000 rows each (no LDS, chunking needs 1,954 > K chunks, no
    hot rows, u = 1, STREAM past 64 chunks), B 64, s 2 (Lam 128), K 4, so k <= 4 and no
    symmetric split (128 / 4 = 32 < 64 lookups per slice).  By hand, G0 = 480,000:
      unsplit: t0 480,000 + 6,370 x 128 = 1,295,360;  t1 480,000 + 25,480 x 128 = 3,741,440
      tau = ceil(5,036,800 / 4) = 1,259,200, above 2 x G0 = 960,000, so k is the smallest
      split whose slice costs at most tau:
      t0: k = 2 gives 480,000 + 6,370 x 64 = 887,680 <= tau            -> k = 2
      t1: k = 2: 2,110,720; k = 3: 1,567,146; k = 4: 1,295,360, all > tau -> k = 4
      LPT: t1's four slices on workers 0-3, then t0's two on workers 0 and 1:
      max 1,295,360 + 887,680 = 2,183,040, sum 6,956,800, LIF floor(4000 x 2,183,040 /
      6,956,800) = 1,255.
    With one shared G1 both tables are split alike: tau = ceil(2,590,720 / 4) = 647,680,
    the bound max(tau, 2 x G0) = 960,000, and k = 2 (887,680) for each."""
    stats = [OPL.Stat(2.0, 2, [], 1.0)] * 2
    p = OPL.plan_reference([1_000_000] * 2, 64, "f32", stats, 64, 4, OPL.Options(gather_lookup_ps=[0.0, 25480.0]))
    ks = {(s.t, s.k, s.cost) for s in p.slices}
    assert ks == {(0, 2, 887_680), (1, 4, 1_295_360)}
    assert all(s.strat == OPL.GATHER for s in p.slices)
    assert sorted((s.wg, s.t) for s in p.slices) == [(0, 0), (0, 1), (1, 0), (1, 1), (2, 1), (3, 1)]
    assert (p.max_ps, p.sum_ps, p.lif_milli) == (2_183_040, 6_956_800, 1255)
    # 0 stands for beta's G1
    q = OPL.plan_reference([1_000_000] * 2, 64, "f32", stats, 64, 4, OPL.Options(gather_lookup_ps=[6370.0, 25480.0]))
    assert q.text() == p.text()
    shared = OPL.plan_reference([1_000_000] * 2, 64, "f32", stats, 64, 4, OPL.Options())
    assert {(s.t, s.k, s.cost) for s in shared.slices} == {(0, 2, 887_680), (1, 2, 887_680)}

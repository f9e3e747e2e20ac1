"""The C++ planner inside libembx against the planner oracle, byte for byte (host only)."""
import subprocess

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import workloads as W
from oracle import plan as OPL

from test_oracle_plan import _random_instance


def _lib():
    import paper_2507_01676_amd as embx
    return embx


def test_library_exports_every_declared_symbol():
    embx = _lib()
    import os
    import re
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    declared = []
    for h in ("embx.h", "embx_fill.h"):
        src = open(os.path.join(root, "include", h)).read()
        declared += re.findall(r"^(?:emb_status_t|const char\*)\s+(\w+)\(", src, flags=re.M)
    assert len(declared) >= 12
    out = subprocess.run(["nm", "-D", "--defined-only", embx.LIB_PATH], capture_output=True, text=True).stdout
    names = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    missing = [d for d in declared if d not in names]
    assert not missing, missing
    assert set(declared) == set(embx.EXPORTED)
    assert embx.status_string(embx.ERR_NOT_BOUND) == "weights not bound"


def test_builtin_coefficients_equal_the_oracles():
    """The library's built-in beta (emb_default_beta) is the oracle's, entry by entry,
    and the binding rejects a beta of the wrong length."""
    embx = _lib()
    for R in (16, 128, 256, 512, 1024):
        assert embx.default_beta(R) == OPL.default_beta(R)
    with pytest.raises(embx.EmbxError):
        embx.default_beta(0)
    with pytest.raises(ValueError):
        embx.plan_text([10], 4, "f32", [dict(mean_pooling=1.0, max_pooling=1, hot_rows=[], hot_freq=[],
                                              unique_frac=1.0)], 8, 2, beta=[1.0] * (embx.BETA_COUNT - 1))


def _cpp(rows, E, dtype, stats, B, K, opts: OPL.Options):
    embx = _lib()
    cst = [dict(mean_pooling=s.mean_pooling, max_pooling=s.max_pooling,
                hot_rows=list(range(len(s.hot_freq))), hot_freq=list(s.hot_freq), unique_frac=s.unique_frac)
           for s in stats]
    return embx.plan_text(rows, E, dtype, cst, B, K, lds_budget=opts.lds_budget, lif_milli=opts.lif_milli,
                          chunk_max_bytes=opts.chunk_max_bytes, order_mode=opts.order_mode, beta=opts.beta,
                          force=opts.force, sym_max=opts.sym_max, no_replication=opts.no_replication,
                          gather_lookup_ps=opts.gather_lookup_ps)


def _both(rows, E, dtype, stats, B, K, opts: OPL.Options):
    want = OPL.plan_reference(rows, E, dtype, stats, B, K, opts).text()
    return _cpp(rows, E, dtype, stats, B, K, opts), want


@pytest.mark.parametrize("seed", range(60))
def test_cpp_planner_equals_oracle_random(seed):
    rows, E, dtype, stats, B, K, opts = _random_instance(seed)
    got, want = _both(rows, E, dtype, stats, B, K, opts)
    assert got == want


@settings(max_examples=80, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(st.integers(0, 10 ** 7), st.sampled_from([None, "skewbeta", "force", "tableg1"]))
def test_cpp_planner_equals_oracle_hypothesis(seed, variant):
    rows, E, dtype, stats, B, K, opts = _random_instance(seed)
    g = np.random.default_rng(seed)
    if variant == "tableg1":   # per-table G1, some left to beta's (0)
        opts.gather_lookup_ps = [float(x) * float(g.integers(0, 2)) for x in g.uniform(1e3, 3e4, size=len(rows))]
    elif variant == "skewbeta":
        opts.beta = [float(x) for x in g.uniform(0.0, 5e4, size=OPL.NBETA)]
        opts.chunk_max_bytes = int(g.choice([0, 4096, 32768]))
    elif variant == "force":
        f = []
        for s in stats:
            choices = [OPL.AUTO, OPL.LDS, OPL.DEDUP, OPL.GATHER, OPL.STREAM] + ([OPL.HOT] if len(s.hot_freq) else [])
            f.append(int(g.choice(choices)))
        opts.force = f
    try:
        want = OPL.plan_reference(rows, E, dtype, stats, B, K, opts).text()
    except OPL.PlanError:
        embx = _lib()
        with pytest.raises(embx.EmbxError):
            _cpp(rows, E, dtype, stats, B, K, opts)
        return
    got, _ = _both(rows, E, dtype, stats, B, K, opts)
    assert got == want


@pytest.mark.parametrize("seed", range(40))
def test_cpp_planner_equals_oracle_with_per_table_lookup_costs(seed):
    rows, E, dtype, stats, B, K, opts = _random_instance(seed)
    g = np.random.default_rng(1000 + seed)
    opts.gather_lookup_ps = [float(x) for x in g.choice([0.0, 3000.0, 6370.0, 11000.0, 25000.0], size=len(rows))]
    got, want = _both(rows, E, dtype, stats, B, K, opts)
    assert got == want


def test_per_table_lookup_costs_are_validated():
    embx = _lib()
    st1 = [dict(mean_pooling=2.0, max_pooling=2, hot_rows=[], hot_freq=[], unique_frac=1.0)] * 2
    for bad in ([1.0], [1.0, -1.0], [1.0, float("nan")], [float("inf"), 1.0]):
        with pytest.raises(OPL.PlanError):
            OPL.plan_reference([100, 100], 64, "f32", [OPL.Stat(2.0, 2, [], 1.0)] * 2, 64, 4,
                               OPL.Options(gather_lookup_ps=bad))
        if len(bad) == 2:
            with pytest.raises(embx.EmbxError):
                embx.plan_text([100, 100], 64, "f32", st1, 64, 4, gather_lookup_ps=bad)
    with pytest.raises(ValueError):
        embx.plan_text([100, 100], 64, "f32", st1, 64, 4, gather_lookup_ps=[1.0])


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_cpp_planner_equals_oracle_on_workloads(cfg):
    c = W.make_config(cfg)
    st_ = W.history_stats(c)
    stats = [OPL.stats_from_workload(s) for s in st_]
    for K in (256, 97):
        got, want = _both(c.rows, c.E, c.dtype, stats, c.batch, K, OPL.Options())
        assert got == want
        assert want.count("\nitem ") >= K or K > 200


def test_cpp_planner_rejects_what_the_oracle_rejects():
    embx = _lib()
    bad = [
        ([0], 64, "f32", [OPL.Stat(1.0)]),
        ([10], 6, "f32", [OPL.Stat(1.0)]),
        ([10], 64, "f32", [OPL.Stat(float("nan"))]),
        ([10], 64, "f32", [OPL.Stat(-1.0)]),
    ]
    for rows, E, dt, stats in bad:
        with pytest.raises(OPL.PlanError):
            OPL.plan_reference(rows, E, dt, stats, 8, 4)
        with pytest.raises(embx.EmbxError):
            embx.plan_text(rows, E, dt, [dict(mean_pooling=x.mean_pooling) for x in stats], 8, 4)
    # a negative coefficient (here the HOT intercept) is refused by both
    beta = OPL.default_beta(256)
    beta[OPL.H0] = -1.0
    with pytest.raises(OPL.PlanError):
        OPL.plan_reference([10, 20], 64, "f32", [OPL.Stat(1.0)] * 2, 8, 4, OPL.Options(beta=beta))
    with pytest.raises(embx.EmbxError):
        embx.plan_text([10, 20], 64, "f32", [dict(mean_pooling=1.0)] * 2, 8, 4, beta=beta)


@pytest.mark.parametrize("T,sym_max", [(150, 0), (150, 200), (40, -1), (300, 64)])
def test_cpp_planner_equals_oracle_with_many_tables(T, sym_max):
    g = np.random.default_rng(T + sym_max)
    rows = [int(x) for x in np.exp(g.uniform(np.log(10), np.log(2e6), size=T))]
    stats = [OPL.Stat(float(g.choice([1.0, 1.0, 4.0, 20.0]))) for _ in range(T)]
    opts = OPL.Options(sym_max=sym_max)
    got, want = _both(rows, 64, "f32", stats, 1024, 128, opts)
    assert got == want
    assert f"symmax {sym_max}" in want


@pytest.mark.parametrize("seed", range(6))
def test_cpp_planner_equals_oracle_when_stream_is_cheapest(seed):
    """Coefficients that make the table scan win for mid-size tables: both planners
    choose STREAM for them and emit the same plan."""
    rows, E, dtype, stats, B, K, opts = _random_instance(1000 + seed)
    beta = list(OPL.default_beta(256))
    beta[OPL.S] = 0.01
    beta[OPL.I] = 1.0
    beta[OPL.L0] = 1000.0
    beta[OPL.G1] = 1e6
    beta[OPL.D1] = 1e6
    beta[OPL.P] = 1e6
    opts.beta = beta
    got, want = _both(rows, E, dtype, stats, B, K, opts)
    assert got == want


@pytest.mark.parametrize("seed", range(4))
def test_cpp_planner_equals_oracle_with_many_tables_of_mixed_shares(seed):
    g = np.random.default_rng(50 + seed)
    T = int(g.integers(65, 160))
    rows = [int(x) for x in np.exp(g.uniform(np.log(100), np.log(2e6), size=T))]
    stats = [OPL.Stat(float(g.choice([0.0, 1.0, 4.0, 20.0]))) for _ in range(T)]
    B = int(g.choice([1024, 4096, 16384]))
    for sym_max in (0, -1, 80):
        got, want = _both(rows, 64, "f32", stats, B, 256, OPL.Options(sym_max=sym_max))
        assert got == want


def test_cpp_planner_equals_oracle_on_the_pinned_instances():
    """The hand-worked literal-solver and hot-set plans and the boundary instances of the P4
    and STREAM rules, through the C++ planner."""
    from test_oracle_plan import _worked
    for norepl, lif in ((True, 2000), (False, 2000), (True, 1500)):
        got, want = _both(*_worked(norepl, lif))
        assert got == want
    for s in (63.0, 64.0, 65.0):
        got, want = _both([1_000_000] * 8, 64, "f32", [OPL.Stat(s, 100, [], 1.0)] * 8, 4, 4, OPL.Options())
        assert got == want
    beta = [0.0] * OPL.NBETA
    beta[OPL.G1], beta[OPL.L1], beta[OPL.I], beta[OPL.D0] = 1e6, 1.0, 1.0, 1e10
    for m in (32768, 32769):
        got, want = _both([m], 64, "f32", [OPL.Stat(1.0, 1, [], 1.0)], 16, 4,
                          OPL.Options(beta=beta, no_replication=True))
        assert got == want
    from test_oracle_plan import HOT_WORKED, _hot_worked
    for freq, SH, _, _ in HOT_WORKED.values():
        got, want = _both(*_hot_worked(freq, SH))
        assert got == want


def test_force_strategy_environment_variable(monkeypatch):
    """EMBX_FORCE_STRATEGY (a debugging switch) forces every table to one strategy, as the
    force_strategy option does; an unknown name is refused."""
    rows, E, dtype, stats, B, K, opts = _random_instance(3)
    embx = _lib()
    for name, code in (("gather", OPL.GATHER), ("dedup", OPL.DEDUP), ("stream", OPL.STREAM)):
        monkeypatch.setenv("EMBX_FORCE_STRATEGY", name)
        got = _cpp(rows, E, dtype, stats, B, K, opts)
        forced = OPL.Options(**{**opts.__dict__, "force": [code] * len(rows)})
        assert got == OPL.plan_reference(rows, E, dtype, stats, B, K, forced).text()
        assert {int(ln.split()[3]) for ln in got.splitlines() if ln.startswith("item ")} == {code}
    monkeypatch.setenv("EMBX_FORCE_STRATEGY", "fastest")
    with pytest.raises(embx.EmbxError):
        _cpp(rows, E, dtype, stats, B, K, opts)
    monkeypatch.setenv("EMBX_FORCE_STRATEGY", "")
    assert _cpp(rows, E, dtype, stats, B, K, opts) == OPL.plan_reference(rows, E, dtype, stats, B, K, opts).text()

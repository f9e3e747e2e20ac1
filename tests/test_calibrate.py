"""The cost-model fit (Eq. (2), OLS): samples priced by the planner oracle's cost
functions with a known beta are recovered by the fit, exactly without noise and
closely with it; the fit's forward model agrees with the oracle's."""
import numpy as np
import pytest

from oracle import plan as OPL
from paper_2507_01676_amd import calibrate as CAL

BETA_TRUE = [350_000.0, 9_000.0, 2_500_000.0, 900.0, 45.0, 300.0, 8_000_000.0, 1_200.0, 17_000_000.0, 28_000.0, 11.0]


def _samples(g, noise=0.0, n=400):
    b = BETA_TRUE
    s = CAL.Samples()
    for _ in range(n):
        lam = float(g.integers(1, 20000))
        R = int(g.choice([128, 256, 512]))
        kind = g.integers(0, 4)
        if kind == 0:
            mu = int(g.integers(1, 131072 // R))
            c = int(g.integers(1, 40)) if g.random() < 0.5 else 1
            if c > 1:
                y, _ = OPL.cost_chunk(b, mu, R, lam, float(c))
            else:
                y, _ = OPL.cost_lds(b, mu, R, lam)
            s.slices.append(CAL.SliceSample(CAL.LDS, lam, float(mu), R, c, ps=float(y)))
        elif kind == 1:
            C = int(g.integers(1, 512))
            h = float(g.random())
            y, _ = OPL.cost_hot(b, C, R, h, lam)
            s.slices.append(CAL.SliceSample(CAL.HOT, lam, float(C), R, 1, h=h, ps=float(y)))
        elif kind == 2:
            u = float(g.uniform(0.01, 1.0))
            y, _ = OPL.cost_dedup(b, u, lam)
            s.slices.append(CAL.SliceSample(CAL.DEDUP, lam, u=u, ps=float(y)))
        else:
            k = int(g.integers(1, 60))
            lams = g.integers(0, 5000, size=k).astype(float)
            y = sum(OPL.cost_gather(b, float(x))[0] for x in lams)
            s.workers.append(CAL.WorkerSample(k, float(lams.sum()), float(y)))
    if noise:
        for x in s.slices + s.workers:
            x.ps *= 1.0 + noise * g.standard_normal()
    return s


def test_noiseless_samples_recover_beta():
    s = _samples(np.random.default_rng(0))
    b = CAL.fit_beta(s)
    # the oracle floors each cost to whole picoseconds: recovery to that resolution
    for got, want in zip(b, BETA_TRUE):
        assert got == pytest.approx(want, rel=1e-5, abs=2.0)


def test_noisy_samples_recover_beta_closely():
    s = _samples(np.random.default_rng(1), noise=0.003, n=4000)
    b = CAL.fit_beta(s)
    for i, (got, want) in enumerate(zip(b, BETA_TRUE)):
        assert got == pytest.approx(want, rel=0.15), i


def test_forward_model_matches_the_planner_oracle():
    g = np.random.default_rng(2)
    s = _samples(g, n=300)
    for x in s.slices + s.workers:
        assert CAL.predict(BETA_TRUE, x) == pytest.approx(x.ps, abs=60.0)


def test_unsampled_strategies_keep_the_base_value():
    g = np.random.default_rng(3)
    s = _samples(g)
    s.slices = [x for x in s.slices if x.strat != CAL.DEDUP]
    base = [float(i) for i in range(CAL.NBETA)]
    b = CAL.fit_beta(s, base)
    assert b[CAL.D0] == 8.0 and b[CAL.D1] == 9.0
    assert b[CAL.G1] == pytest.approx(BETA_TRUE[CAL.G1], rel=1e-5)


def test_a_dropped_term_is_caught():
    """Planted mistake: a fit that ignores the staged-bytes term misses the data."""
    g = np.random.default_rng(4)
    s = _samples(g)
    lds = [x for x in s.slices if x.strat == CAL.LDS]
    A = np.array([[1.0, x.lam / x.c, x.lam if x.c > 1 else 0.0] for x in lds])
    y = np.array([x.ps for x in lds])
    v, *_ = np.linalg.lstsq(A, y, rcond=None)
    resid = np.abs(A @ v - y).max()
    assert resid > 1e5


@pytest.mark.parametrize("seed", range(6))
def test_relative_residuals_keep_the_fixed_cost_of_short_slices(seed):
    """Mostly long HOT slices whose times scatter by 30% (contention) and a few short ones
    (5%) that are nearly all fixed cost: with residuals relative to each slice's predicted
    time the fit recovers H0, what a short slice costs; unweighted, the long slices'
    scatter sets the intercept (off by more than the weighted fit in most seeds)."""
    g = np.random.default_rng(seed)
    b = list(BETA_TRUE)
    b[CAL.H0] = 2e6
    s = CAL.Samples()
    for i in range(600):
        short = i % 10 == 0
        lam = float(g.integers(1, 8)) if short else float(g.integers(2000, 20000))
        C = int(g.integers(1, 4)) if short else int(g.integers(256, 512))
        h = float(g.random())
        y, _ = OPL.cost_hot(b, C, 256, h, lam)
        noise = 0.05 if short else 0.3
        s.slices.append(CAL.SliceSample(CAL.HOT, lam, float(C), 256, 1, h=h, ps=float(y) * (1.0 + noise * g.standard_normal())))
    got = CAL.fit_beta(s, b)
    assert got[CAL.H0] == pytest.approx(b[CAL.H0], rel=0.05)


def test_unweighted_fit_misses_the_fixed_cost():
    """Planted mistake: the same samples fitted without the reweighting miss H0 by more
    than 25% in at least half of the seeds above."""
    misses = 0
    for seed in range(6):
        g = np.random.default_rng(seed)
        b = list(BETA_TRUE)
        b[CAL.H0] = 2e6
        rows, ys = [], []
        for i in range(600):
            short = i % 10 == 0
            lam = float(g.integers(1, 8)) if short else float(g.integers(2000, 20000))
            C = int(g.integers(1, 4)) if short else int(g.integers(256, 512))
            h = float(g.random())
            y, _ = OPL.cost_hot(b, C, 256, h, lam)
            noise = 0.05 if short else 0.3
            ps = float(y) * (1.0 + noise * g.standard_normal())
            rows.append([1.0, C * 256.0, lam])
            ys.append(ps - lam * (h * b[CAL.L1] + (1.0 - h) * b[CAL.G1]))
        x = CAL._lstsq(np.array(rows), np.array(ys))
        misses += abs(x[0] - b[CAL.H0]) > 0.25 * b[CAL.H0]
    assert misses >= 3


def test_samples_csv_round_trip_keeps_each_group(tmp_path):
    """write_samples_csv / read_samples_csv: every field survives (8 significant digits),
    and the cap takes at most max_rows of each group (workers, whole LDS, LDS chunks,
    HOT, DEDUP)."""
    s = _samples(np.random.default_rng(11), n=600)
    p = tmp_path / "s.csv"
    CAL.write_samples_csv(s, str(p), max_rows=1000)
    r = CAL.read_samples_csv(str(p))
    assert len(r.workers) == len(s.workers) and len(r.slices) == len(s.slices)
    key = lambda x: (x.strat, x.lam, x.mu, x.c, x.ps)   # noqa: E731
    for a, b in zip(sorted(s.slices, key=key), sorted(r.slices, key=key)):
        for f in ("strat", "R", "c"):
            assert getattr(a, f) == getattr(b, f)
        for f in ("lam", "mu", "h", "u", "ps"):
            assert getattr(b, f) == pytest.approx(getattr(a, f), rel=1e-7, abs=1e-12)
    for a, b in zip(sorted(s.workers, key=lambda x: (x.lam, x.ps)), sorted(r.workers, key=lambda x: (x.lam, x.ps))):
        assert a.n_slices == b.n_slices and b.ps == pytest.approx(a.ps, rel=1e-7)
    # the fit of what was read equals the fit of what was written, to the rounding
    for x, y in zip(CAL.fit_beta(s), CAL.fit_beta(r)):
        assert y == pytest.approx(x, rel=1e-5, abs=1e-3)
    CAL.write_samples_csv(s, str(p), max_rows=7)
    r = CAL.read_samples_csv(str(p))
    assert len(r.workers) == 7
    groups = [[x for x in r.slices if x.strat == CAL.LDS and x.c == 1],
              [x for x in r.slices if x.strat == CAL.LDS and x.c > 1],
              [x for x in r.slices if x.strat == CAL.HOT], [x for x in r.slices if x.strat == CAL.DEDUP]]
    assert [len(g) for g in groups] == [7, 7, 7, 7]


def test_committed_samples_read_back_as_written():
    import os
    here = os.path.dirname(os.path.abspath(__file__))
    r = CAL.read_samples_csv(os.path.join(here, "golden", "calibration_samples.csv"))
    assert len(r.workers) == 250 and len(r.slices) == 1000
    assert {x.strat for x in r.slices} == {CAL.LDS, CAL.HOT, CAL.DEDUP}


def test_table_lookup_costs_recovered_from_noiseless_workers():
    """Workers' gather phases made from a known shared latency c, G0 per slice and a cost
    per lookup for each table (one table unused): the fit returns each used table's cost
    and 0 for the unused one."""
    from paper_2507_01676_amd.calibrate import fit_table_lookup_costs
    g = np.random.default_rng(7)
    T, K = 6, 200
    g1 = np.array([5200.0, 6400.0, 10800.0, 0.0, 7300.0, 25000.0])
    lam = np.zeros((K, T))
    n = np.zeros(K, dtype=np.int64)
    for w in range(K):
        for t in g.choice([0, 1, 2, 4, 5], size=int(g.integers(1, 3)), replace=False):
            lam[w, t] += float(g.integers(50, 2000))
            n[w] += 1
    c, g0 = 2.5e6, 480_000.0
    ps = c + g0 * n + lam @ g1
    got = fit_table_lookup_costs(ps, n, lam, g0)
    assert got[3] == 0.0
    for t in (0, 1, 2, 4, 5):
        assert abs(got[t] - g1[t]) <= 1e-6 * g1[t], (t, got[t])


def test_table_lookup_costs_without_enough_workers_fall_back():
    """No gather lookups, or fewer workers than unknowns: every table keeps the vector's G1
    (0), rather than an underdetermined fit."""
    from paper_2507_01676_amd.calibrate import fit_table_lookup_costs
    assert fit_table_lookup_costs(np.zeros(0), np.zeros(0), np.zeros((0, 3)), 480_000.0) == [0.0] * 3
    lam = np.array([[100.0, 0.0, 50.0]])
    assert fit_table_lookup_costs(np.array([2e6]), np.array([2]), lam, 480_000.0) == [0.0] * 3

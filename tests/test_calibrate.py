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

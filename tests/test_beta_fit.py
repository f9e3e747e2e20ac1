"""The planner's built-in cost coefficients are the least-squares fit of the committed
calibration samples (Eq. (2); the fit of Sec. III-A), each rounded to three significant
digits.  The fit is written out here with numpy.linalg.lstsq, stage by stage, independently
of the library's calibration module:

  GATHER  per worker:   ps = G0 n_slices + G1 lam
  LDS     whole table:  ps = L0 + S mu R + L1 lam
  LDS     row chunk:    ps - (L0 + S mu R + L1 lam / c) = I lam
  HOT:                  ps - lam (h L1 + (1 - h) G1) = H0 + SH mu R + P lam
  DEDUP:                ps - G1 u lam = D0 + D1 lam

each stage on what the earlier ones leave, and each solved twice: plainly, then with every
row divided by the sample's time as the first solution predicts it (at least 1 us), so that
residuals count relative to the slice's length.
"""
import math
import os

import numpy as np

from oracle import plan as OPL

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLES = os.path.join(HERE, "golden", "calibration_samples.csv")


def _read():
    rows = []
    head = None
    with open(SAMPLES) as f:
        for ln in f:
            if ln.startswith("#") or not ln.strip():
                continue
            v = ln.strip().split(",")
            if head is None:
                head = v
                continue
            d = dict(zip(head, v))
            rows.append({k: (d[k] if k == "kind" else float(d[k])) for k in head})
    return rows


def _solve(A, y, offset):
    x0 = np.linalg.lstsq(A, y, rcond=None)[0]
    w = 1.0 / np.maximum(A @ x0 + offset, 1e6)
    return np.linalg.lstsq(A * w[:, None], y * w, rcond=None)[0]


def _fit(rows):
    wk = [r for r in rows if r["kind"] == "worker"]
    sl = [r for r in rows if r["kind"] == "slice"]
    whole = [r for r in sl if r["strat"] == OPL.LDS and r["c"] == 1]
    chunk = [r for r in sl if r["strat"] == OPL.LDS and r["c"] > 1]
    hot = [r for r in sl if r["strat"] == OPL.HOT]
    dd = [r for r in sl if r["strat"] == OPL.DEDUP]
    arr = lambda rs, f: np.array([f(r) for r in rs], dtype=np.float64)   # noqa: E731
    b = {}
    A = np.stack([arr(wk, lambda r: r["n_slices"]), arr(wk, lambda r: r["lam"])], axis=1)
    b["G0"], b["G1"] = _solve(A, arr(wk, lambda r: r["ps"]), np.zeros(len(wk)))
    A = np.stack([np.ones(len(whole)), arr(whole, lambda r: r["mu"] * r["R"]), arr(whole, lambda r: r["lam"])], axis=1)
    b["L0"], b["S"], b["L1"] = _solve(A, arr(whole, lambda r: r["ps"]), np.zeros(len(whole)))
    off = arr(chunk, lambda r: b["L0"] + b["S"] * r["mu"] * r["R"] + b["L1"] * r["lam"] / r["c"])
    (b["I"],) = _solve(arr(chunk, lambda r: r["lam"])[:, None], arr(chunk, lambda r: r["ps"]) - off, off)
    off = arr(hot, lambda r: r["lam"] * (r["h"] * b["L1"] + (1.0 - r["h"]) * b["G1"]))
    A = np.stack([np.ones(len(hot)), arr(hot, lambda r: r["mu"] * r["R"]), arr(hot, lambda r: r["lam"])], axis=1)
    b["H0"], b["SH"], b["P"] = _solve(A, arr(hot, lambda r: r["ps"]) - off, off)
    off = arr(dd, lambda r: b["G1"] * r["u"] * r["lam"])
    A = np.stack([np.ones(len(dd)), arr(dd, lambda r: r["lam"])], axis=1)
    b["D0"], b["D1"] = _solve(A, arr(dd, lambda r: r["ps"]) - off, off)
    return b


def _round3(x):
    if x == 0.0:
        return 0.0
    e = math.floor(math.log10(abs(x))) - 2
    return float(f"{round(x / 10.0 ** e) * 10.0 ** e:.6g}")


NAMES = ["G0", "G1", "L0", "L1", "S", "I", "H0", "P", "D0", "D1", "SH"]


def test_builtin_coefficients_are_the_fit_of_the_committed_samples():
    rows = _read()
    assert len([r for r in rows if r["kind"] == "worker"]) >= 100
    for st in (OPL.LDS, OPL.HOT, OPL.DEDUP):
        assert len([r for r in rows if r["kind"] == "slice" and r["strat"] == st]) >= 100
    b = _fit(rows)
    assert all(v > 0.0 for v in b.values()), b    # no coefficient needed a non-negativity bound
    want = OPL.default_beta(256)
    got = [_round3(b[n]) for n in NAMES]
    assert got == [want[getattr(OPL, n)] for n in NAMES], (got, want)


def test_the_fit_reproduces_the_samples():
    """The fitted model explains the samples it came from: the median relative error per
    group stays within what the timers' run-to-run scatter allows."""
    rows = _read()
    b = OPL.default_beta(256)
    G0, G1, L0, L1, S, I, H0, P, D0, D1, SH = b

    def pred(r):
        if r["kind"] == "worker":
            return G0 * r["n_slices"] + G1 * r["lam"]
        if r["strat"] == OPL.LDS:
            extra = I * r["lam"] if r["c"] > 1 else 0.0
            return L0 + S * r["mu"] * r["R"] + extra + L1 * r["lam"] / r["c"]
        if r["strat"] == OPL.HOT:
            return H0 + SH * r["mu"] * r["R"] + r["lam"] * (P + r["h"] * L1 + (1.0 - r["h"]) * G1)
        return D0 + D1 * r["lam"] + G1 * r["u"] * r["lam"]

    for grp in ("worker", OPL.LDS, OPL.HOT, OPL.DEDUP):
        rs = [r for r in rows if (r["kind"] == "worker" if grp == "worker" else
                                  (r["kind"] == "slice" and r["strat"] == grp))]
        rel = np.array([abs(pred(r) - r["ps"]) / max(r["ps"], 1e6) for r in rs])
        assert np.median(rel) < 0.25, (grp, float(np.median(rel)))

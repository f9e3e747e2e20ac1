"""Host logic of the batch-size sweep: the Pareto front keeps exactly the points that no
other point beats on both throughput (higher) and P99 (lower)."""
import itertools

import numpy as np

from paper_2507_01676_amd.pareto import p99, pareto_front


def _pt(t, l):
    return {"lookups_per_s": float(t), "p99_us": float(l)}


def test_front_of_a_small_example():
    pts = [_pt(1, 1), _pt(2, 2), _pt(3, 3), _pt(2, 3), _pt(1, 2), _pt(3, 3)]
    front = pareto_front(pts)
    assert [(p["lookups_per_s"], p["p99_us"]) for p in front] == [(1, 1), (2, 2), (3, 3), (3, 3)]


def test_front_matches_brute_force():
    g = np.random.default_rng(3)
    for _ in range(50):
        pts = [_pt(*g.integers(0, 6, size=2)) for _ in range(int(g.integers(1, 9)))]
        front = pareto_front(pts)
        for p in pts:
            dom = any(q["lookups_per_s"] >= p["lookups_per_s"] and q["p99_us"] <= p["p99_us"] and q != p
                      for q in pts)
            assert (p in front) == (not dom) or any(q == p for q in pts if q is not p)


def test_p99_is_nearest_rank():
    xs = list(range(1, 101))
    assert p99(xs) == 99
    assert p99([5.0]) == 5.0
    assert p99(list(range(1, 1001))) == 990


def _table1():
    """The paper's Table I (Sec. IV-A) from tests/golden: (distribution, strategy, workload,
    P99 us, queries/s, bold) per reported cell; bold when either value is printed in bold."""
    import csv
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "table1_p99_tps_batch8192.csv")
    with open(path) as f:
        rows = list(csv.DictReader(line for line in f if not line.startswith("#")))
    out = []
    for r in rows:
        if r["p99_us"] == "--":
            continue
        bold = r["p99_us"].endswith("*") or r["tps"].endswith("*")
        tps = r["tps"].rstrip("*")
        scale = {"k": 1e3, "M": 1e6}.get(tps[-1], 1.0)
        tps = float(tps[:-1] if tps[-1] in "kM" else tps) * scale
        out.append((r["distribution"], r["strategy"], r["workload"], float(r["p99_us"].rstrip("*")), tps, bold))
    return out


def test_the_papers_best_entries_are_on_the_front():
    """Table I prints each workload's best P99 and best throughput in bold. A point best
    in either coordinate is dominated by none, so every bold cell of a (distribution,
    workload) column is on that column's front."""
    cells = _table1()
    assert len(cells) == 51
    cols = {}
    for d, s, w, lat, tps, bold in cells:
        cols.setdefault((d, w), []).append(dict(lookups_per_s=tps, p99_us=lat, strategy=s, bold=bold))
    n_bold = 0
    for key, pts in cols.items():
        front = pareto_front(pts)
        for p in pts:
            if p["bold"]:
                n_bold += 1
                assert p in front, (key, p["strategy"])
        # and the front is what the definition keeps
        for p in pts:
            dominated = any(q is not p and q["lookups_per_s"] >= p["lookups_per_s"] and q["p99_us"] <= p["p99_us"]
                            and (q["lookups_per_s"] > p["lookups_per_s"] or q["p99_us"] < p["p99_us"]) for q in pts)
            assert (p in front) == (not dominated), (key, p["strategy"])
    assert n_bold == 19          # 6 uniform, 6 real, 7 fixed


def test_a_front_that_keeps_dominated_points_is_caught():
    """Planted mistake: comparing throughput the wrong way keeps a dominated cell."""
    cells = _table1()
    pts = [dict(lookups_per_s=t, p99_us=l, strategy=s) for d, s, w, l, t, b in cells
           if d == "uniform" and w == "Criteo-1TB"]

    def wrong_front(points):
        return [p for p in points if not any(q["lookups_per_s"] <= p["lookups_per_s"] and q["p99_us"] <= p["p99_us"]
                                             and q is not p for q in points)]
    assert [p["strategy"] for p in pareto_front(pts)] == ["symmetric"]
    assert [p["strategy"] for p in wrong_front(pts)] != ["symmetric"]

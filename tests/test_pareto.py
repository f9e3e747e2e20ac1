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

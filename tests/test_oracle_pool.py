"""Pins of the pooling oracle against things other than itself.

* brute force: dense count matrices A_t[b, r] (how often row r occurs in bag
  (t, b)) times the table, in float64;
* a library routine: torch.nn.functional.embedding_bag(mode="sum") on the CPU
  in float64;
* the pure-Python loop definition;
* invariants: empty bags, integer-encoded tables that decode back to the index,
  literal one-hot tables, linearity, permutation within a bag, duplicates.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import index as OI
from oracle import pool as OP


def _rand_case(seed, T=3, B=5, E=8, maxpf=4, dtype=np.float32, allow_empty=True):
    g = np.random.default_rng(seed)
    rows = [int(g.integers(1, 30)) for _ in range(T)]
    weights = [g.standard_normal((m, E)).astype(dtype) for m in rows]
    bags = []
    for t in range(T):
        for b in range(B):
            n = int(g.integers(0 if allow_empty else 1, maxpf + 1))
            bags.append([int(x) for x in g.integers(0, rows[t], size=n)])
    bt = W.batch_from_bags(T, B, bags)
    return weights, bt, rows


def _dense_counts(bt, rows, T, B):
    A = [np.zeros((B, rows[t]), dtype=np.float64) for t in range(T)]
    for t in range(T):
        for b in range(B):
            for k in range(bt.offsets[t * B + b], bt.offsets[t * B + b + 1]):
                A[t][b, bt.indices[k]] += 1.0
    return A


@pytest.mark.parametrize("seed", range(6))
def test_matches_dense_count_matrix(seed):
    T, B = 3, 6
    weights, bt, rows = _rand_case(seed, T=T, B=B)
    ref, mag, bad = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    assert bad == 0 and ref.shape == (B, T, 8) and ref.dtype == np.float32
    A = _dense_counts(bt, rows, T, B)
    for t in range(T):
        want = A[t] @ weights[t].astype(np.float64)
        wmag = A[t] @ np.abs(weights[t].astype(np.float64))
        assert np.allclose(ref[:, t, :], want, rtol=1e-6, atol=1e-6)
        assert np.allclose(mag[:, t, :], wmag, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_matches_torch_embedding_bag(seed):
    T, B = 4, 7
    weights, bt, rows = _rand_case(100 + seed, T=T, B=B, maxpf=6)
    ref, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    for t in range(T):
        lo = int(bt.offsets[t * B])
        idx = torch.from_numpy(bt.indices[lo: bt.offsets[t * B + B]].copy())
        off = torch.from_numpy((bt.offsets[t * B: t * B + B] - lo).copy())
        w = torch.from_numpy(weights[t].astype(np.float64))
        got = torch.nn.functional.embedding_bag(idx, w, off, mode="sum").numpy()
        assert np.allclose(ref[:, t, :], got, rtol=1e-6, atol=1e-6)


def test_matches_python_loops_with_fp16_and_bad_indices():
    T, B = 2, 4
    weights, bt, rows = _rand_case(7, T=T, B=B, E=16, dtype=np.float16)
    bt.indices[1] = -1                       # out of range: skipped and counted
    bt.indices[-1] = rows[1] + 3
    ref, mag, bad = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    loops, bad2 = OP.pool_loops(weights, bt.indices, bt.offsets, B)
    assert bad == bad2 == OI.range_errors(bt.indices, bt.offsets, rows, B)
    assert bad >= 1
    assert np.array_equal(ref, np.array(loops, dtype=np.float64).astype(np.float32))


def test_empty_bags_are_positive_zero():
    T, B = 2, 3
    weights = [np.full((4, 8), -1.5, np.float32), np.full((3, 8), -2.0, np.float32)]
    bt = W.batch_from_bags(T, B, [[0, 1], [], [3], [], [2, 2], []])
    ref, mag, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    empty = OP.empty_bag_mask(bt.offsets, T, B)
    assert empty.sum() == 3
    assert np.all(ref[empty] == 0) and not np.any(np.signbit(ref[empty]))
    assert np.all(ref[0, 0] == -3.0) and np.all(ref[2, 0] == -1.5) and np.all(ref[1, 1] == -4.0)


def test_integer_tables_decode_the_index():
    # "one-hot" style pin: with pooling factor 1, the integer-encoded columns
    # return the looked-up row id and the table id exactly
    c = W.make_config(1)
    B = 50
    bt = W.gen_batch(c, 0, B=B)
    weights = [W.table_rows_block(t, 0, c.rows[t], c.E, "f32", seed=11, mode=W.VAL_INTEGER) for t in range(c.T)]
    ref, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    for t in range(c.T):
        idx = bt.indices[bt.offsets[t * B]: bt.offsets[t * B + B]]
        dec = ref[:, t, 1].astype(np.int64) + (ref[:, t, 2].astype(np.int64) << 11) + (ref[:, t, 3].astype(np.int64) << 22)
        assert np.array_equal(dec, idx)
        assert np.all(ref[:, t, 0] == 1) and np.all(ref[:, t, 4] == t + 1)


def test_literal_one_hot_table_gives_histogram():
    E = 32
    Wt = np.eye(E, dtype=np.float32)
    g = np.random.default_rng(3)
    bags = [[int(x) for x in g.integers(0, E, size=int(g.integers(0, 9)))] for _ in range(10)]
    bt = W.batch_from_bags(1, 10, bags)
    ref, _, _ = OP.pool_reference([Wt], bt.indices, bt.offsets, 10)
    for b, bag in enumerate(bags):
        assert np.array_equal(ref[b, 0], np.bincount(np.array(bag, dtype=np.int64), minlength=E).astype(np.float32))


def test_linearity_permutation_duplicates():
    T, B = 3, 5
    w1, bt, rows = _rand_case(21, T=T, B=B)
    g = np.random.default_rng(5)
    w2 = [g.standard_normal(w.shape).astype(np.float32) for w in w1]
    r1, _, _ = OP.pool_reference(w1, bt.indices, bt.offsets, B)
    r2, _, _ = OP.pool_reference(w2, bt.indices, bt.offsets, B)
    r12, _, _ = OP.pool_reference([a.astype(np.float64) + b for a, b in zip(w1, w2)], bt.indices, bt.offsets, B)
    assert np.allclose(r12, r1.astype(np.float64) + r2, rtol=1e-5, atol=1e-5)
    # integer tables: any order inside a bag gives the same bits
    wi = [W.table_rows_block(t, 0, rows[t], 8, "f32", seed=3, mode=W.VAL_INTEGER) for t in range(T)]
    perm = bt.indices.copy()
    for t in range(T):
        for b in range(B):
            lo, hi = bt.offsets[t * B + b], bt.offsets[t * B + b + 1]
            perm[lo:hi] = perm[lo:hi][::-1]
    a, _, _ = OP.pool_reference(wi, bt.indices, bt.offsets, B)
    p, _, _ = OP.pool_reference(wi, perm, bt.offsets, B)
    assert np.array_equal(a, p)
    # k copies of one row -> k * row
    wd = W.table_rows_block(0, 0, 5, 8, "f32", seed=3, mode=W.VAL_INTEGER)
    bt2 = W.batch_from_bags(1, 1, [[2] * 7])
    d, _, _ = OP.pool_reference([wd], bt2.indices, bt2.offsets, 1)
    assert np.array_equal(d[0, 0], 7 * wd[2])


def test_error_metric():
    ref = np.array([1.0, -1.0, 0.0], np.float32)
    mag = np.array([2.0, 3.0, 0.0])
    assert OP.pooled_error(ref, ref, mag) == 0.0
    assert OP.pooled_error(np.array([1.0, -1.0, 1e-3], np.float32), ref, mag) == np.inf
    assert OP.pooled_error(np.array([1.5, -1.0, 0.0], np.float32), ref, mag) == pytest.approx(0.25)


@pytest.mark.parametrize("mistake", ["drop_last", "shift", "transpose"])
def test_planted_mistakes_are_caught(mistake):
    """A plausible slip in the oracle (planted here, on the CPU) fails the brute-force pin."""
    T, B = 3, 6
    weights, bt, rows = _rand_case(77, T=T, B=B, allow_empty=False)
    ref, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    bad = ref.copy()
    if mistake == "drop_last":
        for t in range(T):
            for b in range(B):
                k = bt.offsets[t * B + b + 1] - 1
                bad[b, t] -= weights[t][bt.indices[k]]
    elif mistake == "shift":
        bad = np.roll(bad, 1, axis=0)
    else:
        bad = np.ascontiguousarray(bad.transpose(1, 0, 2)).reshape(B, T, -1)
    A = _dense_counts(bt, rows, T, B)
    want = np.stack([A[t] @ weights[t].astype(np.float64) for t in range(T)], axis=1)
    assert np.allclose(ref, want, rtol=1e-6, atol=1e-6)
    assert not np.allclose(bad, want, rtol=1e-6, atol=1e-6)


# ---- mean pooling and per-lookup weights (Sec. II-B: sum or average)

def _psw(seed, n):
    return np.random.default_rng(seed).uniform(-2.0, 2.0, size=n).astype(np.float32)


def _dense_weighted(bt, rows, T, B, psw):
    """A_t[b, r] = sum of the weights of the lookups of row r in bag (t, b); n[t][b] = bag length."""
    A = [np.zeros((B, rows[t]), dtype=np.float64) for t in range(T)]
    n = np.zeros((T, B), dtype=np.int64)
    for t in range(T):
        for b in range(B):
            lo, hi = bt.offsets[t * B + b], bt.offsets[t * B + b + 1]
            n[t, b] = hi - lo
            for k in range(lo, hi):
                A[t][b, bt.indices[k]] += 1.0 if psw is None else float(psw[k])
    return A, n


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("weighted", [False, True])
def test_mean_and_weights_match_dense_matrices(seed, weighted):
    T, B = 3, 6
    weights, bt, rows = _rand_case(300 + seed, T=T, B=B)
    psw = _psw(seed, bt.indices.size) if weighted else None
    pooling = ["mean", "sum", "mean"]
    ref, mag, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, pooling=pooling, psw=psw)
    A, n = _dense_weighted(bt, rows, T, B, psw)
    for t in range(T):
        want = A[t] @ weights[t].astype(np.float64)
        wmag = np.abs(A[t]) @ np.abs(weights[t].astype(np.float64)) if not weighted else None
        if pooling[t] == "mean":
            want = want / np.maximum(n[t], 1)[:, None]
        assert np.allclose(ref[:, t, :], want, rtol=1e-6, atol=1e-6)
        if wmag is not None:
            wmag = wmag / (np.maximum(n[t], 1)[:, None] if pooling[t] == "mean" else 1)
            assert np.allclose(mag[:, t, :], wmag, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_mean_and_weights_match_torch_embedding_bag(seed):
    T, B = 3, 7
    weights, bt, rows = _rand_case(400 + seed, T=T, B=B, maxpf=6)
    psw = _psw(10 + seed, bt.indices.size)
    mean, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, pooling="mean")
    wsum, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, psw=psw)
    for t in range(T):
        lo = int(bt.offsets[t * B])
        hi = int(bt.offsets[t * B + B])
        idx = torch.from_numpy(bt.indices[lo:hi].copy())
        off = torch.from_numpy((bt.offsets[t * B: t * B + B] - lo).copy())
        w = torch.from_numpy(weights[t].astype(np.float64))
        got_mean = torch.nn.functional.embedding_bag(idx, w, off, mode="mean").numpy()
        got_w = torch.nn.functional.embedding_bag(idx, w, off, mode="sum",
                                                  per_sample_weights=torch.from_numpy(psw[lo:hi].astype(np.float64))).numpy()
        assert np.allclose(mean[:, t, :], got_mean, rtol=1e-6, atol=1e-6)
        assert np.allclose(wsum[:, t, :], got_w, rtol=1e-6, atol=1e-6)


def test_mean_and_weights_match_python_loops_with_fp16_and_bad_indices():
    T, B = 2, 5
    weights, bt, rows = _rand_case(17, T=T, B=B, E=16, dtype=np.float16)
    bt.indices[0] = -4
    bt.indices[-1] = rows[1]
    psw = _psw(3, bt.indices.size)
    for pooling in ("sum", "mean", ["mean", "sum"]):
        ref, _, bad = OP.pool_reference(weights, bt.indices, bt.offsets, B, pooling=pooling, psw=psw)
        loops, bad2 = OP.pool_loops(weights, bt.indices, bt.offsets, B, pooling=pooling, psw=psw)
        assert bad == bad2 >= 1
        assert np.array_equal(ref, np.array(loops, dtype=np.float64).astype(np.float32))


def test_mean_and_weight_invariants():
    T, B = 3, 6
    weights, bt, rows = _rand_case(500, T=T, B=B)
    s, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B)
    # unit weights change nothing; weight 2 doubles every sum exactly (a power of two)
    ones = np.ones(bt.indices.size, np.float32)
    s1, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, psw=ones)
    s2, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, psw=2 * ones)
    assert np.array_equal(s1, s) and np.array_equal(s2, 2 * s)
    # weights are linear: w1 + w2 gives the sum of the two weighted sums
    a, b = _psw(1, bt.indices.size), _psw(2, bt.indices.size)
    ra, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, psw=a)
    rb, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, psw=b)
    rab, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, psw=a.astype(np.float64) + b)
    assert np.allclose(rab, ra.astype(np.float64) + rb, rtol=1e-5, atol=1e-5)
    # a bag of k copies of one row averages to that row, bit for bit; empty bags stay +0.0
    wd = W.table_rows_block(0, 0, 5, 8, "f32", seed=3, mode=W.VAL_INTEGER)
    bt2 = W.batch_from_bags(1, 3, [[4] * 6, [], [1, 3]])
    m, _, _ = OP.pool_reference([wd], bt2.indices, bt2.offsets, 3, pooling="mean")
    assert np.array_equal(m[0, 0], wd[4])
    assert np.all(m[1, 0] == 0) and not np.any(np.signbit(m[1, 0]))
    assert np.array_equal(m[2, 0], ((wd[1].astype(np.float64) + wd[3]) / 2).astype(np.float32))
    # one-hot table under mean pooling: the bag's histogram over its length
    E = 16
    bags = [[1, 1, 5], [0], [15, 2, 2, 2]]
    bt3 = W.batch_from_bags(1, 3, bags)
    h, _, _ = OP.pool_reference([np.eye(E, dtype=np.float32)], bt3.indices, bt3.offsets, 3, pooling="mean")
    for b, bag in enumerate(bags):
        want = np.bincount(np.array(bag), minlength=E) / len(bag)
        assert np.array_equal(h[b, 0], want.astype(np.float32))
    # an out-of-range id adds nothing but still counts in the mean's divisor
    bt4 = W.batch_from_bags(1, 1, [[2, 99]])
    q, _, bad = OP.pool_reference([wd], bt4.indices, bt4.offsets, 1, pooling="mean")
    assert bad == 1 and np.array_equal(q[0, 0], (wd[2].astype(np.float64) / 2).astype(np.float32))


@pytest.mark.parametrize("mistake", ["divide_by_n_plus_1", "ignore_weights", "weights_of_next_lookup",
                                     "mean_before_weights_sum"])
def test_planted_mistakes_in_mean_and_weights_are_caught(mistake):
    """A plausible slip (planted here, on the CPU) fails the dense-matrix pin."""
    T, B = 3, 6
    weights, bt, rows = _rand_case(88, T=T, B=B, allow_empty=False)
    psw = _psw(8, bt.indices.size)
    A, n = _dense_weighted(bt, rows, T, B, psw)
    want = np.stack([(A[t] @ weights[t].astype(np.float64)) / n[t][:, None] for t in range(T)], axis=1)
    ref, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, pooling="mean", psw=psw)
    assert np.allclose(ref, want, rtol=1e-6, atol=1e-6)
    if mistake == "divide_by_n_plus_1":
        bad = ref * (n.T / (n.T + 1))[:, :, None]
    elif mistake == "ignore_weights":
        bad, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, pooling="mean")
    elif mistake == "weights_of_next_lookup":
        bad, _, _ = OP.pool_reference(weights, bt.indices, bt.offsets, B, pooling="mean", psw=np.roll(psw, 1))
    else:   # the mean of the weights times the mean of the rows
        bad = np.zeros_like(ref)
        for t in range(T):
            for b in range(B):
                lo, hi = bt.offsets[t * B + b], bt.offsets[t * B + b + 1]
                bad[b, t] = psw[lo:hi].mean() * weights[t][bt.indices[lo:hi]].astype(np.float64).mean(axis=0)
    assert not np.allclose(bad, want, rtol=1e-6, atol=1e-6)

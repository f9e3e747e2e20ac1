"""Pins of the index-handling oracle (brute force on tiny inputs, invariants)."""
import numpy as np
import pytest

import workloads as W
from oracle import index as OI
from oracle import pool as OP


def test_chunk_local_masks_and_partitions():
    g = np.random.default_rng(0)
    m, c = 103, 4
    bounds = [((i * m) // c, ((i + 1) * m) // c) for i in range(c)]
    assert OI.chunk_partition_ok(m, bounds)
    assert not OI.chunk_partition_ok(m, [(0, 50), (51, 103)])
    idx = g.integers(0, m, size=500)
    hits = np.zeros(idx.size, np.int64)
    for r0, r1 in bounds:
        loc = OI.chunk_local(idx, r0, r1)
        inside = loc >= 0
        hits += inside
        assert np.all(loc[inside] + r0 == idx[inside]) and np.all(loc[inside] < r1 - r0)
    assert np.all(hits == 1)            # every index pooled by exactly one chunk


def test_chunked_pooling_equals_whole_table():
    """Reading of the chunk offset step: masked (not clipped) indices make the sum of the
    per-chunk pools equal the whole-table pool."""
    g = np.random.default_rng(1)
    m, E, B, c = 57, 8, 9, 3
    Wt = W.table_rows_block(0, 0, m, E, "f32", seed=4, mode=W.VAL_INTEGER)
    bags = [[int(x) for x in g.integers(0, m, size=int(g.integers(0, 6)))] for _ in range(B)]
    bt = W.batch_from_bags(1, B, bags)
    full, _, _ = OP.pool_reference([Wt], bt.indices, bt.offsets, B)
    acc = np.zeros_like(full)
    for i in range(c):
        r0, r1 = (i * m) // c, ((i + 1) * m) // c
        loc = OI.chunk_local(bt.indices, r0, r1)
        keep = loc >= 0
        # pool the chunk-local table with out-of-chunk entries dropped
        lens = np.diff(bt.offsets)
        newoff = np.zeros(B + 1, np.int64)
        np.cumsum([int(keep[bt.offsets[b]:bt.offsets[b + 1]].sum()) for b in range(B)], out=newoff[1:])
        part, _, _ = OP.pool_reference([Wt[r0:r1]], loc[keep], newoff, B)
        acc += part
    assert np.array_equal(acc, full)
    # literal clipping would have double counted the boundary rows
    clip_total = sum(np.clip(bt.indices - (i * m) // c, 0, ((i + 1) * m) // c - (i * m) // c - 1).size for i in range(c))
    assert clip_total == c * bt.indices.size > bt.indices.size


def test_hot_slots_brute_force():
    g = np.random.default_rng(2)
    hot = np.array([17, 3, 99, 42, 5], dtype=np.int64)
    idx = g.integers(0, 120, size=1000)
    got = OI.hot_slots(idx, hot)
    pos = {int(r): i for i, r in enumerate(hot)}
    want = np.array([pos.get(int(x), -1) for x in idx])
    assert np.array_equal(got, want)
    assert np.all(OI.hot_slots(idx, np.zeros(0, np.int64)) == -1)


@pytest.mark.parametrize("seed", range(3))
def test_dedup_tile_brute_force(seed):
    g = np.random.default_rng(seed)
    idx = W.zipf_ranks(g, 300, 1.2, 2048)
    u, inv, cnt = OI.dedup_tile(idx)
    assert np.all(np.diff(u) > 0)
    assert np.array_equal(u[inv], idx)
    assert cnt.sum() == idx.size
    assert sorted(set(int(x) for x in idx)) == [int(x) for x in u]
    for k in range(u.size):
        assert cnt[k] == int((idx == u[k]).sum())


def test_range_errors_brute_force():
    bt = W.batch_from_bags(2, 2, [[0, 5], [-1], [2], [3, 3, 7]])
    assert OI.range_errors(bt.indices, bt.offsets, [5, 4], 2) == 3

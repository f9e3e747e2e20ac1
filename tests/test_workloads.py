"""The seeded input generators (shared inputs of oracle and GPU path)."""
import math

import numpy as np
import pytest

import workloads as W


def test_splitmix64_published_outputs():
    # First three outputs of SplitMix64 started from state 0 (state += golden gamma,
    # output = mix(state)), as published with the generator (Steele et al. 2014 /
    # Vigna's reference splitmix64.c).
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    got = [W.splitmix64_mix_scalar(k * W.GOLDEN) for k in (1, 2, 3)]
    assert got == want
    z = np.array([W.GOLDEN, 2 * W.GOLDEN & W.M64, 3 * W.GOLDEN & W.M64], dtype=np.uint64)
    assert [int(v) for v in W._mix_inplace(z)] == want


def test_value_generator_matches_scalar_definition():
    seed, t, lo, hi = 0x1234567890ABCDEF, 3, -0.05, 0.05
    blk = W.table_rows_block(t, 5, 9, 24, "f32", seed=seed, lo=lo, hi=hi)
    for r in range(5, 9):
        for c in range(24):
            key = (t << 40) | (r << 8) | c
            x = W.splitmix64_mix_scalar(key + seed * W.GOLDEN)
            u = x >> 40
            v = np.float32(lo + (hi - lo) * ((u + 0.5) * 2.0 ** -24))
            assert blk[r - 5, c] == v
    h = W.table_rows_block(t, 5, 9, 24, "f16", seed=seed, lo=lo, hi=hi)
    assert h.dtype == np.float16
    assert np.array_equal(h, blk.astype(np.float16))
    assert np.all(blk >= lo) and np.all(blk <= hi)


def test_integer_tables_are_exact_small_integers():
    blk = W.table_rows_block(7, 0, 5000, 64, "f32", seed=99, mode=W.VAL_INTEGER)
    assert np.all(blk == np.round(blk)) and blk.min() >= 0 and blk.max() <= 2047
    r = np.arange(5000)
    assert np.all(blk[:, 0] == 1)
    dec = blk[:, 1].astype(np.int64) + (blk[:, 2].astype(np.int64) << 11) + (blk[:, 3].astype(np.int64) << 22)
    assert np.array_equal(dec, r)
    assert np.all(blk[:, 4] == 8)
    h = W.table_rows_block(7, 0, 5000, 64, "f16", seed=99, mode=W.VAL_INTEGER)
    assert np.array_equal(h.astype(np.float32), blk)


def test_materialize_matches_blocks():
    a = W.materialize_table(2, 70000, 16, "f32", seed=5, threads=4)
    b = W.table_rows_block(2, 0, 70000, 16, "f32", seed=5)
    assert np.array_equal(a, b)


def test_configs_shapes():
    c1 = W.make_config(1)
    assert c1.rows == [100, 1000, 10000, 100000] and c1.E == 32 and c1.batch == 128
    s = W.cfg2_sizes()
    assert s[:10] == [10, 17, 28, 47, 79, 132, 221, 370, 620, 1039]
    assert s[-1] == 4_000_000 and len(s) == 26
    c3 = W.make_config(3)
    assert c3.dtype == "f16" and c3.E == 128 and all(0.8 <= tb.alpha <= 1.2 for tb in c3.tables)
    c4 = W.make_config(4)
    assert c4.rows[0] == 10_000_000 and all(1000 <= m <= 1_000_000 for m in c4.rows[1:])
    assert c4.tables[0].pf_value == 50 and all(tb.pf_value == 1 for tb in c4.tables[1:])
    c5 = W.make_config(5)
    assert c5.T == 100 and sum(c5.rows) * 512 <= 150 * 10 ** 9
    assert all(1000 <= m <= 20_000_000 for m in c5.rows)


def test_batch_determinism_and_csr():
    c = W.make_config(3)
    b1 = W.gen_batch(c, 0, B=64)
    b2 = W.gen_batch(c, 0, B=64)
    assert np.array_equal(b1.indices, b2.indices) and np.array_equal(b1.offsets, b2.offsets)
    lens = np.diff(b1.offsets)
    assert lens.min() >= 1 and lens.max() <= 20 and b1.offsets[0] == 0
    assert b1.offsets[-1] == b1.indices.size
    for t in range(c.T):
        x = b1.indices[b1.offsets[t * 64]: b1.offsets[t * 64 + 64]]
        assert x.min() >= 0 and x.max() < c.rows[t]
    b3 = W.gen_batch(c, 1, B=64)
    assert not np.array_equal(b1.indices, b3.indices)


def test_zipf_goodness_of_fit():
    g = np.random.default_rng(1)
    m, alpha, n = 50, 1.05, 200000
    r = W.zipf_ranks(g, m, alpha, n)
    p = np.arange(1, m + 1, dtype=np.float64) ** -alpha
    p /= p.sum()
    obs = np.bincount(r, minlength=m)
    chi2 = float(((obs - n * p) ** 2 / (n * p)).sum())
    # chi-square with 49 dof: the 99.9% quantile is ~85.4
    assert chi2 < 85.4, chi2
    # alpha below one works too (numpy's own zipf cannot do this)
    r2 = W.zipf_ranks(g, 1000, 0.8, 10000)
    assert r2.min() >= 0 and r2.max() < 1000


def test_stats_from_indices():
    idx = np.array([5, 3, 5, 7, 3, 5, 9], dtype=np.int64)
    pf = np.array([3, 4])
    st = W.stats_from_indices(idx, pf, 20, n_hot=3)
    assert list(st.hot_rows) == [5, 3, 7]
    assert np.allclose(st.hot_freq, [3 / 7, 2 / 7, 1 / 7])
    assert st.unique_frac == pytest.approx(4 / 7) and st.mean_pooling == 3.5


def test_cfg4_skew_matches_zipf_1_5():
    # top row of a Zipf(1.5) table of 1e7 rows takes 1/zeta(1.5) ~ 38% of lookups
    c = W.make_config(4)
    pf, idx = W.gen_table_batch(c, 0, 0, B=512)
    assert pf.sum() == 512 * 50
    _, cnt = np.unique(idx, return_counts=True)
    top = cnt.max() / idx.size
    assert abs(top - 1.0 / 2.612375348685488) < 0.02


def test_query_distributions():
    """The three query distributions of the paper's experiments (Sec. IV-A): the
    workload's own, uniform, and fixed (every lookup of a table on one row)."""
    c = W.make_config(2)
    assert W.with_distribution(c, "config") is c
    with pytest.raises(ValueError):
        W.with_distribution(c, "zipf")
    f = W.with_distribution(c, "fixed")
    assert f.rows == c.rows and f.E == c.E and f.value_seeds == c.value_seeds and f.batch == c.batch
    b0, b1, b = W.gen_batch(f, 0), W.gen_batch(f, 1), W.gen_batch(c, 0)
    assert np.array_equal(b0.offsets, b.offsets)                # pooling factors unchanged
    for t in range(f.T):
        ids = b0.indices[b0.offsets[t * f.batch]:b0.offsets[(t + 1) * f.batch]]
        assert ids.size > 0 and np.all(ids == ids[0]) and 0 <= ids[0] < f.rows[t]
        assert ids[0] == W.fixed_row(2, t, f.rows[t])
    assert np.array_equal(b0.indices, b1.indices)               # the same row in every batch
    st = W.history_stats(f)
    for t in range(f.T):                                        # statistics see the one row
        assert st[t].hot_freq[0] == 1.0 and st[t].hot_rows[0] == W.fixed_row(2, t, f.rows[t])
        assert st[t].unique_frac == 1.0 / W.make_config(2).batch
    u = W.with_distribution(c, "uniform")
    bu = W.gen_batch(u, 0)
    t = c.T - 1                                                 # 4M rows: a uniform draw spreads out
    ids = bu.indices[bu.offsets[t * c.batch]:bu.offsets[(t + 1) * c.batch]]
    assert np.unique(ids).size > 0.99 * ids.size
    assert abs(ids.mean() / c.rows[t] - 0.5) < 0.05

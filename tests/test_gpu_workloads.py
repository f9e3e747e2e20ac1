"""Parity at the five workloads' full sizes, with the plan and launch the benchmark uses.

The smallest workload is checked on every output element; the others on
sampled bags whose rows the oracle regenerates on the host, plus properties
that hold at any size (empty bags, integer-table exactness).
"""
import gc

import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, check_sampled, filled_tables, host_tables, log, plan_for, to_device, upload_tables

pytestmark = pytest.mark.gpu


def _free():
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def _lookup(c, batch, weights, stats=None):
    import torch
    p = plan_for(c, c.batch, stats=stats)
    p.bind(weights)
    idx, off = to_device(batch)
    out = p.lookup(idx, off, batch.B)
    torch.cuda.synchronize()
    assert p.check_errors() == 0
    info = p.info()
    log(f"  plan: {info['n_strategy']} lif={info['lif_milli']} lds={info['lds_bytes']}")
    res = out.cpu().numpy()
    del out, idx, off
    return res


def test_workload1_full():
    log("workload 1 (4 tables, E32 fp32, B128): every element")
    c = W.make_config(1)
    hw = host_tables(c)
    batch = W.gen_batch(c, 0)
    got = _lookup(c, batch, upload_tables(hw))
    err, _ = check_full(got, hw, batch, c.dtype)
    log(f"  pooled error {err:.2e}")
    hi = host_tables(c, W.VAL_INTEGER)
    got = _lookup(c, batch, upload_tables(hi))
    check_full(got, hi, batch, c.dtype, exact=True)


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_workload_full_size_sampled(cfg):
    log(f"workload {cfg}: full size, sampled bags")
    c = W.make_config(cfg)
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    wd = filled_tables(c)
    got = _lookup(c, batch, wd, stats)
    err = check_sampled(c, got, batch, 4000, seed=cfg)
    log(f"  worst pooled error on 4000 bags {err:.2e}")
    # integer-valued tables: sampled bags bit-exact
    wi = filled_tables(c, W.VAL_INTEGER)
    del wd
    _free()
    got = _lookup(c, batch, wi, stats)
    check_sampled(c, got, batch, 4000, seed=100 + cfg, mode=W.VAL_INTEGER, exact=True)
    del wi
    _free()


@pytest.mark.parametrize("cfg,dist", [(1, "fixed"), (2, "fixed"), (2, "uniform"), (4, "fixed")])
def test_workload_query_distributions(cfg, dist):
    """The workloads under the paper's other query distributions (Sec. IV-A): uniform,
    and fixed (every lookup of a table on one row, the paper's stress test for
    same-line conflicts), planned from statistics of that distribution, at full size."""
    log(f"workload {cfg}, {dist} queries: full size")
    c = W.with_distribution(W.make_config(cfg), dist)
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    if cfg == 1:
        hw = host_tables(c)
        got = _lookup(c, batch, upload_tables(hw), stats)
        check_full(got, hw, batch, c.dtype)
        hi = host_tables(c, W.VAL_INTEGER)
        got = _lookup(c, batch, upload_tables(hi), stats)
        check_full(got, hi, batch, c.dtype, exact=True)
        return
    wd = filled_tables(c)
    got = _lookup(c, batch, wd, stats)
    err = check_sampled(c, got, batch, 4000, seed=200 + cfg)
    log(f"  worst pooled error on 4000 bags {err:.2e}")
    wi = filled_tables(c, W.VAL_INTEGER)
    del wd
    _free()
    got = _lookup(c, batch, wi, stats)
    check_sampled(c, got, batch, 4000, seed=300 + cfg, mode=W.VAL_INTEGER, exact=True)
    del wi
    _free()


@pytest.mark.parametrize("cfg", [3, 4])
def test_workload_full_size_sampled_weighted_and_mean(cfg):
    """Weighted lookups with mean and sum tables alternating, at full size, with the
    plan and launch bench.py uses for --weighted --pooling."""
    import torch
    log(f"workload {cfg}: full size, weighted, mean/sum tables, sampled bags")
    c = W.make_config(cfg)
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    wd = filled_tables(c)
    pooling = ["mean" if t % 2 == 0 else "sum" for t in range(c.T)]
    psw = np.random.default_rng(1000).uniform(0.5, 1.5, size=batch.indices.size).astype(np.float32)
    p = plan_for(c, c.batch, stats=stats, pooling=pooling)
    p.bind(wd)
    idx, off = to_device(batch)
    out = p.lookup(idx, off, batch.B, weights=torch.from_numpy(psw).cuda())
    torch.cuda.synchronize()
    assert p.check_errors() == 0
    got = out.cpu().numpy()
    del out, idx, off
    err = check_sampled(c, got, batch, 4000, seed=200 + cfg, pooling=pooling, psw=psw)
    log(f"  worst pooled error on 4000 bags {err:.2e}")
    del wd
    _free()


def test_workload5_full_size_sampled():
    import torch
    log("workload 5 (100 tables <= 150 GB, E128 fp32, B65536): full size, sampled bags")
    c = W.make_config(5)
    log(f"  table bytes {sum(c.rows) * c.row_bytes / 1e9:.1f} GB {c.note}")
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    wd = filled_tables(c)
    torch.cuda.synchronize()
    got = _lookup(c, batch, wd, stats)
    err = check_sampled(c, got, batch, 3000, seed=5)
    log(f"  worst pooled error on 3000 bags {err:.2e}")
    del wd, got
    _free()

"""Parity at the five workloads' full sizes, with the plan and launch the benchmark uses.

Workloads 1-4 are checked on every output element (tables built on the host and
uploaded); workload 5 (132.7 GB of tables) on every bag in the columns that follow from the
indices alone (integer tables) and on sampled bags whose rows the oracle regenerates
on the host, bit-exact on integer tables.  The batch-size sweep's plans
are checked at two of its batch sizes, and workloads 2 and 4 also with two batches in
flight (bench.py --streams 2).
"""
import gc

import numpy as np
import pytest

import workloads as W

from gpu_helpers import (check_full, check_index_columns, check_sampled, filled_tables, host_tables, log, plan_for,
                         to_device, upload_tables)

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
def test_workload_full_size_every_element(cfg):
    """Workloads 2-4 at full size with the plan bench.py uses: every output element against
    the oracle (tables built on the host by the generator and uploaded), uniform values to
    the tolerance and integer values bit for bit."""
    log(f"workload {cfg}: full size, every element")
    c = W.make_config(cfg)
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    for mode in (W.VAL_UNIFORM, W.VAL_INTEGER):
        hw = host_tables(c, mode)
        log(f"  tables built on the host ({sum(w.nbytes for w in hw) / 1e9:.2f} GB, mode {mode})")
        wd = upload_tables(hw)
        got = _lookup(c, batch, wd, stats)
        del wd
        _free()
        err, _ = check_full(got, hw, batch, c.dtype, exact=mode == W.VAL_INTEGER)
        log(f"  {batch.B * c.T * c.E} elements checked, pooled error {err:.2e}")
        del hw, got
        gc.collect()


@pytest.mark.parametrize("cfg", [2, 4])
def test_workload_two_batches_in_flight_every_element(cfg):
    """The launch configuration of bench.py --streams 2 at full size: four batches dealt to
    two streams, a plan each over the same integer tables, each into its own output; every
    element of every batch bit for bit against the oracle."""
    import torch
    log(f"workload {cfg}: full size, two batches in flight, every element")
    c = W.make_config(cfg)
    stats = W.history_stats(c)
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    plans = [plan_for(c, c.batch, stats=stats).bind(wd) for _ in range(2)]
    batches = [W.gen_batch(c, i) for i in range(4)]
    dev = [to_device(b) for b in batches]
    outs = [torch.full((c.batch, c.T, c.E), float("nan"), device="cuda") for _ in range(4)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for i in range(4):
        plans[i % 2].lookup(*dev[i], c.batch, outs[i], stream=streams[i % 2])
    torch.cuda.synchronize()
    assert all(p.check_errors() == 0 for p in plans)
    for i in range(4):
        check_full(outs[i].cpu().numpy(), hw, batches[i], c.dtype, exact=True)
    log(f"  {4 * c.batch * c.T * c.E} elements checked")
    del plans, wd, outs, dev
    _free()


@pytest.mark.parametrize("cfg,dist", [(1, "fixed"), (2, "fixed"), (2, "uniform"), (3, "fixed"), (3, "uniform"),
                                      (4, "fixed"), (4, "uniform")])
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
    """Workload 5 at full size (132.7 GB of tables, 131M lookups) with the plan bench.py uses:
    uniform tables to the tolerance on 3000 sampled bags; integer tables bit-exact on 20000
    sampled bags, and on every bag in columns 0-4 (functions of the row id alone); then weighted lookups with mean and sum tables alternating on the same
    integer tables, to the tolerance on 4000 sampled bags."""
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
    wi = filled_tables(c, W.VAL_INTEGER)
    torch.cuda.synchronize()
    got = _lookup(c, batch, wi, stats)
    check_sampled(c, got, batch, 20000, seed=55, mode=W.VAL_INTEGER, exact=True)
    log("  integer tables: 20000 sampled bags bit-exact")
    check_index_columns(got, batch, c.T)
    log(f"  integer tables: every bag ({batch.B * c.T}), columns 0-4 (count, row digits, table) bit-exact")
    del got
    pooling = ["mean" if t % 2 == 0 else "sum" for t in range(c.T)]
    psw = np.random.default_rng(1005).uniform(0.5, 1.5, size=batch.indices.size).astype(np.float32)
    p = plan_for(c, c.batch, stats=stats, pooling=pooling)
    p.bind(wi)
    idx, off = to_device(batch)
    out = p.lookup(idx, off, batch.B, weights=torch.from_numpy(psw).cuda())
    torch.cuda.synchronize()
    assert p.check_errors() == 0
    got = out.cpu().numpy()
    del out, idx, off
    err = check_sampled(c, got, batch, 4000, seed=56, mode=W.VAL_INTEGER, pooling=pooling, psw=psw)
    log(f"  weighted, mean/sum tables: worst pooled error on 4000 bags {err:.2e}")
    del wi, got
    _free()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_batch_sweep_plans_match_the_oracle(cfg):
    """The batch-size sweep's own plans (made for 1/16 and 1/2 of the workload's batch):
    the output of the plan each point times is checked on sampled bags (every bag for
    workload 1), uniform tables to the tolerance."""
    from paper_2507_01676_amd import pareto

    seen = []

    def verify(cw, batch, out):
        got = out.cpu().numpy()
        n = batch.B * cw.T if cfg == 1 else 3000
        err = check_sampled(cw, got, batch, n, seed=700 + batch.B)
        log(f"  workload {cfg} batch {batch.B}: worst pooled error {err:.2e}")
        seen.append(batch.B)

    pts = pareto.sweep(cfg, fractions=(1 / 16, 1 / 2), steps=5, warmup=2, n_p99=5, n_batches=2,
                       log=lambda m: log("  " + m), verify=verify, streams=(1, 2))
    full = W.make_config(cfg).batch
    assert seen == [max(1, round(full / 16)), max(1, round(full / 2))]
    assert [p["streams"] for p in pts] == [1, 2, 1, 2]
    assert all(p["lookups_per_s"] > 0 for p in pts)

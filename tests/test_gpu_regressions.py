"""GPU regression tests of host-side launch preparation, each against the oracle:

- a runtime batch below the plan's max batch can put one more bag in a batch slice than the
  max batch does (slice j of k is bags [floor(jB/k), floor((j+1)B/k))): every bag must still
  be walked and written;
- a table whose statistics leave the maximum pooling unknown (0) is summed like any other,
  not treated as single-lookup bags;
- a plan launched with nearly all of a workgroup's LDS keeps working after smaller plans
  and the dedup probe have been created and run;
- workers that hold both single-lookup bags and summed bags (the second queue's first
  chunks are rotated past the wavefronts busy with single-lookup chunks) walk every bag once.
"""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, to_device, upload_tables
from test_gpu_parity import STRATS

pytestmark = pytest.mark.gpu


def fixed_pf_config(cfg_id, rows, pfs, E=64, dtype="f32", B=1000):
    tabs = [W.TableSpec(m, "fixed", pf, pf, pf, "uniform") for m, pf in zip(rows, pfs)]
    c = W.Config(cfg_id, f"fixed pooling {pfs}", E, dtype, -1.0, 1.0, B, tabs)
    c.value_seeds = [W.value_seed(cfg_id, t) for t in range(c.T)]
    return c


# runtime batches below 1000 for which some slice of k = 256 (or 4, 64) holds one bag more
# than at 1000, plus edge sizes
RUNTIME_BATCHES = [792, 999, 1000, 513, 257, 256, 255, 100, 7, 1]


@pytest.mark.parametrize("pfs", [[20] * 10, [3] * 10, [1] * 10, [20, 3, 1, 50, 8, 1, 2, 20, 1, 5]])
def test_runtime_batch_below_max_batch_writes_every_bag(pfs):
    import torch
    log(f"max batch 1000, runtime batches {RUNTIME_BATCHES}, pooling {pfs}")
    c = fixed_pf_config(140, [100_000] * 10, pfs)
    hw = host_tables(c, W.VAL_INTEGER)
    p = plan_for(c, 1000).bind(upload_tables(hw))
    log(f"  gather runs per queue {p.info()['gather_runs']}")
    for B in RUNTIME_BATCHES:
        batch = W.gen_batch(c, B, B=B)
        idx, off = to_device(batch)
        out = torch.full((B, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, B, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert not np.isnan(got).any(), f"batch {B}: {int(np.isnan(got).any(axis=2).sum())} bags never written"
        check_full(got, hw, batch, c.dtype, exact=True)
    assert p.check_errors() == 0


def test_runtime_batch_below_max_batch_mean_pooling():
    import torch
    log("mean pooling, max batch 1000, runtime batch 792 (a slice of 256 gains a bag)")
    c = fixed_pf_config(141, [100_000] * 10, [20] * 10)
    hw = host_tables(c)
    p = plan_for(c, 1000, pooling="mean").bind(upload_tables(hw))
    from oracle import pool as OP
    for B in (792, 1000, 333):
        batch = W.gen_batch(c, B, B=B)
        idx, off = to_device(batch)
        out = torch.full((B, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, B, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert not np.isnan(got).any()
        ref, mag, _ = OP.pool_reference(hw, batch.indices, batch.offsets, B, pooling="mean")
        assert OP.pooled_error(got, ref, mag) <= 1e-5


def test_unknown_max_pooling_is_summed_not_single():
    import torch
    log("pooling-8 table with max_pooling 0 (unknown) and a pooling-1 table with max_pooling 1")
    c = fixed_pf_config(142, [50_000, 50_000], [8, 1], B=512)
    stats = W.history_stats(c)
    stats[0].max_pooling = 0
    hw = host_tables(c, W.VAL_INTEGER)
    p = plan_for(c, c.batch, stats=stats).bind(upload_tables(hw))
    runs = p.info()["gather_runs"]
    log(f"  gather runs per queue {runs}")
    # the pooling-1 table promises one lookup per bag (single queue); the other does not
    text = p.serialize()
    t1_slices = sum(1 for ln in text.splitlines() if ln.startswith("item ") and ln.split()[2] == "1")
    assert runs["single"] == t1_slices > 0
    assert runs["sw"] + runs["wave"] > 0
    batch = W.gen_batch(c, 0)
    idx, off = to_device(batch)
    out = torch.full((c.batch, c.T, c.E), float("nan"), device="cuda")
    p.lookup(idx, off, c.batch, out)
    torch.cuda.synchronize()
    check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=True)
    # every table unknown: no single-lookup queue at all, results unchanged
    for s in stats:
        s.max_pooling = 0
    p0 = plan_for(c, c.batch, stats=stats).bind(upload_tables(hw))
    assert p0.info()["gather_runs"]["single"] == 0
    out0 = p0.lookup(idx, off, c.batch)
    torch.cuda.synchronize()
    check_full(out0.cpu().numpy(), hw, batch, c.dtype, exact=True)


def test_large_lds_plan_after_smaller_plans_and_probe():
    import torch

    import paper_2507_01676_amd as embx
    log("a plan using ~159 KiB of LDS, then a small plan and the dedup probe, then the first plan")
    c = fixed_pf_config(143, [260, 5000, 40_000, 100_000], [4, 3, 2, 6], E=128, B=257)
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    big = plan_for(c, c.batch, force=[STRATS["lds"]] * c.T, lds_budget=133_888).bind(wd)
    assert big.info()["lds_bytes"] > 160_000
    small = plan_for(c, c.batch, force=[STRATS["gather"]] * c.T).bind(wd)
    assert small.info()["lds_bytes"] < 16_384
    ids = torch.from_numpy(np.arange(100, dtype=np.int64)[::-1].copy()).cuda()
    uniq, _ = embx.dedup_tile(ids)
    assert uniq.numel() == 100
    batch = W.gen_batch(c, 0)
    idx, off = to_device(batch)
    for p in (big, small, big):
        out = torch.full((c.batch, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, c.batch, out)
        torch.cuda.synchronize()
        check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=True)


def test_tables_beyond_4_gib_read_the_right_rows():
    """Rows past byte 2^32 of a table: 9M rows of 512 bytes (4.6 GB), summed (pooling 3) and
    single-lookup, with ids on both sides of the 4 GiB boundary; integer tables, bit-exact."""
    import torch

    from gpu_helpers import check_sampled, filled_tables
    log("two 9M-row E128 fp32 tables (4.6 GB each) and a small one, ids around the 4 GiB boundary")
    tabs = [W.TableSpec(9_000_000, "fixed", 3, 3, 3, "uniform"), W.TableSpec(9_000_000, "fixed", 1, 1, 1, "uniform"),
            W.TableSpec(1000, "fixed", 2, 2, 2, "uniform")]
    c = W.Config(144, "4 GiB tables", 128, "f32", -1.0, 1.0, 2048, tabs)
    c.value_seeds = [W.value_seed(144, t) for t in range(c.T)]
    wd = filled_tables(c, W.VAL_INTEGER)
    batch = W.gen_batch(c, 0)
    edge = (1 << 32) // 512
    for t in (0, 1):
        lo, hi = batch.offsets[t * c.batch], batch.offsets[(t + 1) * c.batch]
        batch.indices[lo:lo + 6] = [edge - 1, edge, edge + 1, 0, c.rows[t] - 1, edge - 2]
    p = plan_for(c, c.batch).bind(wd)
    idx, off = to_device(batch)
    out = torch.full((c.batch, c.T, c.E), float("nan"), device="cuda")
    p.lookup(idx, off, c.batch, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert not np.isnan(got).any()
    check_sampled(c, got, batch, 3 * c.batch, seed=5, mode=W.VAL_INTEGER, exact=True)
    # the bags holding the boundary ids, checked one by one
    for t in (0, 1):
        bags = [0, 1] if t == 0 else list(range(6))
        for b in bags:
            a0, a1 = batch.offsets[t * c.batch + b], batch.offsets[t * c.batch + b + 1]
            rows = W.table_rows_at(t, batch.indices[a0:a1], c.E, c.dtype, seed=c.value_seeds[t], mode=W.VAL_INTEGER)
            assert np.array_equal(got[b, t], rows.astype(np.float64).sum(axis=0).astype(np.float32)), (t, b)
    assert p.check_errors() == 0


@pytest.mark.parametrize("B", [256, 1000, 4096])
def test_workers_holding_both_queues_walk_every_bag(B):
    """Three workers, every table split over all of them: each worker holds two single-lookup
    runs and one summed run, with 4, 12 or 44 single-lookup chunks (fewer wavefronts busy with
    them than the worker has, or all 16).  Integer tables, bit-exact, also at runtime batches
    below the max batch."""
    import torch
    log(f"3 workers, max batch {B}: pooling-1, pooling-8 and pooling-1 tables on every worker")
    c = fixed_pf_config(145, [30_000, 30_000, 500], [1, 8, 1], B=B)
    hw = host_tables(c, W.VAL_INTEGER)
    p = plan_for(c, B, num_workers=3).bind(upload_tables(hw))
    per = {}
    for ln in p.serialize().splitlines():
        if ln.startswith("item "):
            f = ln.split()
            per.setdefault(int(f[1]), set()).add(int(f[2]))
    assert sorted(per) == [0, 1, 2] and all(v == {0, 1, 2} for v in per.values())
    runs = p.info()["gather_runs"]
    log(f"  gather runs per queue {runs}")
    assert runs["single"] == 6 and runs["sw"] + runs["wave"] == 3
    for Bt in sorted({B, B // 2 + 1, 7}):
        batch = W.gen_batch(c, Bt, B=Bt)
        idx, off = to_device(batch)
        out = torch.full((Bt, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, Bt, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert not np.isnan(got).any(), f"batch {Bt}: bags never written"
        check_full(got, hw, batch, c.dtype, exact=True)
    assert p.check_errors() == 0


def test_plan_with_per_table_lookup_costs():
    """A plan made with a cost per lookup for each table (gather_lookup_ps: two tables
    priced high, one left to the vector's G1) places them differently and still matches the
    oracle bit for bit on integer tables."""
    import torch
    log("per-table lookup costs: 12,000 / 3,000 / 0 (vector's) / 25,000 ps")
    c = fixed_pf_config(146, [200_000, 5_000, 60_000, 300_000], [8, 1, 3, 20], B=2048)
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    base = plan_for(c, c.batch).bind(wd)
    p = plan_for(c, c.batch, gather_lookup_ps=[12_000.0, 3_000.0, 0.0, 25_000.0]).bind(wd)
    assert p.serialize() != base.serialize()
    batch = W.gen_batch(c, 0)
    idx, off = to_device(batch)
    for plan in (p, base):
        out = torch.full((c.batch, c.T, c.E), float("nan"), device="cuda")
        plan.lookup(idx, off, c.batch, out)
        torch.cuda.synchronize()
        check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=True)
        assert plan.check_errors() == 0

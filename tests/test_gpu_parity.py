"""GPU parity: the HIP path against the oracle, element by element, on small inputs
that span several tiles, ragged tails and the method's degenerate cases."""
import numpy as np
import pytest

import workloads as W
from oracle import index as OI
from oracle import pool as OP

from gpu_helpers import TOL, check_full, host_tables, log, plan_for, to_device, upload_tables

pytestmark = pytest.mark.gpu

STRATS = {"auto": -1, "lds": 0, "hot": 1, "dedup": 2, "gather": 3, "stream": 4}
MIXED_ROWS = [1, 7, 300, 512, 513, 2000, 50000, 300000]


def mixed_config(cfg_id, E, dtype, B=97, pf_mean=4.0, pf_hi=12, rows=MIXED_ROWS):
    tabs = []
    for t, m in enumerate(rows):
        dist = "zipf" if t % 2 == 0 else "uniform"
        tabs.append(W.TableSpec(m, "poisson", pf_mean, 0, pf_hi, dist, 1.1))
    c = W.Config(cfg_id, f"mixed E{E} {dtype}", E, dtype, -1.0, 1.0, B, tabs)
    c.value_seeds = [W.value_seed(cfg_id, t) for t in range(c.T)]
    return c


def run(c, batch, weights_dev, force=None, B=None, **opts):
    import torch
    B = batch.B if B is None else B
    if force is not None and force >= 0:
        opts["force"] = [force] * c.T
    p = plan_for(c, c.batch, **opts)
    p.bind(weights_dev)
    idx, off = to_device(batch)
    out = torch.full((B, c.T, c.E), float("nan"), device="cuda")
    p.lookup(idx, off, B, out)
    torch.cuda.synchronize()
    nbad = p.check_errors()
    return p, out.cpu().numpy(), nbad


@pytest.fixture(scope="module")
def gpu():
    import torch
    assert torch.cuda.is_available()
    import paper_2507_01676_amd as embx
    return embx


@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f16"), (32, "f32"), (256, "f32"), (96, "f32"),
                                     (8, "f16"), (4, "f32")])
@pytest.mark.parametrize("strat", list(STRATS))
def test_integer_tables_bit_exact(gpu, E, dtype, strat):
    log(f"integer tables E={E} {dtype} strategy={strat}")
    c = mixed_config(101, E, dtype)
    batch = W.gen_batch(c, 0)
    hw = host_tables(c, W.VAL_INTEGER)
    p, got, nbad = run(c, batch, upload_tables(hw), STRATS[strat])
    check_full(got, hw, batch, dtype, exact=True)
    assert nbad == 0
    if strat != "auto":
        assert p.info()["n_strategy"][strat.upper()] == p.info()["num_items"]


@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f16")])
@pytest.mark.parametrize("strat", list(STRATS))
def test_uniform_tables_within_tolerance_and_deterministic(gpu, E, dtype, strat):
    import torch
    log(f"uniform tables E={E} {dtype} strategy={strat}")
    c = mixed_config(102, E, dtype, B=301, pf_mean=9.0, pf_hi=40)
    batch = W.gen_batch(c, 0)
    hw = host_tables(c)
    wd = upload_tables(hw)
    p, got, nbad = run(c, batch, wd, STRATS[strat])
    err, _ = check_full(got, hw, batch, dtype)
    log(f"  pooled error {err:.2e}")
    # a second launch (chunk counters must have been reset) gives the same bits
    idx, off = to_device(batch)
    out2 = p.lookup(idx, off, batch.B)
    torch.cuda.synchronize()
    assert np.array_equal(out2.cpu().numpy(), got)


def test_chunked_lds_many_chunks_small_budget(gpu):
    import torch
    log("forced LDS with a 4 KiB budget: many row chunks and the chunk combine")
    c = mixed_config(103, 64, "f32", B=200, pf_mean=6.0, pf_hi=20, rows=[5000, 40000, 3])
    batch = W.gen_batch(c, 0)
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    p, got, _ = run(c, batch, wd, STRATS["lds"], lds_budget=4096)
    txt = p.serialize()
    assert max(int(ln.split()[5]) for ln in txt.splitlines() if ln.startswith("item ")) > 100
    check_full(got, hw, batch, "f32", exact=True)
    for _ in range(3):
        idx, off = to_device(batch)
        o = p.lookup(idx, off, batch.B)
        torch.cuda.synchronize()
        assert np.array_equal(o.cpu().numpy(), got)


def test_out_of_range_indices_are_skipped_and_counted(gpu):
    log("out-of-range and negative indices")
    c = mixed_config(104, 64, "f32", B=64)
    batch = W.gen_batch(c, 0)
    g = np.random.default_rng(0)
    pos = g.choice(batch.indices.size, size=40, replace=False)
    bad_vals = np.array([-1, -(1 << 40), 1 << 33], dtype=np.int64)
    batch.indices[pos] = bad_vals[g.integers(0, 3, size=40)]
    t_of = np.searchsorted(batch.offsets, np.arange(batch.indices.size), side="right") - 1
    edge = g.choice(batch.indices.size, size=10, replace=False)
    for k in edge:                                  # exactly m (one past the end)
        batch.indices[k] = c.rows[t_of[k] // batch.B]
    hw = host_tables(c, W.VAL_INTEGER)
    want_bad = OI.range_errors(batch.indices, batch.offsets, c.rows, batch.B)
    for strat in STRATS:
        p, got, nbad = run(c, batch, upload_tables(hw), STRATS[strat])
        _, bad = check_full(got, hw, batch, "f32", exact=True)
        assert nbad == bad == want_bad, (strat, nbad, want_bad)


def test_edge_shapes(gpu):
    import torch
    log("B=1, T=1, m=1, index m-1, batch below max_batch, batch 0, unbound plan")
    # single table of one row, one sample
    c = mixed_config(105, 64, "f32", B=1, rows=[1])
    batch = W.batch_from_bags(1, 1, [[0, 0, 0]])
    hw = host_tables(c, W.VAL_INTEGER)
    for strat in STRATS:
        _, got, _ = run(c, batch, upload_tables(hw), STRATS[strat])
        assert np.array_equal(got[0, 0], 3 * hw[0][0])
    # last row of each table, and a batch smaller than the plan's max
    c = mixed_config(106, 64, "f32", B=97)
    hw = host_tables(c, W.VAL_INTEGER)
    bags = [[m - 1] * (b % 3) for m in c.rows for b in range(50)]
    batch = W.batch_from_bags(c.T, 50, bags)
    for strat in STRATS:
        _, got, _ = run(c, batch, upload_tables(hw), STRATS[strat], B=50)
        check_full(got, hw, batch, "f32", exact=True)
    # batch 0 is a no-op; lookup before binding weights is refused
    import paper_2507_01676_amd as embx
    p = plan_for(c, 97)
    idx, off = to_device(batch)
    with pytest.raises(embx.EmbxError) as e:
        p.lookup(idx, off, 50)
    assert e.value.code == embx.ERR_NOT_BOUND
    p.bind(upload_tables(hw))
    out = torch.full((1, c.T, c.E), 7.0, device="cuda")
    p.lookup(idx, off, 0, out)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
    big_off = torch.zeros(c.T * 98 + 1, dtype=torch.int64, device="cuda")
    big_out = torch.empty((98, c.T, c.E), device="cuda")
    with pytest.raises(embx.EmbxError) as e:
        p.lookup(idx, big_off, 98, big_out)             # batch above the plan's max_batch
    assert e.value.code == embx.ERR_INVALID_ARGUMENT


def test_fixed_distribution_and_long_bags(gpu):
    log("all indices equal (the paper's 'fixed' distribution) and bags longer than a dedup tile")
    c = mixed_config(107, 64, "f32", B=97)
    hw = host_tables(c, W.VAL_INTEGER)
    bags = [[min(5, m - 1)] * 5 for m in c.rows for _ in range(97)]
    batch = W.batch_from_bags(c.T, 97, bags)
    for strat in STRATS:
        _, got, _ = run(c, batch, upload_tables(hw), STRATS[strat])
        check_full(got, hw, batch, "f32", exact=True)
    g = np.random.default_rng(2)
    lens = [0, 3000, 1, 2049, 2048, 0, 700, 5]
    bags = [[int(x) for x in g.integers(0, m, size=lens[(t + b) % len(lens)])] for t, m in enumerate(c.rows)
            for b in range(8)]
    batch = W.batch_from_bags(c.T, 8, bags)
    for strat in STRATS:
        _, got, _ = run(c, batch, upload_tables(hw), STRATS[strat])
        check_full(got, hw, batch, "f32", exact=True)


@pytest.mark.parametrize("n", [0, 1, 2, 3, 100, 1000, 2047, 2048])
def test_dedup_tile_matches_unique(gpu, n):
    import torch
    g = np.random.default_rng(n)
    idx = W.zipf_ranks(g, 5000, 1.1, n) * 7919 % 2_000_000_000
    d = torch.from_numpy(idx).cuda()
    uniq, inv = gpu.dedup_tile(d)
    u, i, _ = OI.dedup_tile(idx)
    assert np.array_equal(uniq.cpu().numpy(), u)
    assert np.array_equal(inv.cpu().numpy(), i)


def test_hot_probe_matches_membership(gpu):
    import torch
    c = mixed_config(108, 64, "f32", B=200)
    stats = W.history_stats(c, 200)
    p = plan_for(c, 200, stats=stats, force=[1] * c.T)
    C = {}
    for ln in p.serialize().splitlines():
        if ln.startswith("item "):
            f = ln.split()
            C[int(f[2])] = int(f[10])
    g = np.random.default_rng(4)
    for t in range(c.T):
        idx = np.concatenate([stats[t].hot_rows[:50], g.integers(0, c.rows[t], size=3000)])
        slot = p.hot_probe(t, torch.from_numpy(idx).cuda()).cpu().numpy()
        want = OI.hot_slots(idx, stats[t].hot_rows[:C[t]])
        assert np.array_equal(slot, want)


@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f16"), (32, "f32"), (256, "f32")])
def test_single_lookup_tables_and_a_broken_promise(gpu, E, dtype):
    """Tables whose statistics promise at most one lookup per bag take their own gather
    walker; bags that break the promise at run time, empty bags, bag counts that are not
    a multiple of a chunk and out-of-range ids must still match the oracle exactly."""
    log(f"single-lookup tables E={E} {dtype}")
    c = mixed_config(109, E, dtype, B=203, pf_mean=0.9, pf_hi=1)
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    stats = W.history_stats(c, c.batch)
    assert all(s.max_pooling == 1 for s in stats)
    # the promised shape: bags of 0 or 1 lookup
    batch = W.gen_batch(c, 0)
    p, got, nbad = run(c, batch, wd, STRATS["gather"])
    check_full(got, hw, batch, dtype, exact=True)
    assert nbad == 0
    # the promise broken: some bags of 2..5 lookups, some empty, a few invalid ids
    g = np.random.default_rng(7)
    bags = []
    for m in c.rows:
        for b in range(c.batch):
            n = int(g.choice([0, 1, 1, 1, 2, 5]))
            bags.append([int(x) for x in g.integers(0, m, size=n)])
    batch2 = W.batch_from_bags(c.T, c.batch, bags)
    pos = g.choice(batch2.indices.size, size=9, replace=False)
    batch2.indices[pos[:3]] = -1
    batch2.indices[pos[3:6]] = 1 << 35
    t_of = np.searchsorted(batch2.offsets, pos[6:], side="right") - 1
    batch2.indices[pos[6:]] = np.asarray(c.rows)[t_of // c.batch]
    want_bad = OI.range_errors(batch2.indices, batch2.offsets, c.rows, c.batch)
    _, got2, nbad2 = run(c, batch2, wd, STRATS["gather"])   # the same statistics (max pooling 1)
    check_full(got2, hw, batch2, dtype, exact=True)
    assert nbad2 == want_bad == 9


def test_many_tables_placed_whole(gpu):
    """300 tables (more than the planner splits over all workers): small tables are placed
    whole on single workers (the asymmetric mapping), large ones split; bit-exact on
    integer tables, single- and multi-lookup bags mixed."""
    log("300 tables, asymmetric placement")
    g = np.random.default_rng(12)
    rows = [int(x) for x in np.exp(g.uniform(np.log(10), np.log(50000), size=300))]
    tabs = []
    for t, m in enumerate(rows):
        if t % 3 == 0:
            tabs.append(W.TableSpec(m, "poisson", 3.0, 0, 9, "zipf", 1.1))
        else:
            tabs.append(W.TableSpec(m, "poisson", 1.0, 1, 1, "uniform", 1.0))
    c = W.Config(110, "many tables E64 f32", 64, "f32", -1.0, 1.0, 256, tabs)
    c.value_seeds = [W.value_seed(110, t) for t in range(c.T)]
    batch = W.gen_batch(c, 0)
    hw = host_tables(c, W.VAL_INTEGER)
    # 256 workers: at the occupancy-sized worker count of the wave gather kernel (several
    # workgroups per CU) the per-worker share is small enough that these tables are split
    p, got, nbad = run(c, batch, upload_tables(hw), num_workers=256)
    check_full(got, hw, batch, "f32", exact=True)
    assert nbad == 0
    ks = [int(ln.split()[8]) for ln in p.serialize().splitlines() if ln.startswith("item ")]
    assert ks.count(1) > 100 and max(ks) <= p.info()["num_workers"]


def test_binding_rejects_bad_tensors_before_launch(gpu):
    """Undersized, mistyped, non-contiguous or host tensors are refused on the host (no
    launch): the kernel trusts the sizes it is given."""
    import torch
    c = mixed_config(108, 64, "f32", rows=[100, 200], B=16)
    batch = W.gen_batch(c, 0)
    p = plan_for(c, 16).bind(upload_tables(host_tables(c)))
    idx, off = to_device(batch)
    B = batch.B
    good = torch.empty((B, c.T, c.E), device="cuda")
    bad = [
        dict(out=torch.empty((B - 1, c.T, c.E), device="cuda")),                     # too small
        dict(out=torch.empty((B, c.T, c.E), device="cuda", dtype=torch.float16)),    # wrong dtype
        dict(out=torch.empty((c.E, c.T, B), device="cuda").permute(2, 1, 0)),         # not contiguous
        dict(idx=idx.to(torch.int32)),
        dict(idx=idx.cpu()),
        dict(off=off[:-1]),
        dict(weights=torch.ones(idx.numel() - 1, device="cuda")),
        dict(weights=torch.ones(idx.numel(), device="cuda", dtype=torch.float64)),
    ]
    for case in bad:
        with pytest.raises(ValueError):
            p.lookup(case.get("idx", idx), case.get("off", off), B, case.get("out", good), weights=case.get("weights"))
    with pytest.raises(ValueError):
        p.bind(upload_tables(host_tables(c))[:1])
    torch.cuda.synchronize()
    assert p.check_errors() == 0
    got = p.lookup(idx, off, B, good)                                               # still usable
    torch.cuda.synchronize()
    check_full(got.cpu().numpy(), host_tables(c), batch, "f32")


def test_more_gather_slices_per_worker_than_lds_holds_is_refused(gpu):
    """A worker's gather run queue lives in LDS (about 3,400 runs of 48 B in 160 KiB):
    3,500 tables that are each split over all workers are refused with
    EMB_ERR_UNSUPPORTED at plan creation, and placing them whole (sym_max < 0) plans them."""
    T = 3500
    stats = [dict(mean_pooling=20.0, max_pooling=40, hot_rows=[], hot_freq=[], unique_frac=1.0)] * T
    with pytest.raises(gpu.EmbxError) as e:
        gpu.Plan([100000] * T, 64, "f32", stats, 4096, num_workers=256)
    assert e.value.code == gpu.ERR_UNSUPPORTED
    p = gpu.Plan([100000] * T, 64, "f32", stats, 4096, sym_max=-1, num_workers=256)
    assert p.info()["num_items"] >= T
    p.close()


def test_run_queue_beyond_64k_of_lds(gpu):
    """1,500 tables split over all workers: each worker's run queue (1,501 records of 48 B,
    72 KB) needs more than the default 64 KiB of dynamic LDS; the lookup matches the
    oracle on sampled bags, bit-exact on integer tables."""
    from gpu_helpers import check_sampled, filled_tables
    T = 1500
    tabs = [W.TableSpec(1000 + 7 * t, "fixed", 16, 16, 16, "uniform") for t in range(T)]
    c = W.Config(110, "1100 tables", 64, "f32", -0.05, 0.05, 1024, tabs)
    c.value_seeds = [W.value_seed(c.cfg_id, t) for t in range(c.T)]
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    idx, off = to_device(batch)
    for mode, exact in ((W.VAL_UNIFORM, False), (W.VAL_INTEGER, True)):
        ws = filled_tables(c, mode)
        p = plan_for(c, c.batch, stats=stats, num_workers=256).bind(ws)
        info = p.info()
        log(f"  {T} tables: {info['num_items']} slices, LDS {info['lds_bytes']} B")
        assert info["num_items"] == T * 256 and info["lds_bytes"] > 65536
        got = p.lookup(idx, off, batch.B).cpu().numpy()
        assert p.check_errors() == 0
        check_sampled(c, got, batch, 2000, seed=11, mode=mode, exact=exact)
        p.close()
        del ws

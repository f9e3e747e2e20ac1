"""GPU parity of mean pooling and per-lookup weights (Sec. II-B: sum or average of the
looked-up rows; weights scale each lookup's row) against the oracle, for every strategy
and walker: mean and sum tables mixed in one plan, weighted and unweighted launches."""
import numpy as np
import pytest

import workloads as W
from oracle import pool as OP

from gpu_helpers import TOL, host_tables, log, plan_for, to_device, upload_tables
from test_gpu_parity import MIXED_ROWS, STRATS, mixed_config

pytestmark = pytest.mark.gpu

POOLING = ["mean", "sum"]


def _weights(n, seed, integer=False):
    g = np.random.default_rng(seed)
    if integer:
        return g.integers(-3, 4, size=n).astype(np.float32)
    return g.uniform(-2.0, 2.0, size=n).astype(np.float32)


def _run(c, batch, dev_tables, pooling, psw=None, force=None, **opts):
    import torch
    if force is not None and force >= 0:
        opts["force"] = [force] * c.T
    p = plan_for(c, c.batch, pooling=pooling, **opts)
    p.bind(dev_tables)
    idx, off = to_device(batch)
    out = torch.full((batch.B, c.T, c.E), float("nan"), device="cuda")
    wd = None if psw is None else torch.from_numpy(psw).cuda()
    p.lookup(idx, off, batch.B, out, weights=wd)
    torch.cuda.synchronize()
    nbad = p.check_errors()
    return p, out.cpu().numpy(), nbad


def _check(got, host, batch, dtype, pooling, psw, exact=False):
    ref, mag, bad = OP.pool_reference(host, batch.indices, batch.offsets, batch.B, pooling=pooling, psw=psw)
    empty = OP.empty_bag_mask(batch.offsets, len(host), batch.B)
    assert np.all(got[empty] == 0) and not np.any(np.signbit(got[empty])), "empty bags must be +0.0"
    if exact:
        diff = np.argwhere(got != ref)
        assert diff.size == 0, f"{diff.shape[0]} elements differ, first {diff[:3].tolist()}"
        return 0.0, bad
    err = OP.pooled_error(got, ref, mag)
    assert err <= TOL[dtype], f"pooled error {err:.3e} > {TOL[dtype]}"
    return err, bad


@pytest.fixture(scope="module")
def gpu():
    import torch
    assert torch.cuda.is_available()
    import paper_2507_01676_amd as embx
    return embx


@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f16"), (32, "f32"), (256, "f32"), (96, "f32")])
@pytest.mark.parametrize("strat", list(STRATS))
@pytest.mark.parametrize("weighted", [False, True])
def test_mean_and_weights_match_oracle(gpu, E, dtype, strat, weighted):
    log(f"pooling E={E} {dtype} strategy={strat} weighted={weighted}")
    c = mixed_config(201, E, dtype)
    batch = W.gen_batch(c, 0)
    pooling = [POOLING[t % 2] for t in range(c.T)]
    psw = _weights(batch.indices.size, 5) if weighted else None
    hw = host_tables(c)
    p, got, nbad = _run(c, batch, upload_tables(hw), pooling, psw, STRATS[strat])
    err, bad = _check(got, hw, batch, dtype, pooling, psw)
    assert nbad == bad == 0
    if strat != "auto":
        assert p.info()["n_strategy"][strat.upper()] == p.info()["num_items"]


@pytest.mark.parametrize("strat", list(STRATS))
def test_integer_weights_on_integer_tables_bit_exact(gpu, strat):
    """Integer rows times integer weights, summed below 2^24: every order gives the exact sum."""
    log(f"integer weights strategy={strat}")
    c = mixed_config(202, 64, "f32")
    batch = W.gen_batch(c, 1)
    psw = _weights(batch.indices.size, 6, integer=True)
    hw = host_tables(c, W.VAL_INTEGER)
    _, got, _ = _run(c, batch, upload_tables(hw), "sum", psw, STRATS[strat])
    _check(got, hw, batch, "f32", "sum", psw, exact=True)


@pytest.mark.parametrize("weighted", [False, True])
def test_chunked_lds_mean_divides_the_combined_sum(gpu, weighted):
    log(f"chunked LDS mean weighted={weighted}")
    c = mixed_config(203, 64, "f32", rows=[5000, 20000, 3])
    batch = W.gen_batch(c, 2)
    psw = _weights(batch.indices.size, 7) if weighted else None
    hw = host_tables(c)
    p, got, _ = _run(c, batch, upload_tables(hw), "mean", psw, STRATS["lds"], lds_budget=16384)
    assert max(int(ln.split()[5]) for ln in p.serialize().splitlines() if ln.startswith("item ")) > 1
    _check(got, hw, batch, "f32", "mean", psw)


@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f16"), (256, "f32")])
@pytest.mark.parametrize("weighted", [False, True])
def test_long_bags_wave_mode(gpu, E, dtype, weighted):
    log(f"long bags E={E} {dtype} weighted={weighted}")
    c = mixed_config(204, E, dtype, B=40, pf_mean=150.0, pf_hi=400, rows=[100000, 3000, 70])
    batch = W.gen_batch(c, 3)
    pooling = ["mean", "sum", "mean"]
    psw = _weights(batch.indices.size, 8) if weighted else None
    hw = host_tables(c)
    _, got, _ = _run(c, batch, upload_tables(hw), pooling, psw, STRATS["gather"])
    _check(got, hw, batch, dtype, pooling, psw)


@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f16")])
def test_single_lookup_tables_mean_and_weights_with_a_broken_promise(gpu, E, dtype):
    """Tables promised at most one lookup per bag get bags of 2..5 at run time, empty bags
    and invalid ids (whose NaN weights must add nothing)."""
    log(f"single-lookup tables E={E} {dtype}")
    tabs = [W.TableSpec(m, "poisson", 1.0, 1, 1, "uniform", 1.0) for m in (1000, 50, 200000)]
    c = W.Config(205, "single", E, dtype, -1.0, 1.0, 300, tabs)
    c.value_seeds = [W.value_seed(205, t) for t in range(c.T)]
    stats = W.history_stats(c)
    g = np.random.default_rng(9)
    bags = []
    for t, m in enumerate(c.rows):
        for b in range(c.batch):
            n = int(g.choice([0, 1, 1, 1, 2, 5]))
            bags.append([int(x) for x in g.integers(0, m, size=n)])
    batch = W.batch_from_bags(c.T, c.batch, bags)
    psw = _weights(batch.indices.size, 10)
    bad_pos = g.choice(batch.indices.size, size=7, replace=False)
    batch.indices[bad_pos] = -3
    psw[bad_pos] = np.nan
    hw = host_tables(c)
    import torch
    for pooling, w in (("mean", None), ("mean", psw), (["sum", "mean", "sum"], psw)):
        p = plan_for(c, c.batch, stats=stats, pooling=pooling)
        p.bind(upload_tables(hw))
        idx, off = to_device(batch)
        out = torch.full((batch.B, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, batch.B, out, weights=None if w is None else torch.from_numpy(w).cuda())
        torch.cuda.synchronize()
        assert p.check_errors() == 7
        got = out.cpu().numpy()
        assert np.all(np.isfinite(got))
        _check(got, hw, batch, dtype, pooling, w)


def test_invalid_ids_ignore_nan_weights_in_every_walker(gpu):
    log("invalid ids with NaN weights")
    c = mixed_config(206, 64, "f32")
    batch = W.gen_batch(c, 4)
    psw = _weights(batch.indices.size, 11)
    g = np.random.default_rng(12)
    pos = g.choice(batch.indices.size, size=40, replace=False)
    batch.indices[pos] = np.where(np.arange(40) % 2 == 0, -1, 1 << 40)
    psw[pos] = np.nan
    hw = host_tables(c)
    for strat in STRATS:
        _, got, nbad = _run(c, batch, upload_tables(hw), "mean", psw, STRATS[strat])
        assert nbad == 40, strat
        assert np.all(np.isfinite(got)), strat
        _check(got, hw, batch, "f32", "mean", psw)


def test_weighted_entry_point_rejects_missing_weights(gpu):
    import ctypes
    import torch
    c = mixed_config(207, 64, "f32", rows=[100, 200])
    batch = W.gen_batch(c, 0)
    p = plan_for(c, c.batch).bind(upload_tables(host_tables(c)))
    idx, off = to_device(batch)
    out = torch.empty((batch.B, c.T, c.E), device="cuda")
    code = gpu._lib.emb_lookup_weighted(p._h, idx.data_ptr(), off.data_ptr(), None, batch.B, out.data_ptr(),
                                        torch.cuda.current_stream().cuda_stream)
    assert code == gpu.ERR_INVALID_ARGUMENT
    with pytest.raises(gpu.EmbxError):
        gpu.Plan(c.rows, c.E, c.dtype, W.history_stats(c), c.batch, pooling=[0, 2])

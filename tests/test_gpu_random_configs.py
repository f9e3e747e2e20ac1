"""Seeded random configurations against the oracle, bit-exact on integer tables: table
counts, row counts (1 .. 300k), E and dtype (every row width both kernels take), pooling
factors (empty bags, single-lookup tables, long bags), index distributions, mean or sum per
table, weights, and a runtime batch below the max batch -- each planned automatically, and
the same configurations again with every table forced to each staged flow."""
import numpy as np
import pytest

import workloads as W
from oracle import pool as OP

from gpu_helpers import host_tables, log, plan_for, to_device, upload_tables

pytestmark = pytest.mark.gpu

SHAPES = [(32, "f32"), (64, "f32"), (96, "f32"), (128, "f32"), (256, "f32"), (64, "f16"), (128, "f16"),
          (256, "f16"), (8, "f16"), (16, "f32")]


def random_config(seed):
    g = np.random.default_rng(seed)
    E, dtype = SHAPES[seed % len(SHAPES)]
    T = int(g.integers(1, 12))
    tabs = []
    for _ in range(T):
        rows = int(g.choice([1, 7, 100, 513, 4000, 70000, 300000]))
        kind = g.integers(0, 4)
        if kind == 0:
            tabs.append(W.TableSpec(rows, "fixed", 1, 1, 1, "uniform"))
        elif kind == 1:
            tabs.append(W.TableSpec(rows, "poisson", float(g.uniform(0.5, 4)), 0, 10, "zipf", float(g.uniform(0.8, 1.5))))
        elif kind == 2:
            tabs.append(W.TableSpec(rows, "poisson", float(g.uniform(10, 60)), 1, 120, "uniform"))
        else:
            tabs.append(W.TableSpec(rows, "fixed", int(g.integers(2, 40)), 0, 0, "fixed"))
    B = int(g.integers(1, 300))
    c = W.Config(5000 + seed, f"random {seed}", E, dtype, -1.0, 1.0, B, tabs)
    c.value_seeds = [W.value_seed(5000 + seed, t) for t in range(c.T)]
    return c, g


@pytest.mark.parametrize("seed", range(48))
def test_random_configuration_matches_the_oracle(seed):
    import torch
    c, g = random_config(seed)
    log(f"seed {seed}: T {c.T}, E {c.E} {c.dtype}, max batch {c.batch}, rows {c.rows}")
    hw = host_tables(c, W.VAL_INTEGER)
    pooling = [("mean" if g.random() < 0.4 else "sum") for _ in range(c.T)]
    p = plan_for(c, c.batch, pooling=pooling).bind(upload_tables(hw))
    info = p.info()
    log(f"  {info['kernel']}, gather steps {info['gather_steps']}, {info['n_strategy']}")
    for B in sorted({c.batch, max(1, c.batch // 3)}):
        batch = W.gen_batch(c, B, B=B)
        idx, off = to_device(batch)
        weighted = bool(g.random() < 0.5)
        psw = g.integers(-3, 4, size=batch.indices.size).astype(np.float32) if weighted else None
        out = torch.full((B, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, B, out, weights=torch.from_numpy(psw).cuda() if weighted else None)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ref, mag, bad = OP.pool_reference(hw, batch.indices, batch.offsets, B, pooling=pooling, psw=psw)
        if any(x == "mean" for x in pooling):
            err = OP.pooled_error(got, ref, mag)
            assert err <= 1e-6, f"batch {B}: pooled error {err:.3e}"
            sums = [t for t in range(c.T) if pooling[t] == "sum"]
            assert np.array_equal(got[:, sums], ref[:, sums]), f"batch {B}: sum tables differ"
        else:
            diff = np.argwhere(got != ref)
            assert diff.size == 0, f"batch {B}: {diff.shape[0]} elements differ, first {diff[:3].tolist()}"
        assert p.check_errors() == bad


@pytest.mark.parametrize("strat", ["lds", "hot", "dedup", "stream"])
@pytest.mark.parametrize("seed", range(20))
def test_random_configuration_with_a_forced_staged_strategy(seed, strat):
    """The same random configurations with every table forced to one staged flow (the
    planner would pick GATHER): row chunks, hot-row caches, tile dedup and chunked scans
    on odd shapes, bit-exact on integer tables at the max batch and a third of it."""
    import torch
    code = {"lds": 0, "hot": 1, "dedup": 2, "stream": 4}[strat]
    c, _ = random_config(seed)
    log(f"seed {seed}, all {strat}: T {c.T}, E {c.E} {c.dtype}, max batch {c.batch}, rows {c.rows}")
    hw = host_tables(c, W.VAL_INTEGER)
    p = plan_for(c, c.batch, force=[code] * c.T).bind(upload_tables(hw))
    for B in sorted({c.batch, max(1, c.batch // 3)}):
        batch = W.gen_batch(c, B, B=B)
        idx, off = to_device(batch)
        out = torch.full((B, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, B, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ref, _, bad = OP.pool_reference(hw, batch.indices, batch.offsets, B)
        diff = np.argwhere(got != ref)
        assert diff.size == 0, f"batch {B}: {diff.shape[0]} elements differ, first {diff[:3].tolist()}"
        assert p.check_errors() == bad

"""The wave-uniform gather kernel is built for 12, 13 and 16 row loads in flight per
step, and a plan picks one.  Every build against the oracle (EMBX_GATHER_STEPS forces
it): integer tables bit-exact and uniform tables to the tolerance, for rows of 16, 32 and
64 lanes, fp32 and fp16, single-lookup and multi-lookup bags in one plan, weighted and
mean; and the automatic choice on the five workloads' plans."""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, to_device, upload_tables
from test_gpu_pooling import _check, _weights

pytestmark = pytest.mark.gpu

STEPS = [12, 13, 16]


def steps_config(cfg_id, E, dtype, B=203):
    """Single-lookup tables (max pooling 1) beside multi-lookup ones of several pooling
    factors, so that both of the kernel's queues run and steps end inside and across bags."""
    tabs = [W.TableSpec(5000, "fixed", 1, 1, 1, "uniform"),
            W.TableSpec(300000, "fixed", 50, 50, 50, "zipf", 1.5),
            W.TableSpec(70, "poisson", 8.0, 1, 20, "uniform"),
            W.TableSpec(120000, "poisson", 20.0, 0, 100, "zipf", 1.1),
            W.TableSpec(1, "fixed", 1, 1, 1, "uniform"),
            W.TableSpec(2000, "poisson", 3.0, 0, 9, "zipf", 1.05)]
    c = W.Config(cfg_id, f"gather steps E{E} {dtype}", E, dtype, -1.0, 1.0, B, tabs)
    c.value_seeds = [W.value_seed(cfg_id, t) for t in range(c.T)]
    return c


@pytest.mark.parametrize("ks", STEPS)
@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f32"), (256, "f32"), (128, "f16"), (256, "f16")])
def test_every_build_matches_the_oracle(monkeypatch, ks, E, dtype):
    import torch
    log(f"gather steps {ks}, E{E} {dtype}")
    monkeypatch.setenv("EMBX_GATHER_STEPS", str(ks))
    c = steps_config(160, E, dtype)
    batch = W.gen_batch(c, 0)
    for mode in (W.VAL_INTEGER, W.VAL_UNIFORM):
        hw = host_tables(c, mode)
        p = plan_for(c, c.batch).bind(upload_tables(hw))
        info = p.info()
        assert info["kernel"] == "gather_kernel" and info["gather_steps"] == ks
        assert info["gather_runs"]["single"] > 0 and info["gather_runs"]["sw"] > 0
        idx, off = to_device(batch)
        out = torch.full((batch.B, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, batch.B, out)
        torch.cuda.synchronize()
        check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=mode == W.VAL_INTEGER)
        assert p.check_errors() == 0
        # a runtime batch below the max batch
        B2 = 97
        b2 = W.gen_batch(c, 1, B=B2)
        i2, o2 = to_device(b2)
        out2 = torch.full((B2, c.T, c.E), float("nan"), device="cuda")
        p.lookup(i2, o2, B2, out2)
        torch.cuda.synchronize()
        check_full(out2.cpu().numpy(), hw, b2, c.dtype, exact=mode == W.VAL_INTEGER)
        p.close()


@pytest.mark.parametrize("ks", STEPS)
@pytest.mark.parametrize("E,dtype", [(64, "f32"), (128, "f32"), (256, "f32"), (128, "f16"), (256, "f16")])
def test_every_build_weighted_and_mean(monkeypatch, ks, E, dtype):
    import torch
    log(f"gather steps {ks}, E{E} {dtype}: weighted, mean and sum tables")
    monkeypatch.setenv("EMBX_GATHER_STEPS", str(ks))
    c = steps_config(161, E, dtype)
    batch = W.gen_batch(c, 0)
    hw = host_tables(c, W.VAL_INTEGER)
    pooling = ["mean" if t % 2 == 0 else "sum" for t in range(c.T)]
    psw = _weights(batch.indices.size, 77, integer=True)
    p = plan_for(c, c.batch, pooling=pooling).bind(upload_tables(hw))
    assert p.info()["gather_steps"] == ks
    idx, off = to_device(batch)
    out = torch.full((batch.B, c.T, c.E), float("nan"), device="cuda")
    p.lookup(idx, off, batch.B, out, weights=torch.from_numpy(psw).cuda())
    torch.cuda.synchronize()
    _check(out.cpu().numpy(), hw, batch, c.dtype, pooling, psw)


def test_unknown_step_count_is_refused(monkeypatch):
    import paper_2507_01676_amd as embx
    monkeypatch.setenv("EMBX_GATHER_STEPS", "14")
    c = steps_config(162, 64, "f32")
    with pytest.raises(embx.EmbxError):
        plan_for(c, c.batch)


def test_the_workloads_choices(monkeypatch):
    """The plan's choice: the fewest row rounds over its multi-lookup chunks, ties to the
    larger; single-lookup bags only (workload 2) keep 12."""
    monkeypatch.delenv("EMBX_GATHER_STEPS", raising=False)
    want = {2: 12, 3: 16, 4: 16, 5: 16}
    for cfg, ks in want.items():
        c = W.make_config(cfg)
        p = plan_for(c, c.batch, stats=W.history_stats(c))
        info = p.info()
        log(f"  workload {cfg}: {info['kernel']}, gather steps {info['gather_steps']}")
        assert info["kernel"] == "gather_kernel" and info["gather_steps"] == ks
        p.close()
    c = W.make_config(1)
    p = plan_for(c, c.batch)
    assert p.info()["kernel"] == "lookup_kernel" and p.info()["gather_steps"] == 0

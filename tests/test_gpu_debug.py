"""The debugging switches on the GPU, each against the oracle:

- EMBX_DEBUG_CHECKS: a plan made with it checks every launch's input on the host first.
  Malformed offsets are refused before anything is launched. Out-of-range ids are
  listed on stderr, then skipped and counted by the kernel as usual. The one launch here
  with malformed offsets (offsets[0] = 1) would read only inside the buffers if it ran.
  The other malformed inputs go only to the check itself, which launches nothing.
- EMBX_LOG: plan creation prints the plan's summary line on stderr.
- EMBX_FORCE_STRATEGY: every table is forced to one strategy, and the results stay the
  oracle's.
"""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, to_device, upload_tables
from test_gpu_regressions import fixed_pf_config

pytestmark = pytest.mark.gpu

B = 64


def _setup(monkeypatch, debug=True):
    if debug:
        monkeypatch.setenv("EMBX_DEBUG_CHECKS", "1")
    else:
        monkeypatch.delenv("EMBX_DEBUG_CHECKS", raising=False)
    c = fixed_pf_config(150, [1000, 5000, 300, 20000], [5, 1, 8, 3], B=B)
    hw = host_tables(c, W.VAL_INTEGER)
    p = plan_for(c, B).bind(upload_tables(hw))
    return c, hw, p, W.gen_batch(c, 0, B=B)


def _nan_out(c):
    import torch
    return torch.full((B, c.T, c.E), float("nan"), device="cuda")


def test_debug_checks_pass_well_formed_input(monkeypatch):
    import torch
    log("EMBX_DEBUG_CHECKS=1: a well-formed batch, bit-exact")
    c, hw, p, batch = _setup(monkeypatch)
    assert p.info()["debug_checks"] == 1
    idx, off = to_device(batch)
    out = _nan_out(c)
    p.lookup(idx, off, B, out)
    torch.cuda.synchronize()
    check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=True)
    assert p.check_errors() == 0
    p.check_input(idx, off, B)
    p.close()
    _, _, q, _ = _setup(monkeypatch, debug=False)
    assert q.info()["debug_checks"] == 0


def test_debug_checks_refuse_malformed_offsets(monkeypatch, capfd):
    import torch

    import paper_2507_01676_amd as embx
    log("EMBX_DEBUG_CHECKS=1: malformed offsets refused before any launch")
    c, hw, p, batch = _setup(monkeypatch)
    # the checks are on, so none of the malformed inputs below reaches a kernel
    assert p.info()["debug_checks"] == 1
    idx, off = to_device(batch)
    out = _nan_out(c)
    o1 = batch.offsets.copy()
    assert o1[1] >= 1
    o1[0] = 1
    with pytest.raises(embx.EmbxError):
        p.lookup(idx, torch.from_numpy(o1).cuda(), B, out)
    assert "offsets[0] = 1" in capfd.readouterr().err
    o2 = batch.offsets.copy()
    o2[10] = o2[9] - 1
    with pytest.raises(embx.EmbxError):
        p.check_input(idx, torch.from_numpy(o2).cuda(), B)
    assert "offsets[10]" in capfd.readouterr().err
    o3 = batch.offsets.copy()
    o3[-1] = 1 << 40
    with pytest.raises(embx.EmbxError):
        p.check_input(idx, torch.from_numpy(o3).cuda(), B)
    assert "run past their allocation" in capfd.readouterr().err
    # weights shorter than the indices: 2^20 ids in their own 8 MiB allocation, 2^20
    # weights where a 2 MiB segment holds 4 KiB
    n = 1 << 20
    big_idx = torch.zeros(n, dtype=torch.int64, device="cuda")
    o4 = np.zeros(c.T * B + 1, np.int64)
    o4[-1] = n
    small_w = torch.ones(1024, dtype=torch.float32, device="cuda")
    p.check_input(big_idx, torch.from_numpy(o4).cuda(), B)
    with pytest.raises(embx.EmbxError):
        p.check_input(big_idx, torch.from_numpy(o4).cuda(), B, weights=small_w)
    assert "weights run past their allocation" in capfd.readouterr().err
    # untouched by the refusals
    p.lookup(idx, off, B, out)
    torch.cuda.synchronize()
    check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=True)


def test_debug_checks_list_out_of_range_ids(monkeypatch, capfd):
    import torch
    log("EMBX_DEBUG_CHECKS=1: out-of-range ids listed, skipped and counted")
    c, hw, p, batch = _setup(monkeypatch)
    assert p.info()["debug_checks"] == 1
    ix = batch.indices.copy()
    lo0 = batch.offsets[0]
    ix[lo0] = -3
    ix[batch.offsets[2 * B] + 1] = c.rows[2] + 7
    bad = W.Batch(batch.B, batch.T, ix, batch.offsets)
    idx = torch.from_numpy(ix).cuda()
    off = torch.from_numpy(batch.offsets).cuda()
    out = _nan_out(c)
    capfd.readouterr()
    p.lookup(idx, off, B, out)
    torch.cuda.synchronize()
    err = capfd.readouterr().err
    assert "table 0" in err and "= -3 outside" in err
    assert "table 2" in err and f"= {c.rows[2] + 7} outside" in err
    assert "2 ids out of range" in err
    assert p.check_errors() == 2
    _, nbad = check_full(out.cpu().numpy(), hw, bad, c.dtype, exact=True)
    assert nbad == 2


def test_log_prints_the_plan_summary(monkeypatch, capfd):
    log("EMBX_LOG=1: plan summary on stderr")
    monkeypatch.setenv("EMBX_LOG", "1")
    c, hw, p, batch = _setup(monkeypatch, debug=False)
    err = capfd.readouterr().err
    info = p.info()
    line = [ln for ln in err.splitlines() if ln.startswith("embx plan:")]
    assert len(line) == 1, err
    assert f"T {c.T} E {c.E} f32" in line[0]
    assert f"K {info['num_workers']}" in line[0] and f"GATHER {info['n_strategy']['GATHER']}" in line[0]
    assert info["kernel"] in line[0]
    monkeypatch.delenv("EMBX_LOG")
    _setup(monkeypatch, debug=False)
    assert "embx plan:" not in capfd.readouterr().err


@pytest.mark.parametrize("name", ["dedup", "stream", "lds"])
def test_force_strategy_variable_keeps_the_oracles_results(monkeypatch, name):
    import torch
    log(f"EMBX_FORCE_STRATEGY={name}: every table forced, bit-exact")
    monkeypatch.setenv("EMBX_FORCE_STRATEGY", name)
    c, hw, p, batch = _setup(monkeypatch, debug=False)
    code = {"lds": "LDS", "dedup": "DEDUP", "stream": "STREAM"}[name]
    ns = p.info()["n_strategy"]
    assert ns[code] > 0 and sum(ns.values()) == ns[code]
    idx, off = to_device(batch)
    out = _nan_out(c)
    p.lookup(idx, off, B, out)
    torch.cuda.synchronize()
    check_full(out.cpu().numpy(), hw, batch, c.dtype, exact=True)

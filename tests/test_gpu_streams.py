"""Two plans used at once from two streams (default priority), as a server holding two
models would: their launches interleave and may run concurrently on the device. Each
plan's chunk workspace, counters and out-of-range counter are its own, so every output
matches the oracle bit-exactly and each plan reports only its own bad indices."""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, upload_tables
from test_gpu_parity import STRATS, mixed_config

pytestmark = pytest.mark.gpu


def test_two_plans_on_two_streams():
    import torch
    log("two plans, two streams, interleaved launches")
    ca = mixed_config(130, 64, "f32")
    cb = mixed_config(131, 128, "f16", rows=[3, 900, 40000, 250000])
    ha, hb = host_tables(ca, W.VAL_INTEGER), host_tables(cb, W.VAL_INTEGER)
    # plan A row-chunks its larger tables (a workspace and arrival counters); plan B is the planner's
    pa = plan_for(ca, ca.batch, force=[STRATS["lds"]] * ca.T).bind(upload_tables(ha))
    pb = plan_for(cb, cb.batch).bind(upload_tables(hb))
    ba = W.gen_batch(ca, 0)
    bb = W.gen_batch(cb, 1)
    ia = ba.indices.copy()
    ia[: 3] = -1                      # three out-of-range indices in plan A's batch only
    dev_a = (torch.from_numpy(ia).cuda(), torch.from_numpy(ba.offsets).cuda())
    dev_b = (torch.from_numpy(bb.indices).cuda(), torch.from_numpy(bb.offsets).cuda())
    n = 12
    outs_a = [torch.full((ca.batch, ca.T, ca.E), float("nan"), device="cuda") for _ in range(n)]
    outs_b = [torch.full((cb.batch, cb.T, cb.E), float("nan"), device="cuda") for _ in range(n)]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    sa.wait_stream(torch.cuda.current_stream())
    sb.wait_stream(torch.cuda.current_stream())
    for i in range(n):
        pa.lookup(*dev_a, ca.batch, outs_a[i], stream=sa)
        pb.lookup(*dev_b, cb.batch, outs_b[i], stream=sb)
    torch.cuda.synchronize()
    assert pa.check_errors() == 3 * n
    assert pb.check_errors() == 0
    batch_a = W.Batch(B=ba.B, T=ba.T, indices=ia, offsets=ba.offsets)
    ref_a = None
    for i in range(n):
        got_a = outs_a[i].cpu().numpy()
        if ref_a is None:
            check_full(got_a, ha, batch_a, "f32", exact=True)
            ref_a = got_a
        assert np.array_equal(got_a, ref_a), f"plan A launch {i} differs"
        check_full(outs_b[i].cpu().numpy(), hb, bb, "f16", exact=True)


def test_two_batches_in_flight_over_the_same_tables():
    """The throughput mode of bench.py --streams 2: consecutive batches dealt to two
    streams, each with its own plan over the same device tables and its own outputs, so
    that one batch's last workers overlap the next batch's first. Integer tables: every
    output bit-exact against the oracle."""
    import torch
    log("two plans over one set of tables, batches dealt to two streams")
    c = mixed_config(132, 64, "f32")
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    plans = [plan_for(c, c.batch).bind(wd) for _ in range(2)]
    log(f"  kernel {plans[0].info()['kernel']}")
    batches = [W.gen_batch(c, s) for s in range(4)]
    dev = [(torch.from_numpy(b.indices).cuda(), torch.from_numpy(b.offsets).cuda()) for b in batches]
    n = 16
    outs = [torch.full((c.batch, c.T, c.E), float("nan"), device="cuda") for _ in range(n)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for i in range(n):
        plans[i % 2].lookup(*dev[i % 4], c.batch, outs[i], stream=streams[i % 2])
    torch.cuda.synchronize()
    for i in range(n):
        check_full(outs[i].cpu().numpy(), hw, batches[i % 4], "f32", exact=True)
    assert all(p.check_errors() == 0 for p in plans)

"""emb_lookup enqueues one kernel and neither allocates nor synchronizes, so a serving
loop may capture it in a HIP graph (torch.cuda.CUDAGraph). A captured lookup of every
strategy is replayed several times over different batches written into the same input
buffers, with eager lookups and synchronizations between the replays; every replay is
checked against the oracle (integer tables: bit-exact) and against the eager lookup."""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, upload_tables
from test_gpu_parity import STRATS, mixed_config

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("strat", list(STRATS))
def test_graph_replays_match_eager_and_oracle(strat):
    import torch
    log(f"graph capture, strategy {strat}")
    c = mixed_config(120, 64, "f32")
    hw = host_tables(c, W.VAL_INTEGER)
    weights = upload_tables(hw)
    force = STRATS[strat]
    plan = plan_for(c, c.batch, **({} if force < 0 else {"force": [force] * c.T}))
    plan.bind(weights)
    batches = [W.gen_batch(c, s) for s in range(3)]
    nnz = max(b.indices.size for b in batches)
    idx = torch.zeros(nnz, dtype=torch.int64, device="cuda")
    off = torch.zeros(c.T * c.batch + 1, dtype=torch.int64, device="cuda")
    out = torch.full((c.batch, c.T, c.E), float("nan"), device="cuda")

    def load(b):
        idx[: b.indices.size].copy_(torch.from_numpy(b.indices))
        off.copy_(torch.from_numpy(b.offsets))

    load(batches[0])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        plan.lookup(idx, off, c.batch, out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan.lookup(idx, off, c.batch, out)
    torch.cuda.synchronize()
    for rep in range(6):
        b = batches[rep % len(batches)]
        load(b)
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        check_full(got, hw, b, "f32", exact=True)
        eager = plan.lookup(idx, off, c.batch)
        torch.cuda.synchronize()
        assert np.array_equal(eager.cpu().numpy(), got), f"replay {rep} differs from the eager lookup"
    assert plan.check_errors() == 0
    del g

"""emb_plan_create_noalloc through the C ABI: the plan's device data in the library's fixed
per-GPU array instead of allocations.  Its lookups equal those of the same plan made by
emb_plan_create, bit for bit (and the oracle on integer tables), on two calls in a row, the
second with a smaller input; the first handle is refused once the second plan has replaced
it; a plan whose device data exceed the array is refused."""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, to_device, upload_tables
from test_gpu_parity import STRATS, mixed_config

pytestmark = pytest.mark.gpu


def _compare(c, strat, rows=None):
    """A regular and a scratch plan of the same tables and options; both lookups of one
    batch, bit-exact against each other and the oracle (integer tables)."""
    import torch

    import paper_2507_01676_amd as embx
    batch = W.gen_batch(c, 0)
    stats = W.history_stats(c)
    hw = host_tables(c, W.VAL_INTEGER)
    wd = upload_tables(hw)
    opts = {} if strat == "auto" else {"force": [STRATS[strat]] * c.T}
    reg = plan_for(c, c.batch, stats=stats, **opts).bind(wd)
    na = embx.Plan(c.rows, c.E, c.dtype, stats, c.batch, noalloc=True, **opts).bind(wd)
    assert na.serialize() == reg.serialize()
    idx, off = to_device(batch)
    outs = []
    for p in (reg, na):
        out = torch.full((c.batch, c.T, c.E), float("nan"), device="cuda")
        p.lookup(idx, off, c.batch, out)
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
        assert p.check_errors() == 0
    assert np.array_equal(outs[0], outs[1])
    check_full(outs[1], hw, batch, c.dtype, exact=True)
    return reg, na


@pytest.mark.parametrize("strat", ["lds", "hot", "auto"])
def test_noalloc_plan_matches_the_allocating_one_twice(strat):
    import paper_2507_01676_amd as embx
    log(f"noalloc plan, strategy {strat}: a large input, then a smaller one")
    c1 = mixed_config(160, 64, "f32", B=301, pf_mean=6.0, pf_hi=20)
    reg1, na1 = _compare(c1, strat)
    c2 = mixed_config(161, 64, "f32", B=97, pf_mean=3.0, pf_hi=9, rows=[5, 700, 3000, 90000])
    reg2, na2 = _compare(c2, strat)
    # the second scratch plan replaced the first: its handle is refused, destroy still works
    with pytest.raises(embx.EmbxError) as e:
        na1.check_errors()
    assert e.value.code == embx.ERR_INVALID_ARGUMENT
    na1.close()
    assert na2.check_errors() == 0
    for p in (reg1, reg2, na2):
        p.close()


def test_noalloc_plan_beyond_the_array_is_refused():
    import paper_2507_01676_amd as embx
    log("noalloc plan whose row-chunk partial sums exceed the array")
    # one 300k-row table of 512-byte rows forced into LDS chunks: [chunks, 1000, 128] fp32
    # partial sums, far beyond 64 MiB
    st = [dict(mean_pooling=4.0, max_pooling=8, hot_rows=[], hot_freq=[], unique_frac=1.0)]
    with pytest.raises(embx.EmbxError) as e:
        embx.Plan([300_000], 128, "f32", st, 1000, noalloc=True, force=[STRATS["lds"]])
    assert e.value.code == embx.ERR_UNSUPPORTED
    p = embx.Plan([300_000], 128, "f32", st, 1000, force=[STRATS["lds"]])   # the allocating one plans it
    p.close()

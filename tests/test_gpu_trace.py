"""A traced launch (emb_plan_set_trace on) computes what an untraced one does, and its
timers are consistent: the staged kernel adds a workgroup barrier per staged slice, the
wave gather kernel only writes time stamps."""
import numpy as np
import pytest

import workloads as W

from gpu_helpers import check_full, host_tables, log, plan_for, to_device, upload_tables
from test_gpu_parity import STRATS, mixed_config

pytestmark = pytest.mark.gpu

KW = 18   # timer entries per worker: start, end of staged slices, end of each of 16 wavefronts


@pytest.mark.parametrize("strat", ["auto", "gather", "lds", "hot", "dedup", "stream"])
def test_traced_launch_is_bit_exact_and_timers_are_monotone(strat):
    import torch
    log(f"traced launch, strategy {strat}")
    c = mixed_config(150, 64, "f32", B=301, pf_mean=6.0, pf_hi=20)
    batch = W.gen_batch(c, 0)
    hw = host_tables(c, W.VAL_INTEGER)
    opts = {} if strat == "auto" else {"force": [STRATS[strat]] * c.T}
    p = plan_for(c, c.batch, **opts).bind(upload_tables(hw))
    idx, off = to_device(batch)
    plain = p.lookup(idx, off, batch.B)
    torch.cuda.synchronize()
    n = p.trace_size()
    info = p.info()
    K = info["num_workers"]
    items = [ln.split() for ln in p.serialize().splitlines() if ln.startswith("item ")]
    assert n == K * KW + 2 * len(items)
    tr = torch.zeros(n, dtype=torch.int64, device="cuda")
    assert p.set_trace(tr) == n
    traced = p.lookup(idx, off, batch.B)
    torch.cuda.synchronize()
    assert p.set_trace(None) == n
    got = traced.cpu().numpy()
    check_full(got, hw, batch, c.dtype, exact=True)
    assert np.array_equal(got, plain.cpu().numpy())
    assert p.check_errors() == 0
    t = tr.cpu().numpy()
    per = t[:K * KW].reshape(K, KW)
    start, staged_end, wave_end = per[:, 0], per[:, 1], per[:, 2:2 + info["block_threads"] // 64]
    assert np.all(start > 0) and np.all(staged_end >= start)
    assert np.all(wave_end >= staged_end[:, None])
    span_us = (wave_end.max() - start.min()) / 100.0
    assert 0 < span_us < 1e5, span_us
    # staged slices: begin and end inside their worker's span; gather slices are not timed
    sl = t[K * KW:].reshape(-1, 2)
    for i, it in enumerate(items):
        w, st_ = int(it[1]), int(it[3])
        if st_ == STRATS["gather"]:
            assert sl[i, 0] == 0 and sl[i, 1] == 0
        else:
            assert start[w] <= sl[i, 0] <= sl[i, 1] <= wave_end[w].max()
    log(f"  K={K} span {span_us:.1f} us, staged slices {sum(1 for it in items if int(it[3]) != 3)}")

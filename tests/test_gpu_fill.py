"""The device table filler reproduces the host value generator bit for bit."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,E", [("f32", 64), ("f16", 128), ("f32", 36), ("f16", 8)])
@pytest.mark.parametrize("mode", [W.VAL_UNIFORM, W.VAL_INTEGER])
def test_fill_matches_host_generator(dtype, E, mode):
    import torch

    import paper_2507_01676_amd as embx
    for t, m, r0, (lo, hi) in [(0, 1000, 0, (-1.0, 1.0)), (25, 5000, 7_000_000_000 // 2, (-0.05, 0.05)),
                               (3, 1, 12345, (-0.05, 0.05))]:
        seed = W.value_seed(9, t)
        w = torch.empty((m, E), dtype=torch.float16 if dtype == "f16" else torch.float32, device="cuda")
        embx.fill_table(w, t, seed, lo, hi, mode, row_begin=r0)
        got = w.cpu().numpy()
        want = W.table_rows_block(t, r0, r0 + m, E, dtype, seed=seed, lo=lo, hi=hi, mode=mode)
        assert np.array_equal(got.view(np.uint16 if dtype == "f16" else np.uint32),
                              want.view(np.uint16 if dtype == "f16" else np.uint32))

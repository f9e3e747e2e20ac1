"""Shared helpers of the GPU tests: device inputs from the seeded generators and
oracle comparisons (full or on sampled bags)."""
from __future__ import annotations

import sys

import numpy as np

import workloads as W
from oracle import pool as OP

TOL = {"f32": 1e-5, "f16": 2e-3}


def log(msg: str):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def torch_dtype(dtype: str):
    import torch
    return torch.float16 if dtype == "f16" else torch.float32


def host_tables(c: W.Config, mode=W.VAL_UNIFORM):
    return [W.materialize_table(t, m, c.E, c.dtype, seed=c.value_seeds[t], lo=c.lo, hi=c.hi, mode=mode)
            for t, m in enumerate(c.rows)]


def upload_tables(host):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(w)).cuda() for w in host]


def filled_tables(c: W.Config, mode=W.VAL_UNIFORM):
    """Device tables written by the library's table filler (same generator as the host)."""
    import torch

    import paper_2507_01676_amd as embx
    ws = []
    for t, m in enumerate(c.rows):
        w = torch.empty((m, c.E), dtype=torch_dtype(c.dtype), device="cuda")
        embx.fill_table(w, t, c.value_seeds[t], c.lo, c.hi, mode)
        ws.append(w)
    return ws


def to_device(batch: W.Batch):
    import torch
    return torch.from_numpy(batch.indices).cuda(), torch.from_numpy(batch.offsets).cuda()


def plan_for(c: W.Config, B: int, stats=None, **opts):
    import paper_2507_01676_amd as embx
    if stats is None:
        stats = W.history_stats(c, B)
    return embx.Plan(c.rows, c.E, c.dtype, stats, B, **opts)


def check_full(got: np.ndarray, weights_host, batch: W.Batch, dtype: str, exact: bool = False):
    ref, mag, bad = OP.pool_reference(weights_host, batch.indices, batch.offsets, batch.B)
    empty = OP.empty_bag_mask(batch.offsets, len(weights_host), batch.B)
    assert np.all(got[empty] == 0) and not np.any(np.signbit(got[empty])), "empty bags must be +0.0"
    if exact:
        bad_el = np.argwhere(got != ref)
        assert bad_el.size == 0, f"{bad_el.shape[0]} elements differ, first {bad_el[:3].tolist()}"
        return 0.0, bad
    err = OP.pooled_error(got, ref, mag)
    assert err <= TOL[dtype], f"pooled error {err:.3e} > {TOL[dtype]}"
    return err, bad


def check_sampled(c: W.Config, got: np.ndarray, batch: W.Batch, n_bags: int, seed: int,
                  mode=W.VAL_UNIFORM, exact: bool = False, pooling=None, psw=None):
    """Oracle on n_bags random (table, sample) bags; table rows regenerated on the host.
    pooling: None / "sum" / "mean" or one per table; psw: per-lookup weights (all lookups)."""
    g = np.random.default_rng(seed)
    B, T = batch.B, c.T
    tsel = g.integers(0, T, size=n_bags)
    bsel = g.integers(0, B, size=n_bags)
    worst = 0.0
    for t in np.unique(tsel):
        bs = np.unique(bsel[tsel == t])
        lo = batch.offsets[t * B + bs]
        hi = batch.offsets[t * B + bs + 1]
        parts = [batch.indices[a:b] for a, b in zip(lo, hi)]
        idx = np.concatenate(parts) if parts else np.zeros(0, np.int64)
        wk = None if psw is None else np.concatenate([psw[a:b] for a, b in zip(lo, hi)])
        mode_t = pooling if (pooling is None or isinstance(pooling, str)) else pooling[int(t)]
        uniq, inv = np.unique(idx, return_inverse=True)
        vals = W.table_rows_at(int(t), uniq, c.E, c.dtype, seed=c.value_seeds[t], lo=c.lo, hi=c.hi, mode=mode)
        off = np.zeros(bs.size + 1, np.int64)
        np.cumsum(hi - lo, out=off[1:])
        ref, mag, _ = OP.pool_reference([vals], inv.reshape(-1).astype(np.int64), off, bs.size,
                                        pooling=mode_t, psw=wk)
        mine = got[bs, t, :][:, None, :]
        if exact:
            assert np.array_equal(mine, ref), f"table {t}: sampled bags differ"
        else:
            err = OP.pooled_error(mine, ref, mag)
            worst = max(worst, err)
            assert err <= TOL[c.dtype], f"table {t}: pooled error {err:.3e}"
        emp = (hi - lo) == 0
        assert np.all(got[bs[emp], t, :] == 0)
    return worst


def check_index_columns(got: np.ndarray, batch: W.Batch, T: int, rows=None):
    """Every bag of an integer-mode lookup, columns 0-4 only: they are functions of the row
    id alone (1, the three base-2048 digits of the row, the table id + 1), so their sums
    follow from the indices without the tables.  Exact in fp32 at any batch size.
    ``rows`` (per table) marks out-of-range ids, which add nothing."""
    B = batch.B
    for t in range(T):
        lo, hi = batch.offsets[t * B], batch.offsets[(t + 1) * B]
        ids = batch.indices[lo:hi]
        ok = np.ones(ids.size, bool) if rows is None else (ids >= 0) & (ids < rows[t])
        idv = np.where(ok, ids, 0)
        cols = np.stack([ok.astype(np.float64), (idv & 2047) * ok, ((idv >> 11) & 2047) * ok,
                         ((idv >> 22) & 2047) * ok, (t + 1.0) * ok], axis=1).astype(np.float64)
        # per-bag sums as differences of running sums (integers below 2^53: exact)
        csum = np.zeros((ids.size + 1, 5))
        np.cumsum(cols, axis=0, out=csum[1:])
        ends = batch.offsets[t * B:(t + 1) * B + 1] - lo
        want = (csum[ends[1:]] - csum[ends[:-1]]).astype(np.float32)
        mine = got[:, t, :5]
        bad = np.argwhere(mine != want)
        assert bad.size == 0, f"table {t}: {bad.shape[0]} of {B * 5} index-column elements differ, first {bad[:3].tolist()}"

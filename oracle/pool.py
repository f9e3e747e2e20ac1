"""Pooled embedding lookup -- the plain definition (test infrastructure only).

Sec. II-B: for table i with sequence length s_i, every sample of the batch
looks up s_i rows of the m_i x E table and reduces them to one E-vector;
Sec. IV-A fixes the reduction to a sum.  With a table-major CSR batch this is

    out[b, t, :] = sum_{k = offsets[t*B+b]}^{offsets[t*B+b+1]-1}  W_t[indices[k], :]

Sec. II-B names averaging as the other reduction: a mean-pooled table divides
its bag's sum by the bag's length n_bt = offsets[t*B+b+1] - offsets[t*B+b].
Each lookup may also carry a weight w_k (per-sample weights); the bag then sums
w_k * W_t[indices[k], :] (before the division, for a mean-pooled table).

Readings (listed in the design notes): fp16 tables are widened exactly to
float; the sum is accumulated in float64 and rounded once to float32; an index
outside [0, m_t) contributes nothing and is counted, but still counts in n_bt;
an empty bag is +0.0 under either reduction.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


POOLING = ("sum", "mean")


def _modes(pooling, T: int) -> List[str]:
    if pooling is None:
        return ["sum"] * T
    if isinstance(pooling, str):
        pooling = [pooling] * T
    modes = [str(x) for x in pooling]
    assert len(modes) == T and all(x in POOLING for x in modes), modes
    return modes


def pool_reference(weights: Sequence[np.ndarray], indices: np.ndarray, offsets: np.ndarray,
                   batch: int, pooling=None, psw=None) -> Tuple[np.ndarray, np.ndarray, int]:
    """Returns (ref fp32 [B,T,E], mag fp64 [B,T,E], number of out-of-range indices).

    mag is the same reduction applied to |w_k| |x| (the scale of the rounding error).
    Per table: gather the rows (a library gather), scale each by its lookup's weight,
    then sum each bag's rows with ``np.add.reduceat`` over the non-empty bags, in
    float64, and divide by the bag length for a mean-pooled table.  pooling: None (all
    "sum"), one of "sum" / "mean", or one per table; psw: None (all weights 1) or a float
    array aligned with indices.
    """
    T = len(weights)
    B = int(batch)
    indices = np.asarray(indices, dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    assert offsets.shape == (T * B + 1,), (offsets.shape, T, B)
    modes = _modes(pooling, T)
    if psw is not None:
        psw = np.asarray(psw, dtype=np.float64)
        assert psw.shape == (int(offsets[-1]),), (psw.shape, offsets[-1])
    E = int(weights[0].shape[1]) if T else 0
    acc = np.zeros((B, T, E), dtype=np.float64)
    mag = np.zeros((B, T, E), dtype=np.float64)
    bad = 0
    for t in range(T):
        W = weights[t]
        m = W.shape[0]
        lo, hi = int(offsets[t * B]), int(offsets[t * B + B])
        if hi == lo:
            continue
        idx = indices[lo:hi]
        ok = (idx >= 0) & (idx < m)
        bad += int(idx.size - np.count_nonzero(ok))
        rows = np.zeros((idx.size, E), dtype=np.float64)
        rows[ok] = W[idx[ok]].astype(np.float64)
        if psw is not None:
            rows *= psw[lo:hi, None]
        starts = offsets[t * B: t * B + B] - lo
        lens = np.diff(offsets[t * B: t * B + B + 1])
        ne = lens > 0
        # consecutive non-empty bags tile [0, hi-lo) exactly, so reduceat's
        # segment i ends where segment i+1 starts
        acc[ne, t, :] = np.add.reduceat(rows, starts[ne], axis=0)
        mag[ne, t, :] = np.add.reduceat(np.abs(rows), starts[ne], axis=0)
        if modes[t] == "mean":
            acc[ne, t, :] /= lens[ne, None]
            mag[ne, t, :] /= lens[ne, None]
    return acc.astype(np.float32), mag, bad


def pool_loops(weights: Sequence[np.ndarray], indices: Sequence[int], offsets: Sequence[int],
               batch: int, pooling=None, psw=None) -> Tuple[List, int]:
    """The definition as pure-Python loops (tiny inputs only).

    Returns (nested list [B][T][E] of python floats computed in binary64, bad count).
    """
    T = len(weights)
    modes = _modes(pooling, T)
    out = []
    bad = 0
    for b in range(batch):
        row_t = []
        for t in range(T):
            W = weights[t]
            m, E = W.shape
            s = [0.0] * E
            k0, k1 = int(offsets[t * batch + b]), int(offsets[t * batch + b + 1])
            for k in range(k0, k1):
                r = int(indices[k])
                if r < 0 or r >= m:
                    bad += 1
                    continue
                wk = 1.0 if psw is None else float(psw[k])
                for e in range(E):
                    s[e] += wk * float(W[r, e])
            if modes[t] == "mean" and k1 > k0:
                s = [x / (k1 - k0) for x in s]
            row_t.append(s)
        out.append(row_t)
    return out, bad


def pooled_error(got: np.ndarray, ref: np.ndarray, mag: np.ndarray) -> float:
    """max |got - ref| / mag over all elements, with 0/0 := 0.

    Any fp32 summation order of n terms stays within (n-1) * 2**-24 * sum|x|
    of the exact sum (recursive-summation bound, Higham, Accuracy and Stability
    of Numerical Algorithms, Sec. 4.2), so this metric accepts every correct
    order while a missing or wrong row moves a sum by about mag / n.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = np.abs(got - ref)
    with np.errstate(invalid="ignore", divide="ignore"):
        r = np.where(mag > 0, d / np.where(mag > 0, mag, 1.0), np.where(d > 0, np.inf, 0.0))
    return float(r.max()) if r.size else 0.0


def empty_bag_mask(offsets: np.ndarray, T: int, B: int) -> np.ndarray:
    """[B, T] boolean mask of bags with no lookups."""
    lens = np.diff(np.asarray(offsets, dtype=np.int64)).reshape(T, B)
    return (lens == 0).T

"""Pooled embedding lookup -- the plain definition (test infrastructure only).

Sec. II-B: for table i with sequence length s_i, every sample of the batch
looks up s_i rows of the m_i x E table and reduces them to one E-vector;
Sec. IV-A fixes the reduction to a sum.  With a table-major CSR batch this is

    out[b, t, :] = sum_{k = offsets[t*B+b]}^{offsets[t*B+b+1]-1}  W_t[indices[k], :]

Readings (listed in the design notes): fp16 tables are widened exactly to
float; the sum is accumulated in float64 and rounded once to float32; an index
outside [0, m_t) contributes nothing and is counted; an empty bag is +0.0.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def pool_reference(weights: Sequence[np.ndarray], indices: np.ndarray, offsets: np.ndarray,
                   batch: int) -> Tuple[np.ndarray, np.ndarray, int]:
    """Returns (ref fp32 [B,T,E], mag fp64 [B,T,E] = sum |x|, number of out-of-range indices).

    Per table: gather the rows (a library gather), then sum each bag's rows with
    ``np.add.reduceat`` over the non-empty bags, in float64.
    """
    T = len(weights)
    B = int(batch)
    indices = np.asarray(indices, dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    assert offsets.shape == (T * B + 1,), (offsets.shape, T, B)
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
        starts = offsets[t * B: t * B + B] - lo
        lens = np.diff(offsets[t * B: t * B + B + 1])
        ne = lens > 0
        # consecutive non-empty bags tile [0, hi-lo) exactly, so reduceat's
        # segment i ends where segment i+1 starts
        acc[ne, t, :] = np.add.reduceat(rows, starts[ne], axis=0)
        mag[ne, t, :] = np.add.reduceat(np.abs(rows), starts[ne], axis=0)
    return acc.astype(np.float32), mag, bad


def pool_loops(weights: Sequence[np.ndarray], indices: Sequence[int], offsets: Sequence[int],
               batch: int) -> Tuple[List, int]:
    """The definition as pure-Python loops (tiny inputs only).

    Returns (nested list [B][T][E] of python floats summed in binary64, bad count).
    """
    T = len(weights)
    out = []
    bad = 0
    for b in range(batch):
        row_t = []
        for t in range(T):
            W = weights[t]
            m, E = W.shape
            s = [0.0] * E
            for k in range(int(offsets[t * batch + b]), int(offsets[t * batch + b + 1])):
                r = int(indices[k])
                if r < 0 or r >= m:
                    bad += 1
                    continue
                for e in range(E):
                    s[e] += float(W[r, e])
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

"""Index handling of the lookup strategies (test infrastructure only).

All results are exact integers; the GPU side must match them bit for bit.

* ``chunk_local``  -- Sec. III-B: a table split into row chunks sees its indices
  shifted by the chunk's first row; an index outside the chunk must not be
  pooled by that chunk (reading: masked, not clipped onto the boundary row, so
  that every index is pooled exactly once over all chunks).
* ``hot_slots``    -- membership of each index in a table's hot-row set (position
  in the hottest-first list, or -1).
* ``dedup_tile``   -- sorted unique rows of a tile of indices with the inverse
  map and counts (each unique row is fetched once).
* ``range_errors`` -- indices outside [0, m_t).
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np


def chunk_local(idx: np.ndarray, r0: int, r1: int) -> np.ndarray:
    """idx - r0 where r0 <= idx < r1, else -1."""
    idx = np.asarray(idx, dtype=np.int64)
    inside = (idx >= r0) & (idx < r1)
    return np.where(inside, idx - r0, -1)


def chunk_partition_ok(m: int, bounds: Sequence[Tuple[int, int]]) -> bool:
    """True iff the [r0, r1) ranges tile [0, m) in order without gaps or overlap."""
    pos = 0
    for r0, r1 in bounds:
        if r0 != pos or r1 < r0:
            return False
        pos = r1
    return pos == m


def hot_slots(idx: np.ndarray, hot_rows: np.ndarray) -> np.ndarray:
    """Position of each index in ``hot_rows`` (distinct ids), -1 if absent."""
    idx = np.asarray(idx, dtype=np.int64)
    hot_rows = np.asarray(hot_rows, dtype=np.int64)
    if hot_rows.size == 0:
        return np.full(idx.shape, -1, dtype=np.int64)
    order = np.argsort(hot_rows, kind="stable")
    srt = hot_rows[order]
    pos = np.searchsorted(srt, idx)
    pos_c = np.minimum(pos, srt.size - 1)
    hit = np.isin(idx, hot_rows) & (srt[pos_c] == idx)
    return np.where(hit, order[pos_c], -1)


def dedup_tile(idx: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(sorted unique rows, inverse map, counts) of one tile of indices."""
    u, inv, cnt = np.unique(np.asarray(idx, dtype=np.int64), return_inverse=True, return_counts=True)
    return u, inv.reshape(-1), cnt


def range_errors(indices: np.ndarray, offsets: np.ndarray, rows: Sequence[int], batch: int) -> int:
    """Number of indices outside [0, rows[t]) of their table."""
    T = len(rows)
    bad = 0
    for t in range(T):
        lo, hi = int(offsets[t * batch]), int(offsets[(t + 1) * batch])
        x = np.asarray(indices[lo:hi], dtype=np.int64)
        bad += int(np.count_nonzero((x < 0) | (x >= rows[t])))
    return bad

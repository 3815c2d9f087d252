"""Expected dispatch plan (test infrastructure only).

The layer evaluates only the experts indexed by the active set (Alg. 1's
online loop); a dispatch groups the kept (expert, token) pairs by expert.  The
plan is defined here by sorting: counts per expert, their exclusive prefix
sum, and the token of every kept pair in (expert ascending, token ascending)
order.
"""
from __future__ import annotations

import numpy as np


def dispatch_plan(topk_idx, keep, N: int):
    idx = np.asarray(topk_idx, dtype=np.int64)
    keep = np.asarray(keep, dtype=bool)
    T, k = idx.shape
    pairs = sorted((int(idx[t, i]), t, i) for t in range(T) for i in range(k) if keep[t, i])
    counts = np.zeros(N, dtype=np.int64)
    for e, _, _ in pairs:
        counts[e] += 1
    offsets = np.zeros(N + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    perm = np.array([t for _, t, _ in pairs], dtype=np.int64)
    slot_row = np.full((T, k), -1, dtype=np.int64)
    for r, (_, t, i) in enumerate(pairs):
        slot_row[t, i] = r
    return dict(counts=counts, offsets=offsets, perm=perm, slot_row=slot_row)

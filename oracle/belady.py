"""Optimal-replacement bounds for the demand sequence of one layer.

Not part of the paper: a yardstick for its LRU (Sec. 3.1) and LFU (Sec. 4.2)
caches.  The demand sequence of a layer is its tokens' selected experts
flattened in rank order.  Belady's MIN evicts the resident expert whose next
use lies furthest ahead (an expert never used again first; ties between those
go to the lower id).  MIN is optimal among demand-paging caches, so LRU and
LFU (with or without the whole-token pinning, which is only a restriction)
never score more hits on the same sequence and the same start state.
"""
from __future__ import annotations

from functools import lru_cache
from typing import Iterable, Sequence

INF = float("inf")


def flatten(ids_per_token: Iterable[Sequence[int]]):
    return [int(e) for row in ids_per_token for e in row]


def min_hits(seq: Sequence[int], slots: int, initial: Sequence[int]) -> int:
    """Hits of Belady's MIN on `seq` from resident set `initial` (-1 = empty)."""
    seq = [int(e) for e in seq]
    resident = {e for e in initial if e >= 0}
    hits = 0
    for i, x in enumerate(seq):
        if x in resident:
            hits += 1
            continue
        if len(resident) < slots:
            resident.add(x)
            continue

        def next_use(e):
            for j in range(i + 1, len(seq)):
                if seq[j] == e:
                    return j
            return INF

        victim = max(resident, key=lambda e: (next_use(e), -e))
        resident.remove(victim)
        resident.add(x)
    return hits


def exhaustive_max_hits(seq: Sequence[int], slots: int, initial: Sequence[int]) -> int:
    """Maximum hits over every demand-paging eviction choice (tiny inputs only)."""
    seq = tuple(int(e) for e in seq)

    @lru_cache(maxsize=None)
    def best(i, resident):
        if i == len(seq):
            return 0
        x = seq[i]
        if x in resident:
            return 1 + best(i + 1, resident)
        if len(resident) < slots:
            return best(i + 1, resident | {x})
        return max(best(i + 1, (resident - {v}) | {x}) for v in resident)

    return best(0, frozenset(e for e in initial if e >= 0))

"""KV budget under recovery: least-recently-used session eviction (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Sec. III-A (state management): the state plane keeps each session's recent-use
time; in recovery, when the KV the new layout needs exceeds the memory
budget, cold sessions are released least recently used first until the
demand fits, and evicted sessions are rebuilt later by replay.

Readings used here:
  * a session is one row of the block table; its demand is the set of live
    block ids in that row (a block shared by several rows counts once);
  * the demand in bytes is (distinct live blocks of the kept rows) x (bytes
    one block occupies in the new layout, over all layers, K and V);
  * sessions are evicted in ascending (last_use, session id) order (ties:
    the lower id goes first) until the demand is within the budget; if even
    no session fits, all are evicted;
  * an evicted row becomes all -1 in the new table; with compaction a kept
    block id p becomes its rank among the kept live ids (ascending), which
    is where it lives in a compact new arena.
"""
from __future__ import annotations

import numpy as np


def demand_blocks(table: np.ndarray, rows) -> int:
    """Distinct live block ids in the given rows of the table."""
    ids = set()
    for s in rows:
        ids.update(int(p) for p in table[s] if p >= 0)
    return len(ids)


def lru_keep(table: np.ndarray, last_use, block_bytes: int, budget: int) -> np.ndarray:
    """Boolean keep flag per session, by evicting the coldest one at a time."""
    n = table.shape[0]
    keep = np.ones(n, dtype=bool)
    for s in sorted(range(n), key=lambda s: (int(last_use[s]), s)):
        if demand_blocks(table, np.flatnonzero(keep)) * block_bytes <= budget:
            break
        keep[s] = False
    return keep


def evicted_table(table: np.ndarray, keep: np.ndarray, compact: bool) -> np.ndarray:
    """The block table after eviction (and, if asked, renumbered to ranks)."""
    out = np.where(keep[:, None], table, -1).astype(np.int32)
    if compact:
        ids = np.unique(out[out >= 0])
        rank = {int(p): r for r, p in enumerate(ids)}
        out = np.vectorize(lambda p: rank[int(p)] if p >= 0 else -1, otypes=[np.int32])(out)
    return out

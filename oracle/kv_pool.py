"""Plain reference of the KV-pool contraction (TEST INFRASTRUCTURE: only
tests/ and bench.py's CPU leg may use it; the library shares no code with it).

Sec. 6.4 of the paper, Steps 1-5, for a pool whose physical blocks
[k_boundary, k_total) are being reclaimed:

1. scan the block tables of the active sequences for blocks with an id at or
   above the boundary (each distinct block once, in the order met);
2. check that the free list holds enough blocks below the boundary and build a
   one-to-one map old -> new onto them (taken in the free list's order);
3. rewrite the tables through the map;
4. copy each moved block's keys and values, in every layer, to its new id;
5. trim the allocator: drop the ids at or above the boundary from the free
   list, and the blocks just taken.
If there are too few free blocks below the boundary nothing changes and the
contraction is deferred (the paper's drain-aware contraction).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np


class Deferred(Exception):
    """Too few free blocks below the boundary for the live blocks above it."""


def contraction_plan(block_table: np.ndarray, free_list: Sequence[int], k_boundary: int) -> Dict:
    table = np.array(block_table, dtype=np.int64, copy=True)
    # Step 1
    evict: List[int] = []
    for b in range(table.shape[0]):
        for j in range(table.shape[1]):
            blk = int(table[b, j])
            if blk >= k_boundary and blk not in evict:
                evict.append(blk)
    # Step 2
    below = [int(f) for f in free_list if f < k_boundary]
    if len(below) < len(evict):
        raise Deferred(f"{len(evict)} live blocks above the boundary, {len(below)} free below it")
    mapping = {old: below[i] for i, old in enumerate(evict)}
    # Step 3
    for b in range(table.shape[0]):
        for j in range(table.shape[1]):
            blk = int(table[b, j])
            if blk in mapping:
                table[b, j] = mapping[blk]
    # Step 5
    taken = set(mapping.values())
    new_free = [int(f) for f in free_list if f < k_boundary and f not in taken]
    return {"src": evict, "dst": [mapping[o] for o in evict], "table": table.astype(np.int32), "free": new_free}


def migrate(k_pages: Sequence[np.ndarray], v_pages: Sequence[np.ndarray], src: Sequence[int], dst: Sequence[int]):
    """Step 4: copies of the pages with block src[i] copied onto dst[i] in every layer."""
    kp = [np.array(a, copy=True) for a in k_pages]
    vp = [np.array(a, copy=True) for a in v_pages]
    for s, d in zip(src, dst):
        for l in range(len(kp)):
            kp[l][d] = k_pages[l][s]
            vp[l][d] = v_pages[l][s]
    return kp, vp

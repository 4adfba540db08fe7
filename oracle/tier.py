"""Eviction plan of the layered context store (reference).

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the product package.

What it computes
----------------
Paper section 3.2.2 ("Layered Storage of Action Context") keeps frequently used
context in GPU memory and, for rarely used data, either recomputes it on demand
or moves it to CPU memory; section 3.2.3 ("Auto Eviction") combines
least-recently-used order with priorities: when GPU memory runs short, the
objects with the smallest effect on outcomes or the lowest cost to recompute go
first, and the least used part moves to CPU memory (vision K/V, cheap to
recompute, is evicted first).  The paper gives no formula.  Reading taken here
for rows of a context (the unit the store evicts):

* every resident row r has a priority p_r (lower = evicted earlier), the tick
  of its last use t_r, the pages it holds n_r, and a flag d_r saying its
  context may be dropped and recomputed from inputs the caller keeps;
* to free P pages, the unpinned resident rows are taken in increasing
  (p_r, t_r, r) -- priority first, least recently used within a priority,
  row index on ties -- until the pages taken reach P; a taken row is dropped
  (recomputed later) when d_r is set and offloaded to host memory otherwise;
* if all candidates together hold fewer than P pages, every candidate is taken
  and the plan reports the shortfall.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

KEEP, OFFLOAD, DROP = 0, 1, 2


def eviction_plan(priority: Sequence[int], last_use: Sequence[int], pages: Sequence[int],
                  droppable: Sequence[bool], resident: Sequence[bool], pinned: Sequence[bool],
                  pages_needed: int) -> Tuple[List[int], int]:
    """Returns (action per row, pages freed)."""
    n = len(priority)
    action = [KEEP] * n
    if pages_needed <= 0:
        return action, 0
    order = sorted((r for r in range(n) if resident[r] and not pinned[r]),
                   key=lambda r: (priority[r], last_use[r], r))
    freed = 0
    for r in order:
        if freed >= pages_needed:
            break
        action[r] = DROP if droppable[r] else OFFLOAD
        freed += pages[r]
    return action, freed

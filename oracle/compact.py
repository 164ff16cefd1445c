"""Storage order of the pruned cache (the "prune" of Algorithm 1).

Test infrastructure only (see ``oracle/__init__``).

Algorithm 1 replaces the cache by the kept set C'_t, and Sec. 3.3 only asks
that |C'_t| <= B; the paper fixes no order for the rows of the pruned cache.
Reading used here ("hole filling"): with L rows in slots 0..L-1 and
B' = min(B, L) kept rows, the pruned cache occupies slots 0..B'-1, and

* a kept row whose slot is below B' stays in that slot;
* the slots below B' that held evicted rows (the holes), taken in ascending
  order, receive the kept rows from slots B'..L-1, taken in ascending order.

This is the layout with the fewest moved rows (every kept row at a slot >= B'
has to move, and no other row does), and among those layouts the only one that
keeps the movers in their old relative order.  The kept set itself does not
depend on it: ties are broken by token position, not by slot.

Parity pinned by: brute force over every bijection of the kept set onto the
first B' slots for tiny L (the layout is the unique order-preserving one of
minimal moves), the fixed points and the bijection property on random masks,
and the closed forms of the single eviction (slot e < B' takes the row of slot
B') and of evictions that all lie at or above B' (identity).
"""
from __future__ import annotations

import numpy as np


def hole_fill(kept_rows, n_rows: int) -> np.ndarray:
    """Slot map of the pruned cache: entry j is the old slot whose row occupies
    new slot j.  ``kept_rows`` is the set of kept old slots (any order, no
    repeats); its size is B' = min(B, L)."""
    kept = np.unique(np.asarray(kept_rows, np.int64))
    if len(kept) != len(np.asarray(kept_rows).ravel()):
        raise ValueError("kept rows repeat")
    if len(kept) and (kept[0] < 0 or kept[-1] >= n_rows):
        raise ValueError("kept row outside the cache")
    nb = len(kept)
    is_kept = np.zeros(n_rows, bool)
    is_kept[kept] = True
    slot_map = np.arange(nb, dtype=np.int64)
    holes = [j for j in range(nb) if not is_kept[j]]
    movers = [i for i in range(nb, n_rows) if is_kept[i]]
    assert len(holes) == len(movers)
    for h, m in zip(holes, movers):
        slot_map[h] = m
    return slot_map

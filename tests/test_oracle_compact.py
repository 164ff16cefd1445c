"""CPU pins of the oracle's pruned-cache storage order (oracle/compact.py):
brute force over every layout on tiny caches, closed forms, and the unit step
carrying every row's state through the slot map."""
import itertools

import numpy as np
import pytest

from oracle import compact, unit


def _minimal_order_preserving_layouts(kept, n_rows):
    """Every bijection of the kept set onto slots 0..B'-1 with the fewest rows
    that change slot and the moved rows in ascending old order."""
    nb = len(kept)
    best, found = None, []
    for perm in itertools.permutations(kept):
        moved = [j for j in range(nb) if perm[j] != j]
        cost = len(moved)
        movers = [perm[j] for j in moved]
        if movers != sorted(movers):
            continue
        if best is None or cost < best:
            best, found = cost, [perm]
        elif cost == best:
            found.append(perm)
    return best, found


@pytest.mark.parametrize("n_rows", [1, 2, 3, 4, 5, 6])
def test_hole_fill_is_the_unique_minimal_order_preserving_layout(n_rows):
    for nb in range(1, n_rows + 1):
        for kept in itertools.combinations(range(n_rows), nb):
            cost, layouts = _minimal_order_preserving_layouts(list(kept), n_rows)
            assert len(layouts) == 1, (kept, layouts)
            got = compact.hole_fill(kept, n_rows)
            assert tuple(got.tolist()) == layouts[0]
            # the minimum is the number of kept rows that sit at or above B'
            assert cost == sum(1 for i in kept if i >= nb)


def test_hole_fill_on_random_masks():
    r = np.random.default_rng(11)
    for _ in range(200):
        L = int(r.integers(1, 400))
        nb = int(r.integers(1, L + 1))
        kept = np.sort(r.choice(L, nb, replace=False))
        sm = compact.hole_fill(r.permutation(kept), L)          # input order does not matter
        assert np.array_equal(np.sort(sm), kept)                  # a bijection onto the kept set
        below = kept[kept < nb]
        assert np.array_equal(sm[below], below)                   # kept rows below B' stay
        moved = np.nonzero(sm != np.arange(nb))[0]
        assert np.all(sm[moved] >= nb) and np.all(np.diff(sm[moved]) > 0)
        assert len(moved) == int((kept >= nb).sum())


def test_hole_fill_closed_forms():
    # one eviction below the budget: the hole takes the last row
    for B, e in ((8, 0), (8, 3), (8, 7), (4096, 1234)):
        kept = np.delete(np.arange(B + 1), e)
        sm = compact.hole_fill(kept, B + 1)
        want = np.arange(B)
        want[e] = B
        assert np.array_equal(sm, want)
    # the newest row evicted, or every evicted row at or above B': identity
    assert np.array_equal(compact.hole_fill(np.arange(10), 11), np.arange(10))
    assert np.array_equal(compact.hole_fill(np.arange(6), 40), np.arange(6))
    # a whole block evicted at the front: the rows after it fill it in order
    sm = compact.hole_fill(np.arange(3, 10), 10)
    assert np.array_equal(sm, [7, 8, 9, 3, 4, 5, 6])


def test_hole_fill_rejects_bad_sets():
    with pytest.raises(ValueError):
        compact.hole_fill([1, 1, 2], 5)
    with pytest.raises(ValueError):
        compact.hole_fill([0, 5], 5)


def test_unit_evict_stores_rows_in_the_hole_fill_order():
    r = np.random.default_rng(4)
    L, d, G = 50, 8, 2
    st = unit.new_student(r.normal(size=(L, d)), r.normal(size=(L, d)), np.arange(L), G=G, scale=0.3)
    for t in range(3):
        unit.decode_step(st, r.normal(size=(G, d)), r.normal(size=d), r.normal(size=d))
        pos_before = st.pos.copy()
        s = r.normal(size=st.L)
        sm = unit.evict(st, s, 20 + t)
        kept_set = np.sort(np.argsort(-s, kind="stable")[:20 + t])
        assert np.array_equal(np.sort(sm), kept_set)
        assert np.array_equal(sm, compact.hole_fill(kept_set, len(pos_before)))
        assert np.array_equal(st.pos, pos_before[sm])

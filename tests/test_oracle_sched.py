"""Pins of the oracle's bit-width-aware I/O planning (Sec. 3.4): the
Hottest-Expert-Bit-First order (Sec. 3.4.3) and the memory-budget scheduler
(Algorithm 2, Sec. 3.4.1), by hand-worked cases from the text and by
properties read off the outputs (not by re-running the same steps)."""
import numpy as np
import pytest

from oracle import oracle as O


def test_hebf_nested_reuse_example():
    """The text's example: three requests select expert 2, one at INT2 and two
    at INT3; all three use the INT2 planes and the two INT3 requests add one
    plane on top.  With expert 0 holding one INT4 request, the first heads
    are e0@4 and e2@2 with one request each: the tie goes to the lower
    expert; then expert 2's units in ascending width, INT3 loading only the
    plane it adds."""
    B = np.zeros((3, 7), int)
    B[2, 0], B[2, 1] = 1, 2          # expert 2: one INT2, two INT3
    B[0, 2] = 1                      # expert 0: one INT4
    assert O.hebf_order(B, 2) == [(0, 4, 0, 4, 1), (2, 2, 0, 2, 1), (2, 3, 2, 3, 2)]


def test_hebf_hand_worked():
    """Heads and counts by hand: queues e0 [2:1, 4:3, 8:2], e1 [3:5], e2 [2:2, 3:2].
    Heads 1, 5, 2 -> e1@3 (5); heads 1, 2 -> e2@2 (2); heads 1, 2 -> e2@3 (2);
    then e0: @2 (1), @4 (3), @8 (2).  Loads are the nested deltas."""
    B = np.array([[1, 0, 3, 0, 0, 0, 2], [0, 5, 0, 0, 0, 0, 0], [2, 2, 0, 0, 0, 0, 0]])
    assert O.hebf_order(B, 2) == [(1, 3, 0, 3, 5), (2, 2, 0, 2, 2), (2, 3, 2, 3, 2),
                                  (0, 2, 0, 2, 1), (0, 4, 2, 4, 3), (0, 8, 4, 8, 2)]
    # expert 1 already holds 5 bits: its unit loads nothing
    assert O.hebf_order(B, 2, [0, 5, 0])[0] == (1, 3, 5, 5, 5)


@pytest.mark.parametrize("seed", range(20))
def test_hebf_properties(seed):
    rng = np.random.default_rng(seed)
    E, L, b_min = int(rng.integers(1, 12)), int(rng.integers(1, 8)), int(rng.integers(1, 3))
    B = rng.integers(0, 5, (E, L))
    B[rng.random((E, L)) < 0.4] = 0
    res = [0 if rng.random() < 0.6 else int(rng.integers(b_min, b_min + L)) for _ in range(E)]
    order = O.hebf_order(B, b_min, res)
    # every nonempty bucket exactly once, with its count
    assert sorted((j, b) for j, b, *_ in order) == sorted(
        (j, b_min + k) for j in range(E) for k in range(L) if B[j, k] > 0)
    assert all(c == B[j, b - b_min] for j, b, _, _, c in order)
    # per expert: ascending widths (constraint 6b), loads chained from the
    # resident width, and the deltas cover exactly (resident, max width]
    for j in range(E):
        mine = [u for u in order if u[0] == j]
        assert [u[1] for u in mine] == sorted(u[1] for u in mine)
        have = res[j]
        for _, b, frm, to, _ in mine:
            assert frm == have and to == max(have, b)
            have = to
    # hottest first: when a unit is emitted, no other expert's next unit has
    # a larger count (or an equal one at a lower expert index)
    for i, (j, b, _, _, c) in enumerate(order):
        for j2 in range(E):
            nxt = next((u for u in order[i:] if u[0] == j2), None)
            if nxt is None or j2 == j:
                continue
            assert nxt[4] < c or (nxt[4] == c and j2 > j)


def test_budget_hand_worked():
    """Two layers of two experts, levels of 10 / 4 / 4 bytes, budget 40.
    Layer 0 wants 3 and 2 levels (18 + 14 = 32 bytes): fits.  Layer 1 wants
    3 and 1 levels (18 + 10 = 28): 8 free, so layer 0's top level goes first
    (expert 0's level 2: 12 free), then level 1 of both (20), then the base
    level of both (40 >= 28); then layer 1 loads."""
    lb = [10, 4, 4]
    acts, res = O.budget_plan([[3, 2], [3, 1]], lb, 40)
    assert acts == [("load", 0, 0, 0), ("load", 0, 0, 1), ("load", 0, 0, 2),
                    ("load", 0, 1, 0), ("load", 0, 1, 1),
                    ("free", 0, 0, 2), ("free", 0, 0, 1), ("free", 0, 1, 1),
                    ("free", 0, 0, 0), ("free", 0, 1, 0),
                    ("load", 1, 0, 0), ("load", 1, 0, 1), ("load", 1, 0, 2),
                    ("load", 1, 1, 0)]
    assert res.tolist() == [[0, 0], [3, 1]]


@pytest.mark.parametrize("seed", range(30))
def test_budget_properties(seed):
    """Replaying the plan: loads go bottom up and frees take an expert's top
    level; a layer being loaded gets every level it wants; frees come only
    from earlier layers, the nearest layer first and its highest level
    first; each batch of frees (one level of one layer) happens only while
    the load does not fit yet; and after every layer the budget holds (here
    every layer alone fits the budget)."""
    rng = np.random.default_rng(100 + seed)
    nl, E, K = int(rng.integers(1, 7)), int(rng.integers(1, 6)), int(rng.integers(1, 8))
    lb = rng.integers(1, 50, K)
    want = rng.integers(0, K + 1, (nl, E))
    largest = max(sum(int(lb[:w].sum()) for w in row) for row in want)
    budget = int(largest + rng.integers(0, 3 * largest + 1))
    acts, res = O.budget_plan(want, lb, budget)
    state = np.zeros((nl, E), int)
    used = 0
    i = 0
    for j in range(nl):
        need = sum(int(lb[state[j, e]:want[j, e]].sum()) for e in range(E))
        last = (j, K)                                # (layer, level) of the last free batch
        while i < len(acts) and acts[i][0] == "free":
            _, jj, e, l = acts[i]
            assert jj < j
            assert (jj, l) == last or jj < last[0] or (jj == last[0] and l < last[1])
            if (jj, l) != last:
                assert used + need > budget          # a new batch only while it does not fit
                last = (jj, l)
            assert l == state[jj, e] - 1
            state[jj, e] -= 1
            used -= lb[l]
            i += 1
        while i < len(acts) and acts[i][0] == "load" and acts[i][1] == j:
            _, _, e, l = acts[i]
            assert l == state[j, e]
            state[j, e] += 1
            used += lb[l]
            i += 1
        assert np.all(state[j] >= want[j])
        assert used <= budget
    assert i == len(acts)
    assert np.array_equal(state, res)


def test_budget_unbounded_only_loads():
    want = np.array([[3, 0, 7], [1, 2, 2]])
    acts, res = O.budget_plan(want, [5, 1, 1, 1, 1, 1, 1], 10 ** 9)
    assert all(a[0] == "load" for a in acts) and len(acts) == want.sum()
    assert np.array_equal(res, want)

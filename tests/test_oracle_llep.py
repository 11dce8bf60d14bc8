"""Pins of the least-loaded plan oracle (oracle/llep.py): conservation,
contiguous windows, the capacity bound, the balanced case, hand-worked
plans, and a brute-force check that no plan can have a smaller largest
load (Sec. 3.3, the recap of LLEP)."""
import itertools

import numpy as np
import pytest

from oracle import llep as OL


def _check_plan(counts, E_p, capacity, lo, hi, load, n_ship):
    counts = np.asarray(counts, np.int64)
    E = len(counts)
    G = E // E_p
    total = int(counts.sum())
    C = max(capacity, -(-total // E_p))
    sizes = hi - lo
    assert np.all(sizes >= 0)
    # every assignment of every expert is computed exactly once
    assert np.array_equal(sizes.sum(axis=0), counts)
    # the windows of an expert tile [0, n_e) without gaps or overlaps
    for e in range(E):
        w = sorted((lo[r, e], hi[r, e]) for r in range(E_p) if hi[r, e] > lo[r, e])
        pos = 0
        for a, b in w:
            assert a == pos
            pos = b
        assert pos == counts[e]
        # the home rank's window (if any) starts at row 0
        home = e // G
        if hi[home, e] > lo[home, e]:
            assert lo[home, e] == 0
    assert np.array_equal(load, sizes.sum(axis=1))
    assert load.max() <= C
    ships = sum(1 for r in range(E_p) for e in range(E) if hi[r, e] > lo[r, e] and e // G != r)
    assert ships == n_ship


def test_balanced_load_moves_nothing():
    counts = [5, 3, 4, 4, 2, 6, 1, 7]  # two ranks of 16 each
    lo, hi, load, ns = OL.llep_plan(counts, 2)
    assert ns == 0 and list(load) == [16, 16]
    assert np.array_equal(hi[0, :4], counts[:4]) and np.array_equal(hi[1, 4:], counts[4:])
    assert np.all(hi[0, 4:] == 0) and np.all(hi[1, :4] == 0)


def test_hand_worked_plan():
    # E = 4 on 2 ranks, total 12, C = 6.  Rank 0 keeps 6 rows of e0 (spill
    # 4) and nothing of the empty e1; rank 1 keeps e2 and e3 (load 2).  The
    # spill of e0 goes to the least loaded rank 1, whose room is 4.
    counts = [10, 0, 1, 1]
    lo, hi, load, ns = OL.llep_plan(counts, 2)
    assert (lo[0, 0], hi[0, 0]) == (0, 6)
    assert (lo[1, 0], hi[1, 0]) == (6, 10)
    assert list(load) == [6, 6] and ns == 1


def test_hand_worked_spill_order_and_least_loaded_target():
    # 3 ranks x 2 experts, counts 9 1 | 2 0 | 0 0: total 12, C = 4.
    # keep: r0 keeps e0 4 (spill 5), e1 0 (spill 1); r1 keeps e2 2; r2 nothing.
    # spill order: e0 (5) then e1 (1).  e0: least loaded r2 (0) takes 4 ->
    # load 4; then r1 (2) takes 1 -> 3.  e1: least loaded r1 (3) takes 1 -> 4.
    counts = [9, 1, 2, 0, 0, 0]
    lo, hi, load, ns = OL.llep_plan(counts, 3)
    assert (lo[0, 0], hi[0, 0]) == (0, 4)
    assert (lo[2, 0], hi[2, 0]) == (4, 8)
    assert (lo[1, 0], hi[1, 0]) == (8, 9)
    assert (lo[1, 1], hi[1, 1]) == (0, 1)
    assert hi[0, 1] == 0
    assert list(load) == [4, 4, 4] and ns == 3


def test_capacity_above_the_mean_moves_less():
    counts = [30, 2, 2, 2, 2, 2, 2, 2]  # 4 ranks, total 44, mean 11
    _, _, load_tight, ns_tight = OL.llep_plan(counts, 4)
    _, _, load_loose, ns_loose = OL.llep_plan(counts, 4, capacity=20)
    assert load_tight.max() == 11 and load_loose.max() == 20
    assert ns_loose <= ns_tight


@pytest.mark.parametrize("seed", range(20))
def test_random_plans_satisfy_the_invariants(seed):
    rng = np.random.default_rng(seed)
    E_p = int(rng.choice([1, 2, 3, 4, 8]))
    G = int(rng.integers(1, 6))
    E = E_p * G
    counts = rng.zipf(1.3, E).clip(max=500) * rng.integers(0, 2, E)
    capacity = int(rng.integers(0, 2)) * int(counts.sum() // max(E_p, 1) + rng.integers(0, 50))
    lo, hi, load, ns = OL.llep_plan(counts, E_p, capacity)
    _check_plan(counts, E_p, capacity, lo, hi, load, ns)


def test_largest_load_is_optimal_by_brute_force():
    # with unrestricted splitting the best possible largest load is
    # ceil(total / E_p); brute force over all splits of tiny cases confirms
    # that no plan does better, and the greedy reaches it
    for counts, E_p in (([3, 0, 1, 2], 2), ([4, 1, 0, 0, 0, 0], 3), ([2, 2, 1, 0], 4)):
        total = sum(counts)
        best = None
        # assign each unit of each expert to a rank
        units = [e for e, c in enumerate(counts) for _ in range(c)]
        for assign in itertools.product(range(E_p), repeat=len(units)):
            loads = np.bincount(np.array(assign, int), minlength=E_p)
            m = int(loads.max())
            best = m if best is None else min(best, m)
        assert best == -(-total // E_p)
        _, _, load, _ = OL.llep_plan(counts, E_p)
        assert int(load.max()) == best


def test_rank_rows_partition_the_assignments():
    rng = np.random.default_rng(3)
    T, k, E, E_p = 40, 3, 8, 4
    idx = np.stack([rng.choice(E, k, replace=False) for _ in range(T)])
    counts = np.bincount(idx.reshape(-1), minlength=E)
    lo, hi, load, _ = OL.llep_plan(counts, E_p)
    seen = []
    for r in range(E_p):
        off, rows = OL.rank_rows(idx, lo, hi, r)
        assert off[-1] == load[r] == len(rows)
        for e in range(E):
            seg = rows[off[e]:off[e + 1]]
            assert np.all(idx.reshape(-1)[seg] == e)
            assert np.all(np.diff(seg) > 0)  # stable order inside a window
        seen.extend(rows.tolist())
    assert sorted(seen) == list(range(T * k))


# ---- the plan in units of g rows (g = the grouped GEMM's row-tile height)

def _units(w, g):
    return -(-np.asarray(w, np.int64) // g)


def _check_granular(counts, E_p, capacity, g, lo, hi, load, n_ship):
    counts = np.asarray(counts, np.int64)
    sizes = hi - lo
    # the row-level invariants hold for any granule
    assert np.array_equal(sizes.sum(axis=0), counts)
    assert np.array_equal(load, sizes.sum(axis=1))
    E = len(counts)
    for r in range(E_p):
        for e in range(E):
            if sizes[r, e] > 0:
                # no window splits a unit: it starts on a multiple of g and
                # ends on one or at the expert's last row
                assert lo[r, e] % g == 0
                assert hi[r, e] % g == 0 or hi[r, e] == counts[e]
    U = int(_units(counts, g).sum())
    C = max(-(-capacity // g), -(-U // E_p))
    unit_load = _units(sizes, g).sum(axis=1)
    assert unit_load.sum() == U  # no unit is cut in two
    assert unit_load.max() <= C


def test_granule_one_is_the_row_plan():
    rng = np.random.default_rng(11)
    for _ in range(10):
        counts = rng.zipf(1.3, 12).clip(max=300) * rng.integers(0, 2, 12)
        a = OL.llep_plan(counts, 4)
        b = OL.llep_plan(counts, 4, 0, 1)
        for x, y in zip(a[:3], b[:3]):
            assert np.array_equal(x, y)
        assert a[3] == b[3]


def test_hand_worked_granular_plan():
    # g = 4, E = 4 on 2 ranks, counts 5 5 | 1 1: units 2 2 | 1 1, U = 6,
    # C = 3.  Rank 0 keeps e0 (2 units, 5 rows) and 1 unit (4 rows) of e1,
    # whose last unit (1 row) spills; rank 1 keeps e2 and e3 (2 units).  The
    # spill goes to the least loaded rank 1: rows [4, 5) of e1.
    lo, hi, load, ns = OL.llep_plan([5, 5, 1, 1], 2, 0, 4)
    assert (lo[0, 0], hi[0, 0]) == (0, 5) and (lo[0, 1], hi[0, 1]) == (0, 4)
    assert (lo[1, 1], hi[1, 1]) == (4, 5)
    assert (hi[1, 2], hi[1, 3]) == (1, 1)
    assert list(load) == [9, 3] and ns == 1
    # the row plan (g = 1) balances rows instead: 6 and 6
    _, _, load1, _ = OL.llep_plan([5, 5, 1, 1], 2)
    assert list(load1) == [6, 6]


def test_hand_worked_granular_spill_in_several_pieces():
    # g = 2, 3 ranks x 1 expert, counts 11 | 0 | 0: units 6, C = 2.  Rank 0
    # keeps 2 units (rows 0..3); the 4 spilled units go to rank 1 (2 units:
    # rows 4..7), then rank 2 (rows 8..10, the last unit holds one row).
    lo, hi, load, ns = OL.llep_plan([11, 0, 0], 3, 0, 2)
    assert (lo[0, 0], hi[0, 0]) == (0, 4)
    assert (lo[1, 0], hi[1, 0]) == (4, 8)
    assert (lo[2, 0], hi[2, 0]) == (8, 11)
    assert list(load) == [4, 4, 3] and ns == 2


@pytest.mark.parametrize("seed", range(20))
def test_random_granular_plans_satisfy_the_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    E_p = int(rng.choice([1, 2, 3, 4, 8]))
    G = int(rng.integers(1, 6))
    E = E_p * G
    g = int(rng.choice([1, 2, 3, 7, 16, 256]))
    counts = rng.zipf(1.3, E).clip(max=900) * rng.integers(0, 2, E)
    capacity = int(rng.integers(0, 2)) * int(counts.sum() // max(E_p, 1) + rng.integers(0, 50))
    lo, hi, load, ns = OL.llep_plan(counts, E_p, capacity, g)
    _check_granular(counts, E_p, capacity, g, lo, hi, load, ns)
    # and the row-level structure (contiguous windows from the home rank)
    for e in range(E):
        w = sorted((lo[r, e], hi[r, e]) for r in range(E_p) if hi[r, e] > lo[r, e])
        pos = 0
        for a, b in w:
            assert a == pos
            pos = b
        assert pos == counts[e]
        if hi[e // G, e] > lo[e // G, e]:
            assert lo[e // G, e] == 0


def _splits(n, parts):
    """Every way of dealing n rows to `parts` ranks (counts per rank)."""
    if parts == 1:
        yield (n,)
        return
    for a in range(n + 1):
        for rest in _splits(n - a, parts - 1):
            yield (a,) + rest


def test_granular_largest_load_is_optimal_by_brute_force():
    # A window of w rows costs ceil(w / g) tiles, so any plan's tile total is
    # at least U = sum ceil(n_e / g) and its largest tile load at least
    # ceil(U / E_p).  Brute force over every way of dealing each expert's
    # rows to the ranks confirms that bound is the optimum on tiny cases,
    # and the granular plan reaches it.
    for counts, E_p, g in (([5, 5, 1, 1], 2, 4), ([7, 0, 2, 3], 2, 3), ([4, 1, 0, 2, 0, 0], 3, 2),
                           ([6, 3, 3], 3, 2), ([9, 0, 0, 0], 4, 4)):
        per_expert = [list(_splits(c, E_p)) for c in counts]
        best = None
        for deal in itertools.product(*per_expert):
            tl = [sum(-(-deal[e][r] // g) for e in range(len(counts))) for r in range(E_p)]
            m = max(tl)
            best = m if best is None else min(best, m)
        U = sum(-(-c // g) for c in counts)
        assert best == -(-U // E_p)
        lo, hi, _, _ = OL.llep_plan(counts, E_p, 0, g)
        assert int(_units(hi - lo, g).sum(axis=1).max()) == best


def test_granular_plan_never_has_more_tiles_than_the_row_plan():
    rng = np.random.default_rng(5)
    for _ in range(30):
        E_p = int(rng.choice([2, 4, 8]))
        E = E_p * int(rng.integers(2, 17))
        counts = rng.zipf(1.2, E).clip(max=20000) * rng.integers(0, 2, E) + rng.integers(0, 400, E)
        g = 256
        lo1, hi1, _, _ = OL.llep_plan(counts, E_p)
        log, hig, _, _ = OL.llep_plan(counts, E_p, 0, g)
        assert _units(hig - log, g).sum(axis=1).max() <= _units(hi1 - lo1, g).sum(axis=1).max()

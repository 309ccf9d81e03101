"""Pins for the controller, cost-table and block-manager oracles (CPU only).

Pinned against: the analytic cost model's closed-form chunk choices
(tests/golden/analytic_cost_model.txt, Sec. 4.1 and Eq. 1), a brute-force
linear scan of Eq. 1, Proposition 1's safety and maximality, numpy's
nearest-rank ("inverted_cdf") percentile and running maximum, exact rational
interpolation, and a hand-worked allocation scenario
(tests/golden/block_manager_scenario.txt).
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import paging, schedule as S

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    with open(os.path.join(GOLD, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_analytic_model_matches_paper_coefficients_and_values():
    rows = _golden("analytic_cost_model.txt")
    coeff = [int(v) for v in next(r for r in rows if r[0] == "coeff")[1:]]
    assert coeff == [350000, 900000, 55000, 400000, 6000]
    for r in rows:
        if r[0] == "value":
            n, c, t = map(int, r[1:])
            assert S.analytic_cost_ns(n, c) == t


def _closed_form(n, budget, c_max, remaining):
    t0 = S.analytic_cost_ns(n, 0)
    if n == 0:
        return min(c_max, remaining)
    if S.analytic_cost_ns(n, 1) > budget:
        return 0
    return max(0, min(c_max, remaining, (budget - t0 - 400_000) // 6_000))


def test_select_chunk_worked_examples():
    for r in _golden("analytic_cost_model.txt"):
        if r[0] != "choice":
            continue
        n, budget, want = map(int, r[1:])
        now = 1_000_000_000
        deadlines = [now + budget + 7 * i for i in range(n)]   # earliest one binds
        c, flags, _ = S.select_chunk(S.analytic_cost_ns, deadlines, now, 100_000, 4096)
        assert c == want == _closed_form(n, budget, 4096, 100_000)
        if want == 0:
            assert flags & S.DECODE_INFEASIBLE


@settings(max_examples=300, deadline=None)
@given(n=st.integers(0, 300), budget=st.integers(-1_000_000, 60_000_000),
       c_max=st.integers(0, 5000), remaining=st.integers(-3, 9000), margin=st.integers(0, 2_000_000))
def test_select_chunk_equals_brute_force_and_closed_form(n, budget, c_max, remaining, margin):
    now = 5_000_000
    deadlines = [now + budget + 1000 * i for i in range(n)]
    c, flags, lookups = S.select_chunk(S.analytic_cost_ns, deadlines, now, remaining, c_max, margin)
    if remaining <= 0:
        assert (c, flags) == (0, S.NO_PENDING)
        return
    cap = min(c_max, remaining)
    if n == 0:
        assert c == cap and flags & S.NO_ACTIVE
        return
    feasible = [x for x in range(cap + 1) if S.analytic_cost_ns(n, x) + margin <= budget]
    brute = max(feasible) if feasible else 0
    assert c == brute
    assert c == _closed_form(n, budget - margin, c_max, remaining)
    # Proposition 1: safe when decode-only is feasible, and maximal
    if S.analytic_cost_ns(n, 0) + margin <= budget:
        assert S.analytic_cost_ns(n, c) + margin <= budget
        assert c == cap or S.analytic_cost_ns(n, c + 1) + margin > budget
        assert not flags & S.DECODE_INFEASIBLE
    else:
        assert c == 0 and flags & S.DECODE_INFEASIBLE
    assert lookups <= math.ceil(math.log2(cap + 1)) + 1


def test_nearest_rank_matches_numpy_inverted_cdf():
    rng = np.random.default_rng(0)
    for k in [1, 2, 3, 7, 99, 100, 101, 250]:
        xs = rng.integers(0, 10**9, size=k)
        for num, den in [(1, 2), (99, 100), (9, 10), (1, 1)]:
            ref = np.percentile(xs, 100.0 * num / den, method="inverted_cdf")
            assert S.nearest_rank(xs, num, den) == int(ref)


def test_cummax_matches_numpy():
    rng = np.random.default_rng(1)
    row = rng.integers(0, 100, size=50)
    assert S.cummax(list(row)) == list(np.maximum.accumulate(row))


def _random_table(rng, nb=4, nc=6, reps=5):
    c_grid = [0] + sorted(rng.choice(np.arange(1, 5000), size=nc - 1, replace=False).tolist())
    b_grid = sorted(rng.choice(np.arange(0, 300), size=nb, replace=False).tolist())
    samples = rng.integers(1_000_000, 30_000_000, size=(nb, nc, reps)).tolist()
    return S.CostTable(c_grid, b_grid, samples)


def test_table_lookup_interpolates_with_ceiling_exactly():
    rng = np.random.default_rng(2)
    for _ in range(20):
        t = _random_table(rng)
        for i, b in enumerate(t.b_grid):
            row = t.t_hat[i]
            assert t.lookup(b, 0) == row[0]
            for j in range(1, len(t.c_grid)):
                assert t.lookup(b, t.c_grid[j]) == row[j]
            for c in rng.integers(1, t.c_grid[-1] + 1, size=40):
                c = int(c)
                j = next(j for j in range(1, len(t.c_grid)) if t.c_grid[j] >= c)
                if j == 1:
                    want = row[1]
                else:
                    frac = Fraction(row[j] - row[j - 1]) * (c - t.c_grid[j - 1]) / (
                        t.c_grid[j] - t.c_grid[j - 1])
                    want = row[j - 1] + math.ceil(frac)
                assert t.lookup(b, c) == want
            vals = [t.lookup(b, c) for c in range(0, t.c_grid[-1] + 1, 7)]
            assert all(x <= y for x, y in zip(vals, vals[1:]))       # monotone in c
        # n rounds up to the next grid point
        for n in range(0, t.b_grid[-1] + 1, 13):
            i = next(i for i, b in enumerate(t.b_grid) if b >= n)
            assert t.lookup(n, 0) == t.t_hat[i][0]
        with pytest.raises(IndexError):
            t.lookup(t.b_grid[-1] + 1, 0)


def test_table_statistics_from_samples():
    rng = np.random.default_rng(3)
    t = _random_table(rng, reps=100)
    for i in range(len(t.b_grid)):
        for j in range(len(t.c_grid)):
            xs = np.sort(t.samples[i][j])
            assert t.p99[i][j] == xs[98] and t.p50[i][j] == xs[49]
        assert t.t_hat[i] == list(np.maximum.accumulate(t.p99[i]))


def test_select_over_table_caps_at_grid_and_matches_scan():
    rng = np.random.default_rng(4)
    for _ in range(30):
        t = _random_table(rng)
        n = int(rng.integers(1, t.b_grid[-1] + 1)) if t.b_grid[-1] > 0 else 0
        now = 0
        budget = int(rng.integers(0, 40_000_000))
        c_max = int(rng.integers(0, 6000))
        rem = int(rng.integers(1, 6000))
        c, flags, _ = S.select_chunk_table(t, [budget] * n, now, rem, c_max)
        cap = min(c_max, rem, t.c_grid[-1])
        if n == 0:
            assert c == cap
            continue
        feas = [x for x in range(cap + 1) if t.lookup(n, x) <= budget]
        assert c == (max(feas) if feas else 0)
        assert bool(flags & S.CAPPED_BY_GRID) == (t.c_grid[-1] < min(c_max, rem))


def test_block_manager_hand_worked_scenario():
    m = paging.BlockManager(8, 16)
    for r in _golden("block_manager_scenario.txt"):
        op = r[0]
        if op == "create":
            m.create(int(r[1]))
        elif op == "reserve":
            try:
                m.reserve(int(r[1]), int(r[2]))
                last_enomem = False
            except paging.OutOfBlocks:
                last_enomem = True
        elif op == "enomem":
            assert last_enomem
        elif op == "expect":
            assert m.block_table(int(r[1])) == [int(v) for v in r[2:]]
        elif op == "free":
            m.free(int(r[1]))
        elif op == "slot":
            assert m.slot(int(r[1]), int(r[2])) == int(r[3])


@settings(max_examples=100, deadline=None)
@given(st.lists(st.tuples(st.sampled_from(["create", "reserve", "free"]), st.integers(0, 5),
                          st.integers(0, 120)), max_size=60))
def test_block_manager_invariants(ops):
    m = paging.BlockManager(20, 16)
    live = set()
    for op, sid, n in ops:
        if op == "create" and sid not in live:
            m.create(sid)
            live.add(sid)
        elif op == "reserve" and sid in live:
            before = {s: m.block_table(s) for s in live}
            free_before = m.free_count()
            try:
                m.reserve(sid, n)
            except paging.OutOfBlocks:
                assert {s: m.block_table(s) for s in live} == before
                assert m.free_count() == free_before
        elif op == "free" and sid in live:
            m.free(sid)
            live.discard(sid)
        used = [b for s in live for b in m.block_table(s)]
        assert len(used) == len(set(used))                      # no block shared
        assert len(used) + m.free_count() == 20
        for s in live:
            assert len(m.block_table(s)) == -(-m.reserved(s) // 16)


def test_iteration_metadata_all_or_nothing():
    m = paging.BlockManager(4, 16)
    for s in (1, 2, 3):
        m.create(s)
    m.reserve(2, 16)
    m.reserve(3, 16)
    with pytest.raises(paging.OutOfBlocks):
        paging.iteration_metadata(m, 40, 1, 0, [2, 3], [16, 16])  # needs 3 + 1 + 1 > 2 free
    assert m.block_table(1) == [] and m.free_count() == 2
    slots, tables = paging.iteration_metadata(m, 10, 1, 0, [2], [15])
    assert tables[1] == [2] and slots == [32 + j for j in range(10)] + [0 * 16 + 15]


def test_context_planes_round_prefix_up():
    """A table with a cached-context axis keeps one (B, C) plane per context
    point; a lookup uses the first point at or above the prefix (the cost of a
    chunk grows with its prefix, so rounding up never under-predicts), and a
    prefix above the last point cannot be priced."""
    c_grid, b_grid, p_grid = [0, 64, 128], [0, 4], [0, 1000, 4000]
    planes = [[[10 * (k + 1) + j + 100 * i for j in range(3)] for i in range(2)] for k in range(3)]
    t = S.CostTable.from_values(c_grid, b_grid, planes, p_grid)
    assert t.lookup(3, 64, 0) == planes[0][1][1]
    assert t.lookup(3, 64, 1000) == planes[1][1][1]
    assert t.lookup(3, 64, 1001) == planes[2][1][1]
    assert t.lookup(0, 96, 2500) == planes[2][0][1] + (-(-(planes[2][0][2] - planes[2][0][1]) * 32 // 64))
    with pytest.raises(IndexError):
        t.lookup(1, 64, 4001)
    flat = S.CostTable.from_values(c_grid, b_grid, planes[0])
    assert flat.lookup(3, 64, 10**6) == flat.lookup(3, 64, 0)     # no context axis: prefix ignored
    # Alg. 1 at a prefix reads that prefix's plane
    pick = lambda pre: S.select_chunk_table(t, [10**9 + 120], 10**9, 500, 128, prefix=pre)[0]
    assert pick(0) == 128 and pick(4000) == 0
    with pytest.raises(IndexError):
        S.select_chunk_table(t, [10**9 + 150], 10**9, 500, 128, prefix=5000)
    assert S.select_chunk_table(t, [], 10**9, 500, 128, prefix=5000)[0] == 128   # nothing to price


def _golden_monotone():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "monotone_table.txt")
    g = {"sample": {}, "p50": {}, "p99": {}, "that": {}}
    for line in open(path):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] in ("c_grid", "b_grid"):
            g[f[0]] = [int(v) for v in f[1:]]
        elif f[0] == "sample":
            g["sample"][(int(f[1]), int(f[2]))] = [int(v) for v in f[3:]]
        elif f[0] in ("p50", "p99", "that"):
            g[f[0]][int(f[1])] = [int(v) for v in f[2:]]
        elif f[0] == "violations":
            g["violations"] = (int(f[1]), int(f[2]))
    samples = [[g["sample"][(b, c)] for c in g["c_grid"]] for b in g["b_grid"]]
    return g, samples


def test_table_statistics_match_hand_worked_golden():
    """P50, P99, running max and the count and size of raw P99 decreases along
    c, against a table worked out by hand (tests/golden/monotone_table.txt):
    an equal step is no decrease, the last column is scanned, and the largest
    drop is the largest of all rows."""
    g, samples = _golden_monotone()
    t = S.CostTable(g["c_grid"], g["b_grid"], samples)
    assert t.p50 == [g["p50"][b] for b in g["b_grid"]]
    assert t.p99 == [g["p99"][b] for b in g["b_grid"]]
    assert t.t_hat == [g["that"][b] for b in g["b_grid"]]
    assert t.monotone_violations() == g["violations"]
    # with a context axis every plane is scanned: two copies double the count
    t2 = S.CostTable(g["c_grid"], g["b_grid"], [samples, samples], p_grid=[0, 4096])
    assert t2.monotone_violations() == (2 * g["violations"][0], g["violations"][1])


def test_iteration_metadata_with_several_prefills_by_hand():
    """Prefill batching (Sec. 3.3): the prefills' reservations come first, in
    the order of their rows, then the decodes; slots worked out by hand on a
    fresh pool of 20 blocks of 16 positions."""
    mgr = paging.BlockManager(20, 16)
    for sid in (1, 2, 3):
        mgr.create(sid)
    # seq 1: positions 0..19 -> blocks 0, 1; seq 2: 0..4 -> block 2; decode 3 at 0 -> block 3
    slots, tables = paging.iteration_metadata(mgr, 25, -1, 0, [3], [0], prefills=[(1, 0, 20), (2, 0, 5)])
    assert slots == list(range(0, 20)) + [32, 33, 34, 35, 36] + [48]
    assert tables == {1: [0, 1], 2: [2], 3: [3]}
    # seq 2: positions 5..16 -> block 2 then a new block 4; seq 1: position 20 in block 1
    slots, tables = paging.iteration_metadata(mgr, 13, -1, 0, [], [], prefills=[(2, 5, 12), (1, 20, 1)])
    assert slots == list(range(37, 48)) + [64] + [20]
    assert tables == {2: [2, 4], 1: [0, 1]}
    # one prefill given either way is the same iteration
    m1, m2 = paging.BlockManager(8, 16), paging.BlockManager(8, 16)
    for m in (m1, m2):
        m.create(5)
    a = paging.iteration_metadata(m1, 17, 5, 0, [], [])
    b = paging.iteration_metadata(m2, 17, -1, 0, [], [], prefills=[(5, 0, 17)])
    assert a == b

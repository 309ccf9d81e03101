"""Oracle for the SLOWeave controller and its cost table.

Test infrastructure only (see ``oracle/__init__``).

* ``select_chunk``: Eq. 1 solved by the binary search of Alg. 1 (Sec. 3.2),
  with the prediction margin of Sec. 3.3.
* ``CostTable``: the profiler of Sec. 5.1 keeps the P50 and P99 iteration
  time at each (decode batch, chunk) grid point and takes a cumulative
  maximum along the chunk axis; Sec. 6.4 interpolates between grid points.
* ``analytic_cost_ns``: the simulator's default cost model of Sec. 4.1, in
  integer nanoseconds.

Times are integer nanoseconds so that every comparison is exact.

Readings (the paper is silent or ambiguous here):
* percentiles are nearest-rank, x_sorted[ceil(q k) - 1] of k samples;
* the decode-batch size n rounds up to the next grid point; n above the
  last grid point is out of range;
* chunk c = 0 reads column 0; 0 < c <= c_1 reads column c_1;
  c_j < c <= c_{j+1} interpolates linearly with a ceiling; c above the last
  grid point is never asked for (the search is capped there);
* Alg. 1 does not clamp the budget at zero (Eq. 1's max(0, .)); the
  decisions agree except when a predicted time plus margin is exactly 0;
* with an empty active set Alg. 1 returns min(C_max, remaining) without a
  cost check; the cap by the last grid point also applies there;
* when even a decode-only iteration misses the budget the result is 0 and
  the DECODE_INFEASIBLE flag is set (Sec. 3.2 falls back to decode-only).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

NO_PENDING = 1
NO_ACTIVE = 2
DECODE_INFEASIBLE = 4
CAPPED_BY_GRID = 8


def nearest_rank(samples, num: int, den: int) -> int:
    """Nearest-rank percentile num/den of integer samples: sorted[ceil(k num/den) - 1]."""
    xs = sorted(int(s) for s in samples)
    k = len(xs)
    if k == 0:
        raise ValueError("no samples")
    rank = -(-k * num // den)          # ceil(k * num / den) in integers
    return xs[max(rank, 1) - 1]


def cummax(row):
    """Running maximum along a row (the profiler's monotone repair, Sec. 5.1)."""
    out = []
    best = None
    for v in row:
        best = v if best is None or v > best else best
        out.append(best)
    return out


@dataclass
class CostTable:
    """Measured iteration times on a (decode batch) x (chunk) grid, optionally
    one such plane per cached-context point (Sec. 5.1 indexes the runtime's
    table by decode batch, cached context and chunk).

    Without p_grid, samples[i][j] holds the raw times (ns) at b_grid[i],
    c_grid[j]; with it, samples[k][i][j] at p_grid[k].  p50, p99 and t_hat
    have the same leading shape.
    """

    c_grid: list
    b_grid: list
    samples: list
    p_grid: list | None = None

    def __post_init__(self):
        c, b = list(map(int, self.c_grid)), list(map(int, self.b_grid))
        if not c or c[0] != 0 or any(x >= y for x, y in zip(c, c[1:])):
            raise ValueError("c_grid must start at 0 and increase strictly")
        if not b or b[0] < 0 or any(x >= y for x, y in zip(b, b[1:])):
            raise ValueError("b_grid must be non-negative and increase strictly")
        self.c_grid, self.b_grid = c, b
        planes = [self.samples] if self.p_grid is None else list(self.samples)
        if self.p_grid is not None:
            pg = list(map(int, self.p_grid))
            if not pg or pg[0] < 0 or any(x >= y for x, y in zip(pg, pg[1:])):
                raise ValueError("p_grid must be non-negative and increase strictly")
            if len(planes) != len(pg):
                raise ValueError("one plane of samples per context point")
            self.p_grid = pg
        p50 = [[[nearest_rank(s, 1, 2) for s in row] for row in pl] for pl in planes]
        p99 = [[[nearest_rank(s, 99, 100) for s in row] for row in pl] for pl in planes]
        t_hat = [[cummax(row) for row in pl] for pl in p99]
        self._t_hat_planes = t_hat
        if self.p_grid is None:
            self.p50, self.p99, self.t_hat = p50[0], p99[0], t_hat[0]
        else:
            self.p50, self.p99, self.t_hat = p50, p99, t_hat

    @classmethod
    def from_values(cls, c_grid, b_grid, values, p_grid=None):
        """A table whose every grid point holds one value (e.g. an analytic model)."""
        if p_grid is None:
            return cls(c_grid, b_grid, [[[int(v)] for v in row] for row in values])
        return cls(c_grid, b_grid, [[[[int(v)] for v in row] for row in pl] for pl in values], p_grid)

    def row_for(self, n: int) -> int:
        for i, b in enumerate(self.b_grid):
            if b >= n:
                return i
        raise IndexError(f"n={n} above the decode-batch grid")

    def plane_for(self, prefix: int) -> int:
        """The plane of the first context point >= prefix (the only plane without a context axis)."""
        if self.p_grid is None:
            return 0
        for k, p in enumerate(self.p_grid):
            if p >= prefix:
                return k
        raise IndexError(f"prefix={prefix} above the context grid")

    def lookup(self, n: int, c: int, prefix: int = 0) -> int:
        """Predicted time T_hat(prefix, n, c) in ns from the cummax P99 table."""
        row = self._t_hat_planes[self.plane_for(prefix)][self.row_for(n)]
        cg = self.c_grid
        if c < 0 or c > cg[-1]:
            raise IndexError(f"c={c} outside [0, {cg[-1]}]")
        if c == 0:
            return row[0]
        j = 1
        while cg[j] < c:
            j += 1
        # now cg[j-1] < c <= cg[j]
        if j == 1:
            return row[1]
        lo_c, hi_c = cg[j - 1], cg[j]
        lo_t, hi_t = row[j - 1], row[j]
        num = (hi_t - lo_t) * (c - lo_c)
        den = hi_c - lo_c
        return lo_t + (-(-num // den))

    def monotone_violations(self):
        """Raw P99 decreases along the chunk axis: (count, largest drop in ns)."""
        count, worst = 0, 0
        rows = self.p99 if self.p_grid is None else [r for pl in self.p99 for r in pl]
        for row in rows:
            for a, b in zip(row, row[1:]):
                if b < a:
                    count += 1
                    worst = max(worst, a - b)
        return count, worst


def analytic_cost_ns(n: int, c: int) -> int:
    """Sec. 4.1: T(n,c) = 0.35 + 1[n>0](0.90 + 0.055 n) + 1[c>0](0.40 + 0.006 c) ms."""
    t = 350_000
    if n > 0:
        t += 900_000 + 55_000 * n
    if c > 0:
        t += 400_000 + 6_000 * c
    return t


def select_chunk(predict, deadlines_ns, now_ns: int, remaining: int, c_max: int,
                 margin_ns: int = 0, c_last: int | None = None):
    """Alg. 1: the largest chunk whose predicted iteration meets the earliest deadline.

    predict(n, c) -> ns is the cost predictor T_hat (monotone in c);
    deadlines_ns are the active decodes' absolute next-token deadlines
    d_i = l_i + D; remaining is the remaining prompt length of the oldest
    pending prefill (<= 0: none pending); c_last caps the search at the
    largest profiled chunk.  Returns (chunk, flags, n_lookups).
    """
    flags = 0
    lookups = 0
    if remaining <= 0:
        return 0, NO_PENDING, 0
    cap = min(c_max, remaining)
    if c_last is not None and c_last < cap:
        cap = c_last
        flags |= CAPPED_BY_GRID
    cap = max(cap, 0)
    n = len(deadlines_ns)
    if n == 0:
        return cap, flags | NO_ACTIVE, 0
    budget = min(int(d) for d in deadlines_ns) - int(now_ns)
    lo, hi = 0, cap
    while lo < hi:
        mid = (lo + hi + 1) // 2
        lookups += 1
        if predict(n, mid) + margin_ns <= budget:
            lo = mid
        else:
            hi = mid - 1
    if lo == 0:
        lookups += 1
        if predict(n, 0) + margin_ns > budget:
            flags |= DECODE_INFEASIBLE
    return lo, flags, lookups


def select_chunk_table(table: CostTable, deadlines_ns, now_ns, remaining, c_max, margin_ns=0, prefix=0):
    """Alg. 1 over a measured table (the capped, interpolated lookup at the
    chunk sequence's cached prefix).

    Alg. 1 returns before any cost query when nothing is pending or nothing
    is active; only then can the decode count or the prefix fall outside the
    table.
    """
    if remaining > 0 and len(deadlines_ns) > 0:
        table.row_for(len(deadlines_ns))          # raises for n above the grid
        table.plane_for(prefix)                   # raises for a prefix above the grid
    return select_chunk(lambda n, c: table.lookup(n, c, prefix), deadlines_ns, now_ns, remaining, c_max,
                        margin_ns, c_last=table.c_grid[-1])

"""Pins for the serving oracle (Sec. 3.1 deadline model, Sec. 4.1 simulator, Sec. 4.3 metrics).

The worked traces below were stepped through by hand with the Sec. 4.1 cost
model T(n, c) = 0.35 + 1[n>0](0.90 + 0.055 n) + 1[c>0](0.40 + 0.006 c) ms;
each expected time is written out as its sum of terms.  They pin the event
logic: chunk sequencing, when the first token appears, when a new arrival
becomes eligible, oldest-first order, decode iterations, finishing.
"""
import numpy as np
import pytest

from oracle import schedule as S
from oracle import serving as V
from paper_2609_07883_amd import synth

MS = 1_000_000


def R(rid, arrival, prompt, output):
    return V.Request(rid, arrival, prompt, output)


def test_single_request_fixed_chunks_by_hand():
    tr = V.simulate([R(0, 0, 100, 3)], cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS,
                    policy="fixed", fixed_chunk=64)
    t1 = 350_000 + 400_000 + 6_000 * 64            # chunk of 64, nothing decoding
    t2 = t1 + 350_000 + 400_000 + 6_000 * 36       # last 36 prompt tokens -> first token
    t3 = t2 + 350_000 + 900_000 + 55_000           # one decode
    t4 = t3 + 350_000 + 900_000 + 55_000
    assert tr.token_ns[0] == [t2, t3, t4]
    assert [(i.chunk, i.n_decode) for i in tr.iterations] == [(64, 0), (36, 0), (0, 1), (0, 1)]
    m = V.request_metrics(R(0, 0, 100, 3), tr.token_ns[0], 10 * MS, 10 * MS)
    assert (m.ttft_ns, m.tpot_p99_ns, m.meets) == (2_100_000, 1_305_000, True)


def test_arrival_during_iteration_waits_for_its_end():
    reqs = [R(0, 0, 10, 2), R(1, 500_000, 5, 1)]
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="fixed", fixed_chunk=64)
    e1 = 350_000 + 400_000 + 6_000 * 10                                  # r0 prompt alone
    e2 = e1 + 350_000 + (900_000 + 55_000) + (400_000 + 6_000 * 5)      # r0 decode + r1 prompt
    assert tr.token_ns == {0: [e1, e2], 1: [e2]}
    assert tr.iterations[1].prefill_rid == 1 and tr.iterations[1].n_decode == 1
    s = V.summarize(reqs, tr.token_ns, ttft_slo_ns=2 * MS, tpot_slo_ns=2 * MS)
    # r0: TTFT 0.81 ms, one gap of 1.735 ms -> meets; r1: TTFT 2.045 ms -> misses
    assert (s["met"], s["goodput_den_ns"], s["makespan_ns"]) == (1, 500_000, e2)
    assert s["p99_ttft_ns"] == e2 - 500_000


def test_sloweave_decisions_by_hand():
    """Alg. 1 on the analytic model: with one decode and a 5 ms objective the chunk
    is floor((5 - T(1,0) - 0.40) / 0.006) = 549 tokens (the closed form of the
    linear model); with nothing decoding it is the cap, 4096."""
    reqs = [R(0, 0, 1, 3), R(1, 0, 10_000, 1)]
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=5 * MS, policy="sloweave", c_max=4096)
    chunks = [i.chunk for i in tr.iterations]
    assert chunks == [1, 549, 549, 4096, 4096, 710]
    assert sum(chunks[1:]) == 10_000
    e1 = 350_000 + 400_000 + 6_000
    e2 = e1 + 350_000 + 955_000 + 400_000 + 6_000 * 549
    e3 = e2 + 350_000 + 955_000 + 400_000 + 6_000 * 549
    assert tr.token_ns[0] == [e1, e2, e3]
    assert e2 - e1 == 4_999_000                    # one microsecond inside the 5 ms deadline
    e6 = e3 + 2 * (350_000 + 400_000 + 6_000 * 4096) + 350_000 + 400_000 + 6_000 * 710
    assert tr.token_ns[1] == [e6]
    assert [i.budget_ns for i in tr.iterations[1:3]] == [5 * MS, 5 * MS]


def test_oldest_first_and_one_token_outputs():
    reqs = [R(5, 100, 20, 1), R(2, 100, 20, 1), R(9, 50, 20, 1)]
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="fixed", fixed_chunk=20)
    assert [i.prefill_rid for i in tr.iterations] == [9, 2, 5]
    assert all(len(v) == 1 for v in tr.token_ns.values())


def test_idle_gap_jumps_to_next_arrival():
    reqs = [R(0, 0, 10, 1), R(1, 50 * MS, 10, 1)]
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="fixed", fixed_chunk=64)
    assert tr.iterations[1].start_ns == 50 * MS
    assert tr.token_ns[1] == [50 * MS + 350_000 + 400_000 + 60_000]


def test_decode_cap_holds_back_prefill():
    reqs = [R(i, 0, 4, 5) for i in range(3)]
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="fixed", fixed_chunk=64,
                    max_decode=2)
    assert max(i.n_decode for i in tr.iterations) == 2
    # the third prompt waits until a decode finishes
    third = [k for k, i in enumerate(tr.iterations) if i.prefill_rid == 2][0]
    assert tr.iterations[third].n_decode < 2


def _small_trace(n, rate, seed):
    t = synth.request_trace(n, rate, seed=seed, long_lo=512, long_hi=2048, short_median=128,
                            output_mean=16)
    return [R(i, int(a), int(p), int(o)) for i, (a, p, o) in enumerate(zip(t.arrival_ns, t.prompt, t.output))]


@pytest.mark.parametrize("policy,chunk", [("sloweave", 0), ("fixed", 256), ("fixed", 2048)])
def test_conservation(policy, chunk):
    reqs = _small_trace(120, 40.0, seed=7)
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=10 * MS, policy=policy, fixed_chunk=chunk,
                    max_decode=32)
    by = {r.rid: r for r in reqs}
    for rid, toks in tr.token_ns.items():
        assert len(toks) == by[rid].output
        assert all(b > a for a, b in zip(toks, toks[1:]))
        assert toks[0] > by[rid].arrival_ns
    per = {}
    for it in tr.iterations:
        if it.chunk:
            per[it.prefill_rid] = per.get(it.prefill_rid, 0) + it.chunk
    assert per == {r.rid: r.prompt for r in reqs}
    for a, b in zip(tr.iterations, tr.iterations[1:]):
        assert b.start_ns >= a.end_ns
        if b.start_ns > a.end_ns:   # only an idle system waits, and only for an arrival
            assert b.start_ns in {r.arrival_ns for r in reqs}
    assert max(i.n_decode for i in tr.iterations) <= 32


def test_prop1_exact_predictions_never_miss():
    """Prop. 1: with exact predictions and a feasible decode-only iteration the
    controller meets every next-token deadline; a large fixed chunk does not."""
    reqs = _small_trace(150, 60.0, seed=11)
    D = 10 * MS
    assert S.analytic_cost_ns(64, 0) <= D
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=D, policy="sloweave", max_decode=64)
    gaps = [b - a for t in tr.token_ns.values() for a, b in zip(t, t[1:])]
    assert gaps and max(gaps) <= D
    fx = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=D, policy="fixed", fixed_chunk=2048,
                    max_decode=64)
    gaps_fx = [b - a for t in fx.token_ns.values() for a, b in zip(t, t[1:])]
    assert max(gaps_fx) > D


def test_margin_is_kept_free_in_every_chunked_iteration():
    """Sec. 3.3: a chunk runs beside decodes only if its predicted time plus the
    margin fits the budget; decode-only iterations are the fallback."""
    reqs = _small_trace(80, 60.0, seed=3)
    delta = 2 * MS
    tr = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=10 * MS, policy="sloweave", max_decode=64,
                    margin_ns=delta)
    mixed = [i for i in tr.iterations if i.n_decode and i.chunk]
    assert mixed and all(i.end_ns - i.start_ns + delta <= i.budget_ns for i in mixed)
    gaps = [b - a for t in tr.token_ns.values() for a, b in zip(t, t[1:])]
    assert max(gaps) <= 10 * MS


def test_table_predictor_matches_analytic_on_a_dense_grid():
    """A table holding the analytic model at every decode count and at chunks 0, 1
    and a coarse grid above reproduces it exactly (linear between grid points)."""
    c_grid = [0, 1, 64, 512, 4096]
    b_grid = list(range(0, 65))
    tab = S.CostTable.from_values(c_grid, b_grid, [[S.analytic_cost_ns(b, c) for c in c_grid] for b in b_grid])
    for n in (0, 1, 7, 64):
        for c in (0, 1, 2, 63, 64, 65, 511, 3000, 4096):
            assert tab.lookup(n, c) == S.analytic_cost_ns(n, c)
    reqs = _small_trace(60, 60.0, seed=5)
    a = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=10 * MS, max_decode=64)
    b = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=10 * MS, max_decode=64, predict=tab.lookup,
                   c_last=4096)
    assert a.token_ns == b.token_ns


def test_tpot_is_nearest_rank_p99_of_gaps():
    toks = list(np.cumsum(np.arange(1, 201)))      # gaps 2, 3, ..., 200
    m = V.request_metrics(R(0, 0, 1, 200), [int(t) for t in toks], 10**9, 10**9)
    # 199 gaps; rank ceil(199 * 0.99) = 198 -> the 198th smallest gap = 199
    assert m.tpot_p99_ns == 199
    assert V.request_metrics(R(0, 0, 1, 1), [5], 10, 0).meets          # no gap: meets any TPOT
    with pytest.raises(ValueError):
        V.request_metrics(R(0, 0, 1, 2), [5], 10, 10)


def test_trace_generator_shape():
    t = synth.request_trace(4000, 4.0, seed=3)
    assert t.arrival_ns[0] == 0 and np.all(np.diff(t.arrival_ns) >= 0)
    assert t.prompt.min() >= 1 and t.prompt.max() <= 16384 and t.output.min() >= 1
    assert abs(t.output.mean() - 256) < 15
    assert 0.4 < np.mean(t.prompt >= 4096) < 0.75
    no_burst = synth.request_trace(4000, 4.0, seed=3, burst_factor=1.0)
    assert abs(no_burst.arrival_ns[-1] / 1e9 - 1000) < 60            # Poisson at 4/s
    assert t.arrival_ns[-1] < no_burst.arrival_ns[-1]                 # bursts add arrivals


def test_telemetry_margin_is_inert_with_exact_predictions():
    """Residuals of an exact predictor are 0, so the margin stays 0 and the run is unchanged."""
    reqs = _small_trace(80, 60.0, seed=21)
    base = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=10 * MS, max_decode=64)
    tele = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=10 * MS, max_decode=64, residual_window=16)
    assert base.token_ns == tele.token_ns
    assert all(i.rel_margin_ppm == 0 for i in tele.iterations)


def _slow_hw(n, c):
    """Hardware 20% slower than the analytic table (every T is a multiple of 1000 ns)."""
    return S.analytic_cost_ns(n, c) * 6 // 5


def test_telemetry_margin_restores_deadlines_on_slow_hardware():
    """Sec. 3.3: a margin bounding the one-sided prediction error keeps Prop. 1.
    With iterations 20% slower than predicted, the plain controller overruns
    the objective; with the telemetry window the first chunked iteration
    leaves a residual of exactly 200000 ppm, every later decision adds 20% to
    its predictions, and no token gap exceeds D."""
    reqs = _small_trace(150, 60.0, seed=11)
    D = 10 * MS
    assert _slow_hw(64, 0) <= D
    plain = V.simulate(reqs, cost_ns=_slow_hw, predict=S.analytic_cost_ns, tpot_ns=D, max_decode=64)
    gaps = [b - a for t in plain.token_ns.values() for a, b in zip(t, t[1:])]
    assert max(gaps) > D
    tele = V.simulate(reqs, cost_ns=_slow_hw, predict=S.analytic_cost_ns, tpot_ns=D, max_decode=64,
                      residual_window=16)
    gaps = [b - a for t in tele.token_ns.values() for a, b in zip(t, t[1:])]
    assert max(gaps) <= D
    first = next(k for k, i in enumerate(tele.iterations) if i.chunk > 0)
    assert tele.iterations[first].rel_margin_ppm == 0
    later = [i.rel_margin_ppm for i in tele.iterations[first + 1:] if i.chunk > 0 or i.n_decode == 0]
    assert later and all(q == 200_000 for q in later if q)


def test_telemetry_window_uses_nearest_rank_p99():
    """The margin is the nearest-rank P99 of the last W residuals: with W = 2
    it is the larger of the last two."""
    reqs = [R(0, 0, 300, 1)]
    costs = iter([1_000_000, 2_000_000, 1_500_000])   # ns of the three chunked iterations
    observed = {}

    def hw(n, c):
        return observed.setdefault((n, c, len(observed)), next(costs))

    tr = V.simulate(reqs, cost_ns=lambda n, c: hw(n, c), predict=lambda n, c: 1_000_000, tpot_ns=MS,
                    policy="sloweave", c_max=100, residual_window=2)
    assert [i.chunk for i in tr.iterations] == [100, 100, 100]
    # residuals: 0, 1e6 ppm, 0.5e6 ppm; margins seen by the 2nd and 3rd decisions
    assert [i.rel_margin_ppm for i in tr.iterations] == [0, 0, 1_000_000]


def _slow_chunks(n, c):
    """Hardware stand-in: the analytic model plus 1.5 ms on every iteration that runs a chunk."""
    return S.analytic_cost_ns(n, c) + (1_500_000 if c > 0 else 0)


def test_telemetry_fallback_by_hand():
    """Sec. 5.1's decode-only fallback, stepped by hand.  The controller
    predicts the analytic model T(n, c) (in ns: 350000 + [n>0](900000 +
    55000 n) + [c>0](400000 + 6000 c)); every chunked iteration really takes
    1.5 ms longer.  Margin delta = 1 ms, fallback window of one residual,
    TPOT 50 ms; A (prompt 100, output 5) and B (prompt 200, output 3) arrive
    at 0.

      1. t=0: no decode, window empty: A's whole prompt, 100 tokens.  Cost
         T(0,100) + 1.5 ms = 1350000 + 1500000 = 2850000; residual 1500000.
      2. t=2850000: window P99 1500000 > delta: decode-only fallback for B's
         turn.  Cost T(1,0) = 1305000, end 4155000; residual 0.
      3. t=4155000: window P99 0 <= delta: Alg. 1 gives B's 200 tokens
         (T(1,200) + 1 ms = 3905000 within 50 ms).  Cost 2905000 + 1500000,
         end 8560000; B's first token.
      4. t=8560000: nothing pending: decode-only, T(2,0) = 1360000, end 9920000.
      5. t=9920000: decode-only, end 11280000: A's fifth and B's third token.
    """
    reqs = [V.Request(0, 0, 100, 5), V.Request(1, 0, 200, 3)]
    tr = V.simulate(reqs, cost_ns=_slow_chunks, predict=S.analytic_cost_ns, tpot_ns=50_000_000,
                    margin_ns=1_000_000, fallback_window=1)
    got = [(i.start_ns, i.end_ns, i.chunk, i.n_decode, i.prefill_rid, i.fallback, i.resid_p99_ns)
           for i in tr.iterations]
    assert got == [(0, 2_850_000, 100, 0, 0, False, 0),
                   (2_850_000, 4_155_000, 0, 1, -1, True, 1_500_000),
                   (4_155_000, 8_560_000, 200, 1, 1, False, 0),
                   (8_560_000, 9_920_000, 0, 2, -1, False, 0),
                   (9_920_000, 11_280_000, 0, 2, -1, False, 0)]
    assert tr.token_ns[0] == [2_850_000, 4_155_000, 8_560_000, 9_920_000, 11_280_000]
    assert tr.token_ns[1] == [8_560_000, 9_920_000, 11_280_000]
    # without the fallback B's chunk runs at once, ending at 2850000 + 4405000
    tr0 = V.simulate(reqs, cost_ns=_slow_chunks, predict=S.analytic_cost_ns, tpot_ns=50_000_000,
                     margin_ns=1_000_000)
    assert tr0.token_ns[1][0] == 7_255_000
    assert not any(i.fallback for i in tr0.iterations)


def test_telemetry_fallback_is_inert_within_the_margin():
    """Residuals at most delta never trigger the fallback: the run equals one without it."""
    tr = synth.request_trace(120, 6.0, seed=4)
    reqs = [V.Request(i, int(a), int(p), int(o)) for i, (a, p, o) in
            enumerate(zip(tr.arrival_ns, tr.prompt, tr.output))]
    cost = lambda n, c: S.analytic_cost_ns(n, c) + (700_000 if c > 0 else 0)
    base = V.simulate(reqs, cost_ns=cost, predict=S.analytic_cost_ns, tpot_ns=25_000_000, margin_ns=700_000,
                      max_decode=256)
    fb = V.simulate(reqs, cost_ns=cost, predict=S.analytic_cost_ns, tpot_ns=25_000_000, margin_ns=700_000,
                    max_decode=256, fallback_window=16)
    assert base.token_ns == fb.token_ns
    assert not any(i.fallback for i in fb.iterations)
    assert max(i.resid_p99_ns for i in fb.iterations) == 700_000

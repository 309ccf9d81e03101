"""The library's serving loop against the serving oracle (CPU: analytic and table executors).

slw_serve with the analytic executor is the Sec. 4.1 simulator; every token
time and every iteration (start, end, chunk, decode count, prefill request,
budget, remaining prompt) must equal the oracle's bit for bit, for both
policies, with the controller reading a table that holds the cost model
exactly (dense grid) or only approximately (a coarse grid: decode counts
round up, chunks interpolate).  The request-level metrics computed by the
product module must equal the oracle's.
"""
import numpy as np
import pytest

from oracle import schedule as S
from oracle import serving as V
from paper_2609_07883_amd import api, serving, synth

MS = 1_000_000
COARSE_C = [0, 32, 64, 128, 256, 512, 1024, 2048, 4096]
COARSE_B = [0, 1, 2, 4, 8, 16, 32, 64, 128, 256]


def _trace(n, rate, seed, **kw):
    return synth.request_trace(n, rate, seed=seed, **kw)


def _oracle_reqs(tr):
    return [V.Request(i, int(a), int(p), int(o)) for i, (a, p, o) in
            enumerate(zip(tr.arrival_ns, tr.prompt, tr.output))]


def _oracle_table(c_grid, b_grid):
    return S.CostTable.from_values(c_grid, b_grid, [[S.analytic_cost_ns(b, c) for c in c_grid] for b in b_grid])


def _compare(tr, res, ref):
    for i, toks in enumerate(res.token_ns):
        assert toks.tolist() == ref.token_ns[i], f"request {i}"
    it = res.iterations
    assert len(it) == len(ref.iterations)
    got = np.stack([it["start_ns"], it["end_ns"], it["chunk"], it["n_decode"], it["prefill_id"], it["budget_ns"],
                    it["rel_margin_ppm"]], 1)
    exp = np.array([[r.start_ns, r.end_ns, r.chunk, r.n_decode, r.prefill_rid, r.budget_ns, r.rel_margin_ppm]
                    for r in ref.iterations])
    bad = np.nonzero((got != exp).any(1))[0]
    assert len(bad) == 0, f"first differing iteration {bad[0]}: {got[bad[0]]} vs {exp[bad[0]]}"


@pytest.mark.parametrize("grid", ["dense", "coarse"])
@pytest.mark.parametrize("tpot_ms,margin_ms", [(25, 0), (10, 0), (10, 2)])
def test_sloweave_matches_oracle(grid, tpot_ms, margin_ms):
    tr = _trace(300, 6.0, seed=3)
    if grid == "dense":
        cg, bg = [0, 1, 64, 512, 4096], list(range(0, 257))
    else:
        cg, bg = COARSE_C, COARSE_B
    tab = api.CostTable.analytic(cg, bg)
    res = serving.run(tr, policy="sloweave", tpot_ms=tpot_ms, max_decode=256, table=tab, margin_ns=margin_ms * MS)
    ot = _oracle_table(cg, bg)
    ref = V.simulate(_oracle_reqs(tr), cost_ns=S.analytic_cost_ns, tpot_ns=tpot_ms * MS, policy="sloweave",
                     predict=ot.lookup, c_last=cg[-1], c_max=4096, margin_ns=margin_ms * MS, max_decode=256)
    _compare(tr, res, ref)


@pytest.mark.parametrize("chunk", [256, 512, 2048])
def test_fixed_matches_oracle(chunk):
    tr = _trace(300, 6.0, seed=4)
    res = serving.run(tr, policy="fixed", fixed_chunk=chunk, tpot_ms=25, max_decode=64)
    ref = V.simulate(_oracle_reqs(tr), cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="fixed",
                     fixed_chunk=chunk, max_decode=64)
    _compare(tr, res, ref)


def test_decode_batch_above_table_is_decode_only():
    tr = _trace(200, 40.0, seed=5, long_lo=256, long_hi=1024, short_median=64, output_mean=64)
    cg, bg = COARSE_C, [0, 1, 2, 4, 8]
    tab = api.CostTable.analytic(cg, bg)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=32, table=tab)
    ref = V.simulate(_oracle_reqs(tr), cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="sloweave",
                     predict=_oracle_table(cg, bg).lookup, c_last=cg[-1], max_decode=32)
    _compare(tr, res, ref)
    it = res.iterations
    over = it[(it["n_decode"] > 8) & (it["remaining"] > 0)]
    assert len(over) > 0 and (over["chunk"] == 0).all()
    assert (over["flags"] & api.SERVE_UNPRICED).all()


def test_decode_cap_flags_and_predictions():
    tr = _trace(200, 40.0, seed=6, long_lo=256, long_hi=1024, short_median=64, output_mean=64)
    tab = api.CostTable.analytic(COARSE_C, COARSE_B)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=4, table=tab)
    it = res.iterations
    assert it["n_decode"].max() == 4
    capped = it[(it["flags"] & api.SERVE_DECODE_CAP) != 0]
    assert len(capped) > 0 and (capped["chunk"] == 0).all() and (capped["n_decode"] >= 4).all()
    ot = _oracle_table(COARSE_C, COARSE_B)
    assert all(r["predicted_ns"] == ot.lookup(int(r["n_decode"]), int(r["chunk"])) for r in it[:500])


def test_metrics_match_oracle():
    tr = _trace(400, 6.0, seed=7)
    tab = api.CostTable.analytic(COARSE_C, COARSE_B)
    for pol, fc, D in [("sloweave", 0, 10), ("fixed", 2048, 10), ("fixed", 256, 25)]:
        res = serving.run(tr, policy=pol, fixed_chunk=fc, tpot_ms=D, max_decode=256, table=tab)
        got = serving.metrics(tr, res.token_ns, ttft_slo_ms=1000, tpot_slo_ms=D)
        ref = V.summarize(_oracle_reqs(tr), {i: t.tolist() for i, t in enumerate(res.token_ns)},
                          ttft_slo_ns=1000 * MS, tpot_slo_ns=D * MS)
        assert got["met"] == ref["met"]
        assert got["arrival_span_ns"] == ref["goodput_den_ns"]
        assert got["makespan_ns"] == ref["makespan_ns"]
        assert got["p99_ttft_ms"] * 1e6 == pytest.approx(ref["p99_ttft_ns"], abs=0.5)
        assert got["p50_ttft_ms"] * 1e6 == pytest.approx(ref["p50_ttft_ns"], abs=0.5)
        assert got["p99_tpot_ms"] * 1e6 == pytest.approx(ref["p99_tpot_ns"], abs=0.5)
        assert got["goodput_req_s"] == pytest.approx(ref["goodput_num"] / ref["goodput_den_ns"] * 1e9)
        per = [V.request_metrics(r, res.token_ns[r.rid].tolist(), 1000 * MS, D * MS) for r in _oracle_reqs(tr)]
        assert got["ttft_missed"] == sum(m.ttft_ns > 1000 * MS for m in per)
        assert got["tpot_missed"] == sum(m.tpot_p99_ns > D * MS for m in per)


def test_sloweave_beats_fixed_at_tight_tpot_in_simulation():
    """Trend of Sec. 4 (no numeric parity: the paper's workload parameters differ):
    at a 10 ms TPOT objective the controller's goodput is at least that of every
    fixed chunk on the config-4 trace under the analytic model."""
    tr = _trace(600, 4.0, seed=3)
    tab = api.CostTable.analytic(COARSE_C, COARSE_B)
    good = {}
    for pol, fc in [("sloweave", 0), ("fixed", 256), ("fixed", 512), ("fixed", 2048)]:
        res = serving.run(tr, policy=pol, fixed_chunk=fc, tpot_ms=10, max_decode=256, table=tab)
        good[(pol, fc)] = serving.metrics(tr, res.token_ns, 1000, 10)["goodput_req_s"]
    assert good[("sloweave", 0)] >= max(v for k, v in good.items() if k[0] == "fixed")


def _scaled_tables(cg, bg, num, den):
    """Controller table (analytic) and a hardware stand-in num/den slower, both as the
    library's tables and the oracle's."""
    vals = [[S.analytic_cost_ns(b, c) * num // den for c in cg] for b in bg]
    return (api.CostTable.analytic(cg, bg), api.CostTable.from_samples(cg, bg, np.array(vals, dtype=np.int64)),
            _oracle_table(cg, bg), S.CostTable.from_values(cg, bg, vals))


@pytest.mark.parametrize("window,num,den,margin_ms", [(16, 6, 5, 0), (1, 5, 4, 0), (64, 11, 10, 1), (8, 9, 10, 0)])
def test_telemetry_margin_matches_oracle(window, num, den, margin_ms):
    """The relative-residual window, its P99 and the widened predictions are
    the oracle's bit for bit, on hardware faster or slower than the table."""
    tr = _trace(250, 6.0, seed=8)
    ctl, hw, octl, ohw = _scaled_tables(COARSE_C, COARSE_B, num, den)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, table=ctl, exec_table=hw,
                      residual_window=window, margin_ns=margin_ms * MS)
    ref = V.simulate(_oracle_reqs(tr), cost_ns=ohw.lookup, predict=octl.lookup, c_last=COARSE_C[-1],
                     tpot_ns=25 * MS, max_decode=256, residual_window=window, margin_ns=margin_ms * MS)
    _compare(tr, res, ref)
    if num > den:
        assert res.iterations["rel_margin_ppm"].max() > 0


def test_telemetry_margin_cuts_deadline_misses():
    tr = _trace(300, 6.0, seed=9)
    ctl, hw, _, _ = _scaled_tables(COARSE_C, COARSE_B, 6, 5)
    miss = {}
    for w in (0, 32):
        res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, table=ctl, exec_table=hw,
                          residual_window=w)
        gaps = np.concatenate([np.diff(t) for t in res.token_ns if len(t) > 1])
        miss[w] = int(np.sum(gaps > 25 * MS))
    assert miss[0] > 0 and miss[32] < miss[0]


def test_errors():
    tr = _trace(10, 4.0, seed=1)
    with pytest.raises(api.SloweaveError) as e:
        api.serve([1, 1], [0, 5], [4, 4], [1, 1], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.SloweaveError) as e:      # SLOWeave without a table
        serving.run(tr, policy="sloweave", tpot_ms=10, max_decode=4)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.SloweaveError) as e:      # GPU executor without a context
        api.serve([0], [0], [4], [1], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4,
                  executor=api.EXEC_GPU)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.SloweaveError) as e:      # iteration cap
        api.serve([0], [0], [400], [50], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4,
                  iter_cap=10)
    assert e.value.code == api.ERANGE
    with pytest.raises(api.SloweaveError) as e:
        api.serve([0], [0], [0], [1], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4)
    assert e.value.code == api.EINVAL
    tok, its = api.serve([], [], [], [], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4)
    assert tok == [] and len(its) == 0
    with pytest.raises(api.SloweaveError) as e:      # table executor without its table
        api.serve([0], [0], [4], [1], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4,
                  executor=api.EXEC_TABLE)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.SloweaveError) as e:
        api.serve([0], [0], [4], [1], policy=api.POLICY_FIXED, fixed_chunk=8, tpot_ns=MS, max_decode=4,
                  residual_window=-1)
    assert e.value.code == api.ERANGE


CTX_P = [0, 2048, 4096, 8192, 16384]


def _ctx_tables(kappa_ctl, kappa_hw):
    """Tables with a cached-context axis: the analytic model plus kappa ns per
    chunk token per 1024 prefix tokens (the chunk's attention over its prefix)."""
    def vals(kappa):
        return [[[S.analytic_cost_ns(b, c) + kappa * c * p // 1024 for c in COARSE_C] for b in COARSE_B]
                for p in CTX_P]
    v_ctl, v_hw = vals(kappa_ctl), vals(kappa_hw)
    lib_t = lambda v: api.CostTable.from_samples(COARSE_C, COARSE_B, np.array(v, dtype=np.int64), p_grid=CTX_P)
    ora_t = lambda v: S.CostTable.from_values(COARSE_C, COARSE_B, v, CTX_P)
    return lib_t(v_ctl), lib_t(v_hw), ora_t(v_ctl), ora_t(v_hw)


@pytest.mark.parametrize("kappa_ctl,kappa_hw,window", [(400, 400, 0), (0, 600, 0), (300, 600, 16)])
def test_context_tables_match_oracle(kappa_ctl, kappa_hw, window):
    """Decisions and iteration times priced at the oldest prompt's cached
    prefix, bit for bit against the oracle (with and without telemetry)."""
    tr = _trace(250, 6.0, seed=12)
    ctl, hw, octl, ohw = _ctx_tables(kappa_ctl, kappa_hw)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, table=ctl, exec_table=hw,
                      residual_window=window)
    ref = V.simulate(_oracle_reqs(tr), cost_ns=ohw.lookup, predict=octl.lookup, c_last=COARSE_C[-1],
                     tpot_ns=25 * MS, max_decode=256, residual_window=window, prefix_aware=True)
    _compare(tr, res, ref)
    it = res.iterations
    assert np.all(it["predicted_ns"][it["chunk"] > 0] > 0)


def test_context_axis_removes_long_prefix_misses():
    """On hardware whose chunk cost grows with the prefix, a controller that
    prices at the profiled prefix 0 overruns deadlines; pricing at the
    chunk's own prefix does not."""
    tr = _trace(300, 6.0, seed=13)
    ctl_ctx, hw, _, _ = _ctx_tables(600, 600)
    flat = api.CostTable.analytic(COARSE_C, COARSE_B)
    miss = {}
    for name, tab in (("flat", flat), ("ctx", ctl_ctx)):
        res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, table=tab, exec_table=hw)
        gaps = np.concatenate([np.diff(t) for t in res.token_ns if len(t) > 1])
        miss[name] = int(np.sum(gaps > 25 * MS))
    assert miss["flat"] > 0 and miss["ctx"] == 0


@pytest.mark.parametrize("window,num,den,margin_ms", [(1, 6, 5, 0), (16, 11, 10, 1), (64, 5, 4, 2), (8, 9, 10, 0)])
def test_telemetry_fallback_matches_oracle(window, num, den, margin_ms):
    """The absolute-residual window, its P99, the decode-only fallback and its
    record flag are the oracle's bit for bit, on hardware faster or slower
    than the table."""
    tr = _trace(250, 6.0, seed=12)
    ctl, hw, octl, ohw = _scaled_tables(COARSE_C, COARSE_B, num, den)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, table=ctl, exec_table=hw,
                      margin_ns=margin_ms * MS, fallback_window=window)
    ref = V.simulate(_oracle_reqs(tr), cost_ns=ohw.lookup, predict=octl.lookup, c_last=COARSE_C[-1],
                     tpot_ns=25 * MS, max_decode=256, margin_ns=margin_ms * MS, fallback_window=window)
    _compare(tr, res, ref)
    it = res.iterations
    fb = (it["flags"] & api.SERVE_FALLBACK) != 0
    assert fb.tolist() == [r.fallback for r in ref.iterations]
    assert it["resid_p99_ns"].tolist() == [r.resid_p99_ns for r in ref.iterations]
    assert np.all(it["chunk"][fb] == 0)
    if num > den:
        assert fb.any()
    else:
        assert not fb.any()


def test_telemetry_fallback_hand_worked_case():
    """The hand-stepped oracle case (tests/test_oracle_serving.py) on the
    library's table executor: a controller table over the analytic model and
    a hardware table 1.5 ms slower wherever a chunk runs."""
    cg, bg = [0, 1, 100, 200], [0, 1, 2]
    ctl = api.CostTable.from_samples(cg, bg, np.array([[S.analytic_cost_ns(b, c)] * 1 for b in bg for c in cg],
                                                      dtype=np.int64).reshape(len(bg), len(cg), 1))
    hw = api.CostTable.from_samples(cg, bg, np.array([[S.analytic_cost_ns(b, c) + (1_500_000 if c else 0)]
                                                      for b in bg for c in cg], dtype=np.int64)
                                    .reshape(len(bg), len(cg), 1))
    tok, its = api.serve([0, 1], [0, 0], [100, 200], [5, 3], policy=api.POLICY_SLOWEAVE, tpot_ns=50 * MS,
                         max_decode=8, margin_ns=MS, table=ctl, executor=api.EXEC_TABLE, exec_table=hw,
                         fallback_window=1)
    assert tok[0].tolist() == [2_850_000, 4_155_000, 8_560_000, 9_920_000, 11_280_000]
    assert tok[1].tolist() == [8_560_000, 9_920_000, 11_280_000]
    assert its["chunk"].tolist() == [100, 0, 200, 0, 0]
    assert ((its["flags"] & api.SERVE_FALLBACK) != 0).tolist() == [False, True, False, False, False]
    assert its["resid_p99_ns"].tolist() == [0, 1_500_000, 0, 0, 0]


def test_progress_lines_leave_the_run_unchanged(capfd):
    """log_every only writes status lines: the iteration records and token
    times are those of a silent run; a negative period is refused."""
    tr = synth.request_trace(12, 2.0, seed=5)
    quiet = serving.run(tr, policy="fixed", fixed_chunk=256, tpot_ms=25, max_decode=64)
    loud = serving.run(tr, policy="fixed", fixed_chunk=256, tpot_ms=25, max_decode=64, log_every=100)
    err = capfd.readouterr().err
    fields = [f for f in quiet.iterations.dtype.names if f != "decide_ns"]  # host timing of Alg. 1
    assert np.array_equal(quiet.iterations[fields], loud.iterations[fields])
    assert all(np.array_equal(a, b) for a, b in zip(quiet.token_ns, loud.token_ns))
    assert err.count("slw_serve:") == len(loud.iterations) // 100
    with pytest.raises(api.SloweaveError):
        serving.run(tr, policy="fixed", fixed_chunk=256, tpot_ms=25, max_decode=64, log_every=-1)

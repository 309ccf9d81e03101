"""The Sec. 4 simulator study on the library's serving loop (CPU).

Workload generator: the stated medians, mix and offered rates of Sec. 4.2
hold for the drawn traces.  Loop: on a simulator workload, the library's
loop with the analytic executor equals the serving oracle iteration for
iteration.  Study: at the 25 ms objective SLOWeave leads on the mixed and
long workloads and matches the best policy on chat, the trend of the
paper's Table 3 (its absolute numbers depend on unstated length spreads and
are not reproduced).
"""
import numpy as np
import pytest

from oracle import schedule as S
from oracle import serving as V
from paper_2609_07883_amd import api, serving, simulator, synth

MS = 1_000_000


@pytest.mark.parametrize("name", list(synth.SIM_WORKLOADS))
def test_workload_statistics(name):
    w = synth.SIM_WORKLOADS[name]
    tr = synth.sim_trace(name, 4000, seed=11)
    assert np.all(np.diff(tr.arrival_ns) >= 0) and tr.arrival_ns[0] == 0
    rate = (len(tr) - 1) / (tr.arrival_ns[-1] / 1e9)
    assert rate == pytest.approx(w.rate_per_s, rel=0.12)
    assert np.median(tr.output) == pytest.approx(w.output_median, rel=0.1)
    assert tr.prompt.min() >= 1 and tr.prompt.max() <= synth.SIM_PROMPT_CAP
    logp = np.log(tr.prompt)
    if w.long_share == 0:
        assert np.median(tr.prompt) == pytest.approx(w.prompt_median, rel=0.1)
        assert np.std(logp) == pytest.approx(synth.SIM_SIGMA, rel=0.1)
    else:   # two log-normal components: the share above their geometric midpoint
        mid = np.sqrt(w.prompt_median * w.long_median)
        z = np.log(mid / w.prompt_median) / synth.SIM_SIGMA
        from math import erf, sqrt
        p_hi = 0.5 * (1 - erf(z / sqrt(2)))            # P(short > mid) = P(long < mid)
        expect = w.long_share * (1 - p_hi) + (1 - w.long_share) * p_hi
        assert np.mean(tr.prompt > mid) == pytest.approx(expect, abs=0.03)


def test_bursty_alternates_rates():
    tr = synth.sim_trace("bursty", 6000, seed=5)
    gaps = np.diff(tr.arrival_ns) / 1e9
    # a two-state process is overdispersed: coefficient of variation of the gaps above 1
    assert np.std(gaps) / np.mean(gaps) > 1.1
    plain = synth.sim_trace("mixed", 6000, seed=5)
    g2 = np.diff(plain.arrival_ns) / 1e9
    assert np.std(g2) / np.mean(g2) == pytest.approx(1.0, abs=0.06)


def test_loop_on_a_simulator_workload_matches_oracle():
    tr = synth.sim_trace("mixed", 200, seed=2)
    cg, bg = list(range(0, 4097, 64)), list(range(0, 257))
    tab = api.CostTable.analytic(cg, bg)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, table=tab)
    reqs = [V.Request(i, int(a), int(p), int(o)) for i, (a, p, o) in enumerate(zip(tr.arrival_ns, tr.prompt, tr.output))]
    ot = S.CostTable.from_values(cg, bg, [[S.analytic_cost_ns(b, c) for c in cg] for b in bg])
    ref = V.simulate(reqs, cost_ns=S.analytic_cost_ns, tpot_ns=25 * MS, policy="sloweave", predict=ot.lookup,
                     c_last=cg[-1], c_max=4096, max_decode=256)
    for i, toks in enumerate(res.token_ns):
        assert toks.tolist() == ref.token_ns[i], f"request {i}"
    assert len(res.iterations) == len(ref.iterations)
    assert res.iterations["chunk"].tolist() == [r.chunk for r in ref.iterations]


def test_study_trends_at_25ms():
    rows = simulator.study(workloads=("chat", "mixed", "long"), tpots=(25.0,), n=1000, seeds=(0, 1))
    good = {(r["workload"], r["policy"]): r["goodput_req_s"] for r in rows}
    for wname in ("mixed", "long"):
        best_other = max(v for (w, p), v in good.items() if w == wname and p != "SLOWeave")
        assert good[(wname, "SLOWeave")] > 1.1 * best_other, wname
    best_chat = max(v for (w, p), v in good.items() if w == "chat" and p != "SLOWeave")
    assert good[("chat", "SLOWeave")] >= 0.97 * best_chat
    slw = [r for r in rows if r["policy"] == "SLOWeave"]
    assert all(r["p99_tpot_ms"] <= 25.0 + 1e-6 for r in slw)   # the controller keeps every gap within D


def test_request_classes_trend():
    """Sec. 3.5 on the simulator (mixed workload, 3% of requests interactive at
    D = 10 ms, the rest at 50 ms): with each request's own objective the
    controller keeps far more interactive requests within their SLOs than a
    controller told D = 50 ms for all, and serves both classes at least as
    well as one told D = 10 ms for all (it uses the batch slack whenever no
    interactive request decodes)."""
    from paper_2609_07883_amd import simulator as M
    rows = {r["policy"]: r for r in M.classes_study(workload="mixed", n=1000, seeds=(0,), interactive=0.03)}
    per, tight, loose = (rows["SLOWeave per-request D"], rows["SLOWeave D = 10 ms for all"],
                         rows["SLOWeave D = 50 ms for all"])
    assert per["interactive_slo_attainment"] >= loose["interactive_slo_attainment"] + 0.2
    assert per["interactive_slo_attainment"] >= tight["interactive_slo_attainment"]
    assert per["batch_slo_attainment"] >= tight["batch_slo_attainment"]
    assert per["goodput_req_s"] > tight["goodput_req_s"]


def test_first_fit_batching_trend():
    """Sec. 3.3 prefill batching on the simulator: with up to four prompts per
    iteration SLOWeave's goodput on the mixed workload at 25 ms is higher
    than with one (the fixed per-chunk cost of the analytic model is paid
    once for several short prompts), and no TPOT objective is missed more."""
    from paper_2609_07883_amd import simulator as M
    rows = {r["policy"]: r for r in M.study(workloads=("mixed",), tpots=(25.0,), n=1000, seeds=(0,),
                                            policies=(M.POLICIES[-1], M.BATCHING_POLICY))}
    one, batch = rows["SLOWeave"], rows[M.BATCHING_POLICY[0]]
    assert batch["goodput_req_s"] > 1.2 * one["goodput_req_s"]
    assert batch["p99_tpot_ms"] <= 25.0 + 1e-9

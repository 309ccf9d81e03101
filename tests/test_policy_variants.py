"""Policy variants of the serving loop (Sec. 3.3-3.5): per-request objectives and
class margins, queue disciplines, admission control, aging and first-fit
prefill batching.

The oracle is pinned first, independently of its own search code: every
decision of a run is re-derived by brute force from the token times it
produced (the active set, l_i and the pending prompts at each iteration
start are reconstructed, and the largest admissible chunk is found by
scanning the cost model), and small cases are worked out in closed form from
the analytic cost T(n, c) = 0.35 + 1[n>0](0.90 + 0.055 n) + 1[c>0](0.40 +
0.006 c) ms.  The library's loop (analytic executor, table over the same
cost model) must then equal the oracle bit for bit on random traces.
"""
import numpy as np
import pytest

from oracle import schedule as S
from oracle import serving as V
from paper_2609_07883_amd import api, serving, synth

MS = 1_000_000
C_GRID = [0, 1, 64, 512, 4096]
B_GRID = list(range(0, 257))


def _t(n, c):
    return S.analytic_cost_ns(n, c)


def _trace(n=160, rate=8.0, seed=5):
    return synth.request_trace(n, rate, seed=seed, short_median=256, long_lo=1024, long_hi=4096, output_mean=48)


def _classes(n, seed, inter_ms=10):
    """Two request classes: interactive (D inter_ms, delta 0.3 ms) and batch (D 50 ms, delta 0)."""
    rng = np.random.default_rng(seed)
    inter = rng.random(n) < 0.5
    return (np.where(inter, inter_ms * MS, 50 * MS).astype(np.int64), np.where(inter, 300_000, 0).astype(np.int64),
            np.where(inter, 500 * MS, 4000 * MS).astype(np.int64))


def _reqs(tr, tpot=None, margin=None, ttft=None):
    out = []
    for i, (a, p, o) in enumerate(zip(tr.arrival_ns, tr.prompt, tr.output)):
        out.append(V.Request(i, int(a), int(p), int(o), int(tpot[i]) if tpot is not None else 0,
                             int(margin[i]) if margin is not None else -1, int(ttft[i]) if ttft is not None else 0))
    return out


def _replay(reqs, tr, D, margin, c_max, queue="oldest"):
    """Brute-force re-derivation of every decision of an oracle run (oldest /
    srpt / edf queue, no decode cap, no aging, one prompt per iteration)."""
    tok = {rid: np.asarray(v, dtype=np.int64) for rid, v in tr.token_ns.items()}
    done = {r.rid: 0 for r in reqs}
    decided = 0
    for it in tr.iterations:
        t = it.start_ns
        arrived = [r for r in reqs if r.arrival_ns <= t and r.rid not in tr.rejected]
        active = [r for r in arrived if 0 < np.sum(tok[r.rid] <= t) < r.output]
        assert it.n_decode == len(active)
        dl = {r.rid: int(tok[r.rid][tok[r.rid] <= t].max()) + (r.tpot_ns or D) for r in active}
        assert it.budget_ns == (min(dl.values()) - t if active else 0)
        pending = [r for r in arrived if done[r.rid] < r.prompt]
        if queue == "srpt":
            pending.sort(key=lambda r: (r.prompt - done[r.rid], r.arrival_ns, r.rid))
        elif queue == "edf":
            pending.sort(key=lambda r: (r.arrival_ns + r.ttft_ns if r.ttft_ns else float("inf"), r.arrival_ns, r.rid))
        else:
            pending.sort(key=lambda r: (r.arrival_ns, r.rid))
        if not pending:
            assert it.chunk == 0
            continue
        head = pending[0]
        cap = min(head.prompt - done[head.rid], c_max)
        if active:
            # the chunk must satisfy T(n, c) + delta_i <= d_i - t for every active i
            room = min(dl[r.rid] - t - (r.margin_ns if r.margin_ns >= 0 else margin) for r in active)
            cs = np.arange(cap + 1)
            cost = np.where(cs > 0, 400_000 + 6_000 * cs, 0) + _t(len(active), 0)
            ok = np.nonzero(cost <= room)[0]
            exp = int(ok.max()) if len(ok) else 0
        else:
            exp = cap
        assert it.chunk == exp, f"iteration at {t}: chunk {it.chunk}, brute force {exp}"
        if exp:
            assert it.prefill_rid == head.rid
            done[head.rid] += exp
            decided += 1
        assert it.end_ns - t == _t(len(active), it.chunk)
    return decided


@pytest.mark.parametrize("queue", ["oldest", "srpt", "edf"])
def test_oracle_decisions_by_brute_force(queue):
    tr = _trace(120, 6.0, seed=2)
    tpot, margin, ttft = _classes(len(tr), 4)
    reqs = _reqs(tr, tpot, margin, ttft)
    ref = V.simulate(reqs, cost_ns=_t, tpot_ns=25 * MS, policy="sloweave", c_max=2048, margin_ns=100_000,
                     queue=queue)
    assert _replay(reqs, ref, 25 * MS, 100_000, 2048, queue) > 50


@pytest.mark.parametrize("queue,expect", [("oldest", [0, 1, 2]), ("srpt", [1, 2, 0]), ("edf", [2, 1, 0])])
def test_oracle_queue_order_closed_form(queue, expect):
    """Three one-token requests at t = 0 with prompts 300 / 100 / 200 and TTFT
    objectives none / 300 ms / 100 ms: with no decode active each iteration
    runs one whole prompt, in the queue's order (a request without a TTFT
    objective goes last under earliest-deadline queueing)."""
    reqs = [V.Request(0, 0, 300, 1), V.Request(1, 0, 100, 1, ttft_ns=300 * MS), V.Request(2, 0, 200, 1, ttft_ns=100 * MS)]
    tr = V.simulate(reqs, cost_ns=_t, tpot_ns=25 * MS, policy="sloweave", c_max=4096, queue=queue)
    assert [it.prefill_rid for it in tr.iterations] == expect
    assert [it.chunk for it in tr.iterations] == [reqs[i].prompt for i in expect]


def test_oracle_admission_closed_form():
    """20 requests at t = 0, D = 2 ms, admit at D: T(n, 0) = 1.25 + 0.055 n ms
    admits n <= 13 with delta 0 and n <= 10 with delta 0.2 ms (even ids)."""
    reqs = [V.Request(i, 0, 64, 50, 0, 200_000 if i % 2 == 0 else 0) for i in range(20)]
    tr = V.simulate(reqs, cost_ns=_t, tpot_ns=2 * MS, policy="sloweave", admit_ppm=1_000_000)
    assert sorted(set(range(20)) - tr.rejected) == list(range(10)) + [11, 13, 15]
    for rid in tr.rejected:
        assert tr.token_ns[rid] == []
    assert all(len(tr.token_ns[r.rid]) == r.output for r in reqs if r.rid not in tr.rejected)


def test_oracle_aging_bounds_starvation():
    """A decode at D = 1.4 ms leaves no room for any chunk (T(1, 1) = 1.711 ms):
    without aging the long prompt waits for the decode to finish; with aging
    every chunk is forced, at least aging_ns after the previous one and at
    most one iteration later, and the decode's deadline slips only then."""
    reqs = [V.Request(0, 0, 16, 400), V.Request(1, MS, 2000, 2)]
    kw = dict(cost_ns=_t, tpot_ns=1_400_000, policy="sloweave", c_max=4096)
    plain = V.simulate(reqs, **kw)
    first1 = min(it.start_ns for it in plain.iterations if it.prefill_rid == 1)
    assert first1 >= plain.token_ns[0][-1]
    aged = V.simulate(reqs, aging_ns=20 * MS, aging_chunk=256, **kw)
    runs = [it for it in aged.iterations if it.prefill_rid == 1]
    assert [it.chunk for it in runs] == [256] * 7 + [208] and all(it.aged for it in runs)
    waited = [MS] + [it.end_ns for it in runs[:-1]]
    for w, it in zip(waited, runs):
        assert 20 * MS <= it.start_ns - w < 20 * MS + _t(1, 256)
    gaps = np.diff(aged.token_ns[0])
    late = gaps[gaps > 1_400_000]
    assert late.tolist() == [_t(1, 256)] * 7 + [_t(1, 208)]


def test_oracle_prefill_batching_closed_form():
    """Five one-token requests of 100-token prompts at t = 0, c_max 256, up to
    four prompts per iteration: 100 + 100 + 56, then 44 + 100 + 100."""
    reqs = [V.Request(i, 0, 100, 1) for i in range(5)]
    tr = V.simulate(reqs, cost_ns=_t, tpot_ns=25 * MS, policy="sloweave", c_max=256, max_prefills=4)
    assert [(it.chunk, it.n_prefill) for it in tr.iterations] == [(256, 3), (244, 3)]
    t1 = _t(0, 256)
    assert [tr.token_ns[i][0] for i in range(5)] == [t1, t1, t1 + _t(0, 244), t1 + _t(0, 244), t1 + _t(0, 244)]


def test_oracle_prefill_batching_is_first_fit():
    """With decodes active, every iteration's prefill total S meets the budget,
    and unless S is at c_max, the prompt count is at its cap or no prompt
    tokens are left waiting, one more token would not (T(n, S + 1) > budget)."""
    tr = synth.request_trace(300, 10.0, seed=6, short_median=48, long_lo=256, long_hi=1024, output_mean=48)
    reqs = _reqs(tr)
    ref = V.simulate(reqs, cost_ns=_t, tpot_ns=5 * MS, policy="sloweave", c_max=2048, max_prefills=8)
    placed = 0
    checked = 0
    for it in ref.iterations:
        waiting = sum(r.prompt for r in reqs if r.arrival_ns <= it.start_ns) - placed
        if it.n_decode and it.chunk:
            assert _t(it.n_decode, it.chunk) <= it.budget_ns
        if it.n_decode and it.chunk < 2048 and waiting > it.chunk and it.n_prefill < 8:
            assert _t(it.n_decode, it.chunk + 1) > it.budget_ns
            checked += 1
        placed += it.chunk
    assert checked > 10
    assert sum(it.n_prefill > 1 for it in ref.iterations) > 10
    single = V.simulate(reqs, cost_ns=_t, tpot_ns=5 * MS, policy="sloweave", c_max=2048)
    assert max(it.n_prefill for it in single.iterations) == 1


def _compare(res, ref):
    for i, toks in enumerate(res.token_ns):
        exp = ref.token_ns[i] if i not in ref.rejected else [-1] * len(toks)
        assert toks.tolist() == exp, f"request {i}"
    it = res.iterations
    assert len(it) == len(ref.iterations)
    got = np.stack([it["start_ns"], it["end_ns"], it["chunk"], it["n_decode"], it["prefill_id"], it["budget_ns"],
                    it["n_prefill"], (it["flags"] & api.SERVE_AGED) != 0], 1)
    exp = np.array([[r.start_ns, r.end_ns, r.chunk, r.n_decode, r.prefill_rid, r.budget_ns, r.n_prefill, r.aged]
                    for r in ref.iterations])
    bad = np.nonzero((got != exp).any(1))[0]
    assert len(bad) == 0, f"first differing iteration {bad[0]}: {got[bad[0]]} vs {exp[bad[0]]}"


VARIANTS = [  # (name, interactive D in ms, options)
    ("classes", 10, dict()),
    ("srpt", 10, dict(queue="srpt")),
    ("edf", 10, dict(queue="edf")),
    ("admission", 10, dict(admit_ppm=190_000)),
    ("aging", 2, dict(aging_ns=40 * MS, aging_chunk=128)),
    ("batching", 10, dict(max_prefills=4)),
    ("all", 2, dict(queue="srpt", admit_ppm=900_000, aging_ns=40 * MS, aging_chunk=128, max_prefills=4)),
]


@pytest.mark.parametrize("name,inter_ms,kw", VARIANTS, ids=[v[0] for v in VARIANTS])
def test_loop_matches_oracle(name, inter_ms, kw):
    tr = _trace(200, 9.0, seed=8)
    tpot, margin, ttft = _classes(len(tr), 9, inter_ms)
    tab = api.CostTable.analytic(C_GRID, B_GRID)
    res = serving.run(tr, policy="sloweave", tpot_ms=25, max_decode=256, c_max=2048, table=tab, margin_ns=50_000,
                      slo_tpot_ms=tpot / MS, slo_margin_ns=margin, slo_ttft_ms=ttft / MS, **kw)
    ot = S.CostTable.from_values(C_GRID, B_GRID, [[_t(b, c) for c in C_GRID] for b in B_GRID])
    ref = V.simulate(_reqs(tr, tpot, margin, ttft), cost_ns=_t, predict=ot.lookup, c_last=C_GRID[-1],
                     tpot_ns=25 * MS, policy="sloweave", c_max=2048, margin_ns=50_000, max_decode=256, **kw)
    _compare(res, ref)
    m = serving.metrics(tr, res.token_ns, ttft / MS, tpot / MS)
    s = V.summarize(_reqs(tr, tpot, margin, ttft), ref.token_ns, 0, 0, rejected=ref.rejected)
    assert m["rejected"] == s["rejected"] == len(ref.rejected)
    if name in ("admission", "all"):
        assert 0 < len(ref.rejected) < len(tr)
    if name in ("aging", "all"):
        assert sum(r.aged for r in ref.iterations) > 10
    if name in ("batching", "all"):
        assert sum(r.n_prefill > 1 for r in ref.iterations) > 10


def test_fixed_policy_with_classes_matches_oracle():
    tr = _trace(150, 9.0, seed=10)
    tpot, margin, ttft = _classes(len(tr), 11)
    res = serving.run(tr, policy="fixed", fixed_chunk=256, tpot_ms=25, max_decode=64, slo_tpot_ms=tpot / MS,
                      queue="edf", slo_ttft_ms=ttft / MS)
    ref = V.simulate(_reqs(tr, tpot, None, ttft), cost_ns=_t, tpot_ns=25 * MS, policy="fixed", fixed_chunk=256,
                     max_decode=64, queue="edf")
    _compare(res, ref)


def test_variant_argument_errors():
    tr = _trace(10, 5.0, seed=1)
    tab = api.CostTable.analytic(C_GRID, B_GRID)
    base = dict(policy="sloweave", tpot_ms=25, max_decode=16, table=tab)
    with pytest.raises(api.SloweaveError):  # negative admission threshold
        api.serve(np.arange(10), tr.arrival_ns, tr.prompt, tr.output, policy=0, tpot_ns=25 * MS, max_decode=16,
                  table=tab, admit_ppm=-1)
    with pytest.raises(api.SloweaveError):  # aging without a chunk size
        serving.run(tr, aging_ns=MS, **base)
    with pytest.raises(api.SloweaveError):  # admission without a table
        serving.run(tr, policy="fixed", fixed_chunk=64, tpot_ms=25, max_decode=16, admit_ppm=500_000)
    with pytest.raises(api.SloweaveError) as e:  # a GPU iteration takes at most SLW_MAX_PREFILLS prompts
        api.serve(np.arange(10), tr.arrival_ns, tr.prompt, tr.output, policy=0, tpot_ns=25 * MS, max_decode=16,
                  table=tab, executor=api.EXEC_GPU, max_prefills=api.MAX_PREFILLS + 1)
    assert e.value.code == api.ERANGE

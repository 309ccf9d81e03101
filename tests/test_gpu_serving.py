"""The serving loop on the GPU executor (through the C ABI), on a 2-layer Tiny stack.

Each iteration really runs on the device and is timed on the host clock, so
token times are not reproducible; what must hold exactly is checked instead:
every SLOWeave decision replays bit-exactly through the oracle's Alg. 1 on
the same measured table (the record holds the decision's inputs: start
time, earliest deadline, decode count, remaining prompt); each request gets
its output tokens in order after its arrival; chunks add up to the prompts;
the decode batch respects its cap; the KV pool is whole again at the end;
fixed-chunk runs cut prompts into min(chunk, remaining) pieces.
"""
import numpy as np
import pytest

from oracle import schedule as S
from paper_2609_07883_amd import api, serving, synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

C_GRID = [0, 16, 32, 64, 128, 256]
B_GRID = [0, 1, 2, 4, 8, 16]


@pytest.fixture(scope="module")
def setup():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_07883_amd.runtime import Session
    sess = Session(synth.with_layers(synth.TINY, 2), num_blocks=1024, max_c=256, max_b=16)
    ct = sess.ctx.build_cost_table(C_GRID, B_GRID, prefix_len=64, ctx_lo=16, ctx_hi=128, seed=3, warmup=1,
                                   repeats=5, x_in=sess.x_in.data_ptr(), x_out=sess.x_out.data_ptr(),
                                   ws=sess.ws.data_ptr(), ws_bytes=sess.ws_bytes,
                                   stream=sess.stream())
    tr = synth.request_trace(40, 400.0, seed=9, short_median=48, long_lo=128, long_hi=400, output_mean=6)
    return sess, ct, tr


def _check_run(sess, tr, res, max_decode):
    n = len(tr)
    for i in range(n):
        t = res.token_ns[i]
        assert len(t) == tr.output[i]
        assert t[0] > tr.arrival_ns[i] and np.all(np.diff(t) > 0)
    it = res.iterations
    assert np.all(it["end_ns"] > it["start_ns"])
    assert np.all(it["start_ns"][1:] >= it["end_ns"][:-1])
    assert it["n_decode"].max() <= max_decode
    per = np.zeros(n, np.int64)
    np.add.at(per, it["prefill_id"][it["chunk"] > 0], it["chunk"][it["chunk"] > 0])
    assert per.tolist() == tr.prompt.tolist()
    assert sess.ctx.free_blocks() == sess.num_blocks


@pytest.mark.parametrize("tpot_ms,margin_us", [(4.0, 0), (1.5, 200)])
def test_sloweave_on_gpu(setup, tpot_ms, margin_us):
    sess, ct, tr = setup
    res = serving.run(tr, policy="sloweave", tpot_ms=tpot_ms, max_decode=16, c_max=256, table=ct,
                      margin_ns=margin_us * 1000, session=sess)
    torch.cuda.synchronize()
    _check_run(sess, tr, res, 16)
    ot = S.CostTable(C_GRID, B_GRID, ct.values(api.TABLE_SAMPLES).tolist())
    decided = 0
    for r in res.iterations:
        if r["remaining"] <= 0:
            continue
        n = int(r["n_decode"])
        dl = [int(r["start_ns"] + r["budget_ns"])] * n
        exp = S.select_chunk_table(ot, dl, int(r["start_ns"]), int(r["remaining"]), 256, margin_us * 1000)
        assert int(r["chunk"]) == exp[0], f"record {r}"
        assert int(r["flags"]) & 0xFF == exp[1]
        decided += 1
    assert decided > 10
    print(f"D={tpot_ms} ms: {len(res.iterations)} iterations, "
          f"{serving.metrics(tr, res.token_ns, 1000, tpot_ms)}")


def test_fixed_on_gpu(setup):
    sess, _, tr = setup
    res = serving.run(tr, policy="fixed", fixed_chunk=64, tpot_ms=4.0, max_decode=4, session=sess)
    torch.cuda.synchronize()
    _check_run(sess, tr, res, 4)
    it = res.iterations
    run = it[it["chunk"] > 0]
    assert np.all(run["chunk"] == np.minimum(64, run["remaining"]))
    assert np.all(it[(it["flags"] & api.SERVE_DECODE_CAP) != 0]["chunk"] == 0)


def test_kv_wait_when_the_pool_is_small(setup):
    """A pool that holds only a few requests at a time delays prompts instead of failing."""
    from paper_2609_07883_amd.runtime import Session
    _, _, tr = setup
    need = max(int(-(-(p + o - 1) // 16)) for p, o in zip(tr.prompt, tr.output))
    sess = Session(synth.with_layers(synth.TINY, 2), num_blocks=need + 8, max_c=256, max_b=16)
    res = serving.run(tr, policy="fixed", fixed_chunk=128, tpot_ms=4.0, max_decode=16, session=sess)
    torch.cuda.synchronize()
    _check_run(sess, tr, res, 16)
    assert np.any(res.iterations["flags"] & api.SERVE_KV_WAIT)


def test_telemetry_margin_on_gpu(setup):
    """With the telemetry window on, every decision's margin is the nearest-rank
    P99 of the relative residuals of the chunked iterations before it (recomputed
    from the records), and the chunk is Alg. 1 on the widened predictions."""
    sess, ct, tr = setup
    W = 8
    res = serving.run(tr, policy="sloweave", tpot_ms=3.0, max_decode=16, c_max=256, table=ct,
                      residual_window=W, session=sess)
    torch.cuda.synchronize()
    _check_run(sess, tr, res, 16)
    ot = S.CostTable(C_GRID, B_GRID, ct.values(api.TABLE_SAMPLES).tolist())
    resid = []
    checked = 0
    for r in res.iterations:
        if r["remaining"] > 0:
            q = min(max(S.nearest_rank(resid[-W:], 99, 100), 0), 10**8) if resid else 0
            assert int(r["rel_margin_ppm"]) == q
            n = int(r["n_decode"])

            def widened(nn, cc, q=q):
                v = ot.lookup(nn, cc)
                return v + -(-q * v // 10**6)
            exp = S.select_chunk(widened, [int(r["start_ns"] + r["budget_ns"])] * n, int(r["start_ns"]),
                                 int(r["remaining"]), 256, 0, c_last=C_GRID[-1])
            assert int(r["chunk"]) == exp[0]
            checked += 1
        if r["chunk"] > 0 and r["predicted_ns"] > 0:
            pred = int(r["predicted_ns"])
            resid.append((int(r["end_ns"]) - int(r["start_ns"]) - pred) * 10**6 // pred)
    assert checked > 10


def _check_variant_run(sess, tr, res, queue_key):
    n = len(tr)
    served = [i for i in range(n) if res.token_ns[i][0] >= 0]
    for i in range(n):
        t = res.token_ns[i]
        if i in served:
            assert t[0] > tr.arrival_ns[i] and np.all(np.diff(t) > 0)
        else:
            assert np.all(t == -1)
    it = res.iterations
    assert it["n_decode"].max() <= 16 and np.all(it["n_prefill"] <= 1)
    done = np.zeros(n, np.int64)
    aged = 0
    for r in it:
        if r["chunk"] > 0:
            waiting = [i for i in served if tr.arrival_ns[i] <= r["start_ns"] and done[i] < tr.prompt[i]]
            best = min(waiting, key=lambda i: queue_key(i, done))
            assert r["prefill_id"] == best
            if r["flags"] & api.SERVE_AGED:
                assert r["chunk"] == min(32, tr.prompt[best] - done[best])
                aged += 1
            done[best] += r["chunk"]
    assert done[served].tolist() == [int(tr.prompt[i]) for i in served]
    assert sess.ctx.free_blocks() == sess.num_blocks
    return n - len(served), aged


def test_policy_variants_on_gpu(setup):
    """Request classes with shortest-remaining-prompt queueing and admission
    control, then aging, on the GPU executor: every chunk goes to the prompt
    the queue puts first, refused requests emit nothing, aged chunks are
    min(aging_chunk, remaining) and the pool is whole at the end.

    Admission: twelve requests arrive together, so every admission decision
    is taken before anything runs and the refused set follows from the
    measured table alone (interactive D = 4 T_hat(1, 0), admitted while the
    decode batch they join costs at most halfway between the cheapest and the
    dearest decode-only row; batch D 20x larger)."""
    sess, ct, tr = setup
    t_dec = ct.lookup(1, 0)
    n = 12
    burst = synth.RequestTrace(np.full(n, 1000, np.int64), np.arange(20, 20 + 7 * n, 7, dtype=np.int64),
                               np.full(n, 8, np.int64))
    inter = np.arange(n) % 2 == 0
    d_ns = np.where(inter, 4 * t_dec, 80 * t_dec).astype(np.int64)
    # threshold halfway between the cheapest and the dearest decode-only row
    rows = [ct.lookup(b, 0) for b in (1, 2, 4, 8, 16)]
    assert max(rows) > min(rows)
    admit = int((min(rows) + max(rows)) // 2 * 1_000_000 // (4 * t_dec))
    res = serving.run(burst, policy="sloweave", tpot_ms=4.0, max_decode=16, c_max=256, table=ct, session=sess,
                      slo_tpot_ms=d_ns / 1e6, queue="srpt", admit_ppm=admit)
    torch.cuda.synchronize()
    refused, _ = _check_variant_run(sess, burst, res,
                                    lambda i, done: (burst.prompt[i] - done[i], burst.arrival_ns[i], i))
    expect, admitted = [], 0
    for i in range(n):
        if ct.lookup(admitted + 1, 0) * 1_000_000 > d_ns[i] * admit:
            expect.append(i)
        else:
            admitted += 1
    assert [i for i in range(n) if res.token_ns[i][0] < 0] == expect and refused == len(expect) > 0
    # aging: a D below one decode-only iteration leaves no admissible chunk
    res = serving.run(tr, policy="sloweave", tpot_ms=0.5 * t_dec / 1e6, max_decode=16, c_max=256, table=ct,
                      session=sess, aging_ns=int(2 * t_dec), aging_chunk=32)
    torch.cuda.synchronize()
    _, aged = _check_variant_run(sess, tr, res, lambda i, done: (tr.arrival_ns[i], i))
    assert aged > 0
    print(f"variants: {refused} refused, {aged} aged chunks")


def test_telemetry_fallback_on_gpu(setup):
    """Sec. 5.1's decode-only fallback on measured iterations: the controller
    reads a table at half the measured times, so observed residuals exceed the
    50 us margin.  Replayed from the records: each decision's window P99 is
    the nearest-rank P99 of the absolute residuals of the priced iterations
    before it; above the margin (with a prompt to serve and decodes active)
    the iteration is decode-only and flagged, otherwise the chunk is Alg. 1
    on the optimistic table.  Prompts still finish."""
    sess, ct, tr = setup
    FW, margin = 4, 50_000
    samples = ct.values(api.TABLE_SAMPLES)
    fast = api.CostTable.from_samples(C_GRID, B_GRID, samples // 2)
    res = serving.run(tr, policy="sloweave", tpot_ms=3.0, max_decode=16, c_max=256, table=fast,
                      margin_ns=margin, fallback_window=FW, session=sess)
    torch.cuda.synchronize()
    _check_run(sess, tr, res, 16)
    ot = S.CostTable(C_GRID, B_GRID, (samples // 2).tolist())
    window, events, decided = [], 0, 0
    for r in res.iterations:
        fb = bool(int(r["flags"]) & api.SERVE_FALLBACK)
        if r["remaining"] > 0:
            n = int(r["n_decode"])
            p99 = S.nearest_rank(window[-FW:], 99, 100) if window and n > 0 else 0
            assert int(r["resid_p99_ns"]) == p99
            if n > 0 and window and p99 > margin:
                assert fb and int(r["chunk"]) == 0
                events += 1
            else:
                assert not fb
                exp = S.select_chunk_table(ot, [int(r["start_ns"] + r["budget_ns"])] * n, int(r["start_ns"]),
                                           int(r["remaining"]), 256, margin)
                assert int(r["chunk"]) == exp[0]
                decided += 1
        else:
            assert not fb
        if r["predicted_ns"] > 0:
            window.append(int(r["end_ns"]) - int(r["start_ns"]) - int(r["predicted_ns"]))
    print(f"fallback: {events} events, {decided} Alg. 1 decisions, {len(res.iterations)} iterations")
    assert events > 0 and decided > 0


def test_prefill_batching_on_gpu(setup):
    """First-fit prefill batching (Sec. 3.3) on the GPU executor: iterations
    that finish one prompt take the next ones in queue order.  Checked from
    the records: some iterations serve several prompts; every prompt token
    runs exactly once (the chunks add up to the prompts); every chunked
    iteration beside decodes keeps its predicted time within the budget, the
    total included (Prop. 1's safety on the table); tokens come in order; the
    pool is whole at the end."""
    sess, ct, _ = setup
    # bursts of short prompts: several fit one iteration
    n = 24
    tr = synth.RequestTrace(np.repeat(np.arange(4, dtype=np.int64) * 30_000_000, 6),
                            np.arange(n, dtype=np.int64) * 7 % 50 + 12, np.full(n, 3, np.int64))
    res = serving.run(tr, policy="sloweave", tpot_ms=4.0, max_decode=16, c_max=256, table=ct, session=sess,
                      max_prefills=4)
    torch.cuda.synchronize()
    for i in range(n):
        t = res.token_ns[i]
        assert len(t) == tr.output[i] and t[0] > tr.arrival_ns[i] and np.all(np.diff(t) > 0)
    it = res.iterations
    assert int(it["chunk"].sum()) == int(tr.prompt.sum())
    assert it["n_prefill"].max() > 1 and np.all(it["n_prefill"][it["chunk"] > 0] >= 1)
    assert np.all(it["chunk"] <= 256) and it["n_decode"].max() <= 16
    chunked = it[(it["chunk"] > 0) & (it["n_decode"] > 0)]
    assert np.all(chunked["predicted_ns"] <= chunked["budget_ns"])
    assert sess.ctx.free_blocks() == sess.num_blocks
    print(f"batching: {int(np.sum(it['n_prefill'] > 1))} of {len(it)} iterations serve several prompts "
          f"(up to {int(it['n_prefill'].max())})")

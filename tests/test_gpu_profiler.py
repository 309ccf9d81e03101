"""The profiler and controller on a measured table (GPU), through the C ABI.

slw_build_cost_table times real mixed iterations over a (decode batch) x
(chunk) grid (Sec. 5.1).  Everything derived from the raw samples must match
the oracle bit-exactly: nearest-rank P50/P99, the running maximum along the
chunk axis, interpolated lookups and the chunk Alg. 1 selects; the table the
controller reads must be monotone in C; the temporary sequences must be
returned to the pool.
"""
import math

import numpy as np
import pytest

from oracle import schedule as S
from paper_2609_07883_amd import api, synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def measured():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_07883_amd.runtime import Session
    sess = Session(synth.TINY, num_blocks=256, max_c=128, max_b=4)
    flush = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    free0 = sess.ctx.free_blocks()
    c_grid, b_grid = [0, 16, 32, 64, 128], [0, 1, 4]
    ct = sess.ctx.build_cost_table(c_grid, b_grid, prefix_len=64, ctx_lo=16, ctx_hi=64, seed=3,
                                   warmup=1, repeats=7, x_in=sess.x_in.data_ptr(),
                                   x_out=sess.x_out.data_ptr(), ws=sess.ws.data_ptr(),
                                   ws_bytes=sess.ws_bytes, flush_buf=flush.data_ptr(),
                                   flush_bytes=flush.numel(),
                                   stream=torch.cuda.current_stream().cuda_stream)
    return sess, ct, c_grid, b_grid, free0


def test_table_statistics_match_oracle(measured):
    sess, ct, c_grid, b_grid, free0 = measured
    samples = ct.values(api.TABLE_SAMPLES)
    assert samples.shape == (len(b_grid), len(c_grid), 7)
    assert (samples > 0).all()
    ot = S.CostTable(c_grid, b_grid, samples.tolist())
    assert ct.values(api.TABLE_P50).tolist() == ot.p50
    assert ct.values(api.TABLE_P99).tolist() == ot.p99
    t_hat = ct.values(api.TABLE_THAT)
    assert t_hat.tolist() == ot.t_hat
    assert (np.diff(t_hat, axis=1) >= 0).all()          # monotone in C for the controller
    assert ct.monotone() == ot.monotone_violations()
    assert sess.ctx.free_blocks() == free0               # temporary sequences released


def test_controller_on_measured_table_matches_oracle(measured):
    sess, ct, c_grid, b_grid, _ = measured
    ot = S.CostTable(c_grid, b_grid, ct.values(api.TABLE_SAMPLES).tolist())
    rng = np.random.default_rng(0)
    lo, hi = int(ot.t_hat[0][0]), int(max(max(r) for r in ot.t_hat))
    for _ in range(300):
        n = int(rng.integers(0, 5))
        now = int(rng.integers(0, 10**9))
        budget = int(rng.integers(lo // 2, 2 * hi + 2))
        dl = (now + budget + rng.integers(0, 10**5, size=n)).tolist()
        rem = int(rng.integers(-1, 300))
        cmax = int(rng.integers(0, 300))
        margin = int(rng.integers(0, 10**5))
        got = api.select_chunk(ct, dl, now, rem, cmax, margin)
        want = S.select_chunk_table(ot, dl, now, rem, cmax, margin)
        # chunk and flags as the oracle's bisection; the library searches for
        # the same first infeasible chunk in its own order, with as many
        # lookups as a bisection over [0, C_max] at most
        assert got[:2] == want[:2]
        assert got[2] <= math.ceil(math.log2(max(cmax, 1) + 2)) + 2
    for n in range(0, 5):
        for c in range(0, 129, 5):
            assert ct.lookup(n, c) == ot.lookup(n, c)


def test_iterations_still_correct_after_profiling(measured):
    """The profiler's temporary sequences do not disturb later iterations."""
    from tests.parity import Mirror, check
    sess, *_ = measured
    mir = Mirror(sess)
    mir.create(1)
    mir.install_context(1, 50)
    mir.create(2)
    b = api.Batch(40, 2, 0, [1], [50])
    y, yr, sg, sr = mir.step(b, synth.embeddings(41, 256, seed=1, stream=77))
    assert sg == sr
    check(y, yr, "after profiling")


def test_context_table_on_gpu():
    """slw_build_cost_table_ctx: one plane per cached-context point, its
    statistics and lookups bit-exact against the oracle on the exported
    samples, monotone along C in every plane, temporary sequences released."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_07883_amd.runtime import Session
    sess = Session(synth.TINY, num_blocks=256, max_c=128, max_b=4)
    free0 = sess.ctx.free_blocks()
    c_grid, b_grid, p_grid = [0, 32, 128], [0, 2, 4], [0, 256, 1024]
    ct = sess.ctx.build_cost_table(c_grid, b_grid, prefix_len=0, ctx_lo=16, ctx_hi=64, seed=5, warmup=1,
                                   repeats=5, x_in=sess.x_in.data_ptr(), x_out=sess.x_out.data_ptr(),
                                   ws=sess.ws.data_ptr(), ws_bytes=sess.ws_bytes,
                                   stream=torch.cuda.current_stream().cuda_stream, p_grid=p_grid)
    assert ct.prefixes().tolist() == p_grid
    samples = ct.values(api.TABLE_SAMPLES)
    assert samples.shape == (3, 3, 3, 5) and (samples > 0).all()
    ot = S.CostTable(c_grid, b_grid, samples.tolist(), p_grid)
    assert ct.values(api.TABLE_THAT).tolist() == ot.t_hat
    assert (np.diff(ct.values(api.TABLE_THAT), axis=2) >= 0).all()
    for p in (0, 1, 256, 257, 1024):
        for n in range(0, 5):
            for c in range(0, 129, 16):
                assert ct.lookup(n, c, p) == ot.lookup(n, c, p)
    assert sess.ctx.free_blocks() == free0

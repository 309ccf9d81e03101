"""GPU parity of the mixed iteration against the oracle, through the C ABI.

Block tables and slots must match the oracle's block-manager twin
bit-exactly; outputs and appended K/V must match the float64 oracle within
the 2e-2 relative bound (see tests/parity.py for the denominator).

Shapes: the Tiny model (d 256, 4 MHA heads of 64, FFN 704) run as a 512-token
prompt in four 128-token chunks next to four decodes whose contexts
(uniform in [64, 256]) are themselves built by prefill iterations; and the
8B-shaped layer (d 4096, 32/8 GQA heads of 128, FFN 14336) at small ragged
batches covering the degenerate cases (decode-only, prefill-only, empty
prefix, context 0 and 1, chunks of 1, block-boundary crossings, several
attention tiles with ragged tails).
"""
import numpy as np
import pytest

from paper_2609_07883_amd import api, synth
from tests.parity import TOL, Mirror, check, rel_err, stage_errors

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def tiny_sessions():
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    return {qk: Session(synth.TINY, num_blocks=256, max_c=256, max_b=4, qk_std=qk)
            for qk in (None, 0.16)}


@pytest.mark.parametrize("qk_std", [None, 0.16], ids=["plain", "sharp"])
def test_tiny_prompt_in_chunks_with_decodes(tiny_sessions, qk_std):
    sess = tiny_sessions[qk_std]
    mir = Mirror(sess)
    ctx_lens = synth.uniform_lengths(4, 64, 256, seed=2).tolist()
    dec = [11, 12, 13, 14]
    stream = 0
    for sid, L in zip(dec, ctx_lens):          # contexts built by prefill iterations
        mir.create(sid)
        x = synth.embeddings(L, synth.TINY.d_model, seed=1, stream=100 + sid)
        b = api.Batch(L, sid, 0, [], [])
        y, yr, sg, sr = mir.step(b, x)
        assert sg == sr
        check(y, yr, f"context prefill of seq {sid}")
    prompt = 99
    mir.create(prompt)
    xp = synth.embeddings(512, synth.TINY.d_model, seed=1, stream=0)
    lens = list(ctx_lens)
    for it in range(4):
        xd = synth.embeddings(4, synth.TINY.d_model, seed=1, stream=200 + it)
        b = api.Batch(128, prompt, 128 * it, dec, lens)
        y, yr, sg, sr = mir.step(b, np.concatenate([xp[128 * it: 128 * (it + 1)], xd]))
        assert sg == sr, f"slots differ at iteration {it}"
        check(y, yr, f"iteration {it}")
        assert mir.kv_error(b) <= TOL
        for sid in dec + [prompt]:
            assert sess.ctx.block_table(sid) == mir.mgr.block_table(sid)
        lens = [L + 1 for L in lens]
        stream += 1


def test_tiny_long_chunk_stream_k():
    """903 rows (a 900-token chunk at prefix 100 and three decodes): the
    output projection (256 x 256 wide) runs the stream-K schedule, whose
    pieces and fixup must reproduce every row."""
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    sess = Session(synth.TINY, num_blocks=512, max_c=1024, max_b=4, qk_std=0.16)
    mir = Mirror(sess)
    pre = 7
    mir.create(pre)
    mir.install_context(pre, 100)
    dec = [21, 22, 23]
    ctx = [40, 130, 257]
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, L)
    b = api.Batch(900, pre, 100, dec, ctx)
    x = synth.embeddings(b.rows, synth.TINY.d_model, seed=1, stream=903)
    y, yr, sg, sr = mir.step(b, x)
    assert sg == sr
    check(y, yr, "903-row iteration")
    assert mir.kv_error(b) <= TOL


@pytest.mark.parametrize("C", [100, 150, 600, 850, 1000])
def test_tiny_gemm_plan_bands(C):
    """Row counts in several of the GEMM planner's bands on the Tiny shapes
    (narrow projections: the tile fallbacks for widths that are not a
    multiple of 256, forced splits refused where k does not divide): every
    row of the iteration against the oracle."""
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    sess = Session(synth.TINY, num_blocks=512, max_c=1024, max_b=4, qk_std=0.16)
    mir = Mirror(sess)
    pre = 7
    mir.create(pre)
    mir.install_context(pre, 64)
    dec = [21, 22, 23]
    ctx = [17, 300, 64]
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, L)
    b = api.Batch(C, pre, 64, dec, ctx)
    x = synth.embeddings(b.rows, synth.TINY.d_model, seed=1, stream=C)
    y, yr, sg, sr = mir.step(b, x)
    assert sg == sr
    check(y, yr, f"{b.rows}-row iteration")


@pytest.fixture(scope="module")
def l8b():
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    return Session(synth.LLAMA8B_LAYER, num_blocks=2048, max_c=512, max_b=8)


CASES = [
    # (C, P, decode contexts)
    (77, 50, [1, 16, 33, 100, 300]),
    (0, 0, [0, 15, 16, 17, 1000]),
    (200, 0, []),
    (33, 1000, [64]),
    (1, 7, [5]),
    (130, 16, [2047, 4]),
    (512, 3, [700, 1, 63, 64, 65, 127, 128, 129]),
    (64, 8192, [1000, 3]),        # few query tiles: key axis split across work-groups
    (100, 3000, []),              # split with a ragged final tile
    (512, 0, [2]),                # 8 query tiles, split with a causal diagonal in every tile
]


@pytest.mark.parametrize("case", CASES, ids=[f"C{c}_P{p}_B{len(d)}" for c, p, d in CASES])
def test_8b_layer_ragged_batches(l8b, case):
    C, P, ctx = case
    sess = l8b
    sess.ctx.kv_init(sess.k_pool.data_ptr(), sess.v_pool.data_ptr(), sess.num_blocks)
    mir = Mirror(sess, seed=3)
    pre = 500
    mir.create(pre)
    mir.install_context(pre, P)
    dec = list(range(600, 600 + len(ctx)))
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, L)
    b = api.Batch(C, pre, P, dec, ctx)
    x = synth.embeddings(b.rows, synth.LLAMA8B_LAYER.d_model, seed=1, stream=C * 7 + len(ctx))
    y, yr, sg, sr = mir.step(b, x)
    assert sg == sr
    stages = stage_errors(mir, b, x)
    kv_err = mir.kv_error(b)
    print(f"case {case}: kv {kv_err:.3e} stages {stages}")
    e = check(y, yr, f"case {case} (stages {stages})")
    print(f"case {case}: out {e}")
    assert kv_err <= TOL


def test_8b_repeated_iteration_is_idempotent(l8b):
    """Re-running the same batch rewrites the same slots and gives the same output."""
    sess = l8b
    sess.ctx.kv_init(sess.k_pool.data_ptr(), sess.v_pool.data_ptr(), sess.num_blocks)
    mir = Mirror(sess, seed=4)
    mir.create(1)
    mir.install_context(1, 40)
    mir.create(2)
    mir.install_context(2, 90)
    b = api.Batch(64, 1, 40, [2], [90])
    x = synth.embeddings(65, 4096, seed=1, stream=5)
    sess.run(b, x)
    y1 = sess.output(65)
    s1 = sess.ctx.last_slots()
    sess.run(b, x)
    y2 = sess.output(65)
    assert sess.ctx.last_slots() == s1
    np.testing.assert_array_equal(y1, y2)


def test_errors_are_reported_not_faulted(l8b):
    sess = l8b
    sess.ctx.kv_init(sess.k_pool.data_ptr(), sess.v_pool.data_ptr(), sess.num_blocks)
    sess.ctx.seq_create(1)
    with pytest.raises(api.SloweaveError) as e:       # prefix not cached
        sess.run(api.Batch(10, 1, 5, [], []))
    assert e.value.code == api.EINVAL
    with pytest.raises(api.SloweaveError) as e:       # unknown decode sequence
        sess.run(api.Batch(0, 0, 0, [77], [3]))
    assert e.value.code == api.EINVAL
    sess.ctx.seq_create(2)
    with pytest.raises(api.SloweaveError) as e:       # duplicate
        sess.run(api.Batch(4, 1, 0, [2, 2], [0, 0]))
    assert e.value.code == api.EINVAL
    with pytest.raises(api.SloweaveError) as e:       # workspace far too small: refused before any launch
        sess.ctx.mixed_iteration(api.Batch(30000, 1, 0, [], []), sess.x_in.data_ptr(),
                                 sess.x_out.data_ptr(), sess.ws.data_ptr(), sess.ws_bytes)
    assert e.value.code == api.ENOMEM
    with pytest.raises(ValueError):                   # more rows than the session's buffers hold
        sess.run(api.Batch(600, 1, 0, [], []))
    sess.ctx.seq_reserve(2, 16 * (sess.ctx.free_blocks() - 10))
    sess.ctx.seq_create(3)
    free = sess.ctx.free_blocks()
    with pytest.raises(api.SloweaveError) as e:       # pool exhaustion leaves state unchanged
        sess.ctx.seq_reserve(3, 16 * (free + 1))
    assert e.value.code == api.ENOMEM and sess.ctx.free_blocks() == free
    with pytest.raises(api.SloweaveError) as e:       # an iteration that cannot be covered
        sess.run(api.Batch(16 * (free + 1), 3, 0, [], []))
    assert e.value.code == api.ENOMEM and sess.ctx.free_blocks() == free


def test_tiny_batched_prefills():
    """Prefill batching (Sec. 3.3): three prompts' chunks (one fresh, two at a
    cached prefix) next to two decodes in one iteration, then two prompts
    again with one chunk spanning two query tiles; every row against the
    oracle, slots and block tables bit-exact."""
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    sess = Session(synth.TINY, num_blocks=512, max_c=400, max_b=4, qk_std=0.16)
    mir = Mirror(sess)
    for sid, L in ((1, 70), (2, 0), (3, 130), (21, 40), (22, 257)):
        mir.create(sid)
        mir.install_context(sid, L)
    steps = [
        api.Batch.batched([(1, 70, 100), (2, 0, 37), (3, 130, 64)], [21, 22], [40, 257]),
        api.Batch.batched([(2, 37, 300), (1, 170, 5)], [21, 22], [41, 258]),
    ]
    for i, b in enumerate(steps):
        x = synth.embeddings(b.rows, synth.TINY.d_model, seed=1, stream=500 + i)
        y, yr, sg, sr = mir.step(b, x)
        assert sg == sr
        e = check(y, yr, f"batched prefills, iteration {i}")
        assert mir.kv_error(b) <= TOL
        for sid in (1, 2, 3, 21, 22):
            assert sess.ctx.block_table(sid) == mir.mgr.block_table(sid)
        print(f"batched prefills iteration {i}: {e}", flush=True)


@pytest.mark.parametrize("pre", [
    ((500, 3000, 70), (501, 0, 130), (502, 500, 1)),   # a long prefix: its tiles' keys split and merged
    ((501, 0, 64), (502, 0, 63), (500, 16, 65), (503, 7, 33)),
], ids=["split_keys", "tile_edges"])
def test_8b_batched_prefills(l8b, pre):
    sess = l8b
    sess.ctx.kv_init(sess.k_pool.data_ptr(), sess.v_pool.data_ptr(), sess.num_blocks)
    mir = Mirror(sess, seed=6)
    for sid, p0, _ in pre:
        mir.create(sid)
        mir.install_context(sid, p0)
    dec, ctx = [600, 601], [5, 1000]
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, L)
    b = api.Batch.batched(pre, dec, ctx)
    x = synth.embeddings(b.rows, synth.LLAMA8B_LAYER.d_model, seed=1, stream=b.rows)
    y, yr, sg, sr = mir.step(b, x)
    assert sg == sr
    e = check(y, yr, f"8B batched prefills {pre}")
    kv = mir.kv_error(b)
    print(f"8B batched prefills {pre}: out {e} kv {kv:.3e}", flush=True)
    assert kv <= TOL

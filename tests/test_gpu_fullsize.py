"""Full-size parity on sampled outputs, in the launch configuration the benchmark times.

The oracle computes every row's K/V (later rows attend to them) but the
layer output only for sampled rows: the first and last chunk rows, rows at
query-tile and KV-block boundaries, random chunk rows, and decode rows of
the shortest and longest contexts.  Slots of every row and block tables of
every sequence must match the oracle's block manager bit-exactly; sampled
outputs and the K/V appended at sampled positions must meet the parity bar.

Workloads (8B-shaped layer: d 4096, 32/8 heads x 128, FFN 14336, bf16):
  * layer sweep extreme point: C = 2048 at prefix 8192 with B = 32 decodes,
    contexts uniform in [512, 2048];
  * long context: C = 4096 at prefix 28672, B = 8 decodes with contexts
    uniform in [16384, 32768];
  * chat/bursty: C = 32 at a seeded chunk boundary of a log-normal prompt,
    B = 256 decodes with log-normal contexts (median 700, sigma 0.8, cap 8192).
"""
import functools

import numpy as np
import pytest

from paper_2609_07883_amd import api, synth
from tests.parity import Mirror, check, rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _sample_rows(C, B, rng, extra=6):
    rows = {0, max(C - 1, 0), 63, 64, 255, 256}
    rows |= set(int(r) for r in rng.integers(0, max(C, 1), size=extra))
    rows = {r for r in rows if r < C}
    if B:
        rows |= {C, C + B - 1}
        rows |= set(int(C + r) for r in rng.integers(0, B, size=3))
    return sorted(rows)


def _run(C, P, ctx, seed):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_07883_amd.runtime import Session
    shape = synth.LLAMA8B_LAYER
    B = len(ctx)
    blocks = (P + C) // 16 + 2 + sum(L // 16 + 2 for L in ctx)
    sess = Session(shape, num_blocks=blocks, max_c=C, max_b=B)
    mir = Mirror(sess, seed=seed)
    pre = 7
    mir.create(pre)
    mir.install_context(pre, P)
    dec = list(range(1000, 1000 + B))
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, int(L))
    print(f"C={C} P={P} B={B}: contexts installed", flush=True)
    batch = api.Batch(C, pre, P, dec, [int(L) for L in ctx])
    x = synth.embeddings(batch.rows, shape.d_model, seed=1, stream=seed)
    rng = np.random.default_rng(seed)
    rows = _sample_rows(C, B, rng)
    y, yr, sg, sr = mir.step(batch, x, rows=rows)
    print(f"C={C} P={P} B={B}: iteration and oracle done", flush=True)
    assert sg == sr, "slot mapping differs"
    for sid in [pre] + dec:
        assert sess.ctx.block_table(sid) == mir.mgr.block_table(sid)
    e = check(y[rows], yr[rows], f"sampled rows {rows}")
    kv = mir.kv_error(batch, rows=rows)
    print(f"C={C} P={P} B={B}: rows {len(rows)} out {e} kv {kv:.3e}")
    assert kv <= 2e-2


def test_layer_sweep_extreme_point():
    ctx = synth.uniform_lengths(32, 512, 2048, seed=2)
    _run(2048, 8192, ctx, seed=11)


def test_layer_sweep_mid_point():
    ctx = synth.uniform_lengths(32, 512, 2048, seed=2)
    _run(1024, 2048, ctx, seed=12)


def test_long_context_point():
    ctx = synth.uniform_lengths(8, 16384, 32768, seed=2)
    _run(4096, 28672, ctx, seed=13)


def test_whole_query_tiles_point():
    """C = 2048 at prefix 16384, B = 8: query tiles of similar length, which
    the planner hands out whole (longest first to the least loaded
    work-group), so no tile is split and none is merged."""
    ctx = synth.uniform_lengths(8, 16384, 32768, seed=2)
    _run(2048, 16384, ctx, seed=18)


def test_chat_bursty_point():
    ctx = synth.lognormal_lengths(256, 700, 0.8, 8192, seed=2)
    prompt = int(synth.lognormal_lengths(1, 1024, 0.8, 8192, seed=4)[0])
    C = 32
    k = int(np.random.default_rng(5).integers(0, max(1, prompt // C)))
    _run(C, k * C, ctx, seed=14)


def test_decode_only_batch():
    """C = 0, B = 64: every GEMM runs the weight-streaming kernel on 64 rows."""
    ctx = synth.lognormal_lengths(64, 700, 0.8, 8192, seed=2)
    _run(0, 0, ctx, seed=15)


def test_small_chunk_with_decodes():
    """C = 32 at prefix 512 with B = 64 decodes (96 rows: two token waves)."""
    ctx = synth.lognormal_lengths(64, 700, 0.8, 8192, seed=3)
    _run(32, 512, ctx, seed=16)


def test_single_decode():
    """C = 0, B = 1: one row through every kernel."""
    _run(0, 0, [1500], seed=17)


@pytest.mark.parametrize("B", [5, 8, 9, 16, 24])
def test_small_decode_batches(B):
    """Decode-only batches at the narrow kernel's row limits: qkv, output and
    down projections on it up to 8 rows, the output projection up to 24
    (one 16-row token group up to 16 rows, two beyond; the last rows of a
    group padding at 5, 9 and 24)."""
    ctx = synth.lognormal_lengths(B, 700, 0.8, 8192, seed=20 + B)
    cfgs = [api.gemm_plan(B, n, k)["cfg"] for n, k in ((6144, 4096), (4096, 4096), (4096, 14336))]
    assert api.GEMM_NARROW in cfgs
    _run(0, 0, ctx, seed=30 + B)


@functools.lru_cache(maxsize=None)
def _plan_cover():
    """Row counts that together reach every GEMM variant (tile configuration,
    epilogue, plain / split-K / stream-K) the planner picks for the four
    projections of this layer between 33 and 4104 rows, chosen greedily from
    the plans the library reports."""
    shape = synth.LLAMA8B_LAYER
    d, F = shape.d_model, shape.ffn_dim
    qkv = (shape.n_q_heads + 2 * shape.n_kv_heads) * shape.head_dim
    proj = {"qkv": (qkv, d), "o": (d, shape.n_q_heads * shape.head_dim), "gateup": (2 * F, d), "down": (d, F)}

    def variants(m):
        out = set()
        for name, (n, k) in proj.items():
            p = api.gemm_plan(m, n, k)
            mode = "sk" if p["sk_workers"] else "split" if p["splits"] > 1 else "plain"
            out.add((name, p["cfg"], mode))
        return out

    cover = {m: variants(m) for m in range(33, 4105)}
    left = set().union(*cover.values())
    chosen = []
    while left:
        m = max(cover, key=lambda x: (len(cover[x] & left), -x))
        chosen.append(m)
        left -= cover[m]
    return sorted(chosen)


@pytest.mark.parametrize("part", range(4))
def test_gemm_plan_variants(part):
    """Prefill-only iterations (B = 0, P = 0) at row counts that reach every
    GEMM kernel variant of the planner (a quarter of them per case), sampled
    rows against the oracle."""
    ms = _plan_cover()[part::4]
    print(f"row counts {ms}", flush=True)
    for m in ms:
        _run(m, 0, [], seed=40 + m % 97)

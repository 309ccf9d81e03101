"""The C ABI on the CPU: exports, controller, cost table and block manager.

No GPU is touched: these entry points are host code.  The controller, the
table statistics and the block manager must agree bit-exactly with the
oracle twins (oracle/schedule.py, oracle/paging.py).
"""
import math
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import paging, schedule as S
from paper_2609_07883_amd import api, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "sloweave.h")) as f:
        declared = set(re.findall(r"^\s*(?:int|void|const char\*)\s+(slw_\w+)\s*\(", f.read(), re.M))
    L = api.lib()
    assert declared == set(api.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def _analytic_table(c_grid, b_grid):
    vals = [[S.analytic_cost_ns(b, c) for c in c_grid] for b in b_grid]
    return api.CostTable.from_samples(c_grid, b_grid, np.array(vals)[:, :, None]), \
        S.CostTable.from_values(c_grid, b_grid, vals)


def test_select_chunk_on_full_resolution_analytic_table_matches_worked_examples():
    c_grid = list(range(0, 4097))
    b_grid = [0, 1, 8, 32, 128, 256]
    tab, _ = _analytic_table(c_grid, b_grid)
    now = 10**9
    for n, budget, want in [(32, 25_000_000, 3598), (32, 10_000_000, 1098), (1, 25_000_000, 3882),
                            (8, 10_000_000, 1318), (128, 10_000_000, 218), (256, 10_000_000, 0)]:
        c, flags, lookups = api.select_chunk(tab, [now + budget] * n, now, 100_000, 4096)
        assert c == want
        assert lookups <= math.ceil(math.log2(4097)) + 1
        assert bool(flags & api.FLAG_DECODE_INFEASIBLE) == (want == 0)


@settings(max_examples=200, deadline=None)
@given(seed=st.integers(0, 2**31), n=st.integers(0, 300), budget=st.integers(-2_000_000, 40_000_000),
       c_max=st.integers(-5, 6000), rem=st.integers(-2, 7000), margin=st.integers(0, 3_000_000))
def test_select_chunk_bit_exact_vs_oracle(seed, n, budget, c_max, rem, margin):
    rng = np.random.default_rng(seed)
    nc, nb, reps = int(rng.integers(1, 8)), int(rng.integers(1, 6)), int(rng.integers(1, 5))
    c_grid = [0] + sorted(rng.choice(np.arange(1, 5000), size=nc - 1, replace=False).tolist())
    b_grid = sorted(rng.choice(np.arange(0, 300), size=nb, replace=False).tolist())
    samples = rng.integers(500_000, 30_000_000, size=(nb, nc, reps))
    ct = api.CostTable.from_samples(c_grid, b_grid, samples)
    ot = S.CostTable(c_grid, b_grid, samples.tolist())
    now = int(rng.integers(0, 10**12))
    deadlines = (now + budget + rng.integers(0, 5_000_000, size=n)).tolist()
    want_err = rem > 0 and n > 0 and n > b_grid[-1]
    if want_err:
        with pytest.raises(api.SloweaveError) as e:
            api.select_chunk(ct, deadlines, now, rem, c_max, margin)
        assert e.value.code == api.ERANGE
        with pytest.raises(IndexError):
            S.select_chunk_table(ot, deadlines, now, rem, c_max, margin)
        return
    got = api.select_chunk(ct, deadlines, now, rem, c_max, margin)
    want = S.select_chunk_table(ot, deadlines, now, rem, c_max, margin)
    # chunk and flags bit-exact; the library bisects Eq. 1 in its own probe
    # order, within the same logarithmic number of table lookups
    assert got[:2] == want[:2]
    cap = max(0, min(c_max, rem, c_grid[-1]))
    assert got[2] <= math.ceil(math.log2(cap + 1)) + 1


def test_cost_table_statistics_and_lookup_bit_exact():
    rng = np.random.default_rng(5)
    c_grid = [0, 32, 64, 128, 256, 512, 1024, 2048]
    b_grid = [0, 1, 4, 16, 64, 256]
    samples = rng.integers(1_000_000, 20_000_000, size=(len(b_grid), len(c_grid), 100))
    ct = api.CostTable.from_samples(c_grid, b_grid, samples)
    ot = S.CostTable(c_grid, b_grid, samples.tolist())
    assert (ct.values(api.TABLE_SAMPLES) == samples).all()
    assert ct.values(api.TABLE_P50).tolist() == ot.p50
    assert ct.values(api.TABLE_P99).tolist() == ot.p99
    assert ct.values(api.TABLE_THAT).tolist() == ot.t_hat
    for n in range(0, 257, 7):
        for c in list(range(0, 2049, 37)) + c_grid:
            assert ct.lookup(n, c) == ot.lookup(n, c)
    assert ct.monotone() == ot.monotone_violations()
    with pytest.raises(api.SloweaveError):
        ct.lookup(257, 0)
    with pytest.raises(api.SloweaveError):
        ct.lookup(0, 2049)


def test_cost_table_save_load_roundtrip(tmp_path):
    rng = np.random.default_rng(6)
    samples = rng.integers(0, 10**9, size=(3, 4, 7))
    ct = api.CostTable.from_samples([0, 5, 9, 100], [0, 2, 8], samples)
    p = str(tmp_path / "t.txt")
    ct.save(p)
    back = api.CostTable.load(p)
    for w in (api.TABLE_SAMPLES, api.TABLE_P50, api.TABLE_P99, api.TABLE_THAT):
        assert (back.values(w) == ct.values(w)).all()
    assert [g.tolist() for g in back.grids()] == [[0, 5, 9, 100], [0, 2, 8]]


@pytest.mark.parametrize("c_grid,b_grid", [([1, 2], [0]), ([0, 5, 5], [0]), ([0], [3, 1]), ([0], [-1])])
def test_cost_table_rejects_bad_grids(c_grid, b_grid):
    with pytest.raises(api.SloweaveError) as e:
        api.CostTable.from_samples(c_grid, b_grid, np.ones((len(b_grid), len(c_grid), 1)))
    assert e.value.code == api.EINVAL


def _host_ctx(num_blocks):
    ctx = api.Context.from_shape(synth.TINY)
    ctx.kv_init(0x10000, 0x20000, num_blocks)   # addresses are only stored, never touched here
    return ctx


@settings(max_examples=60, deadline=None)
@given(st.lists(st.tuples(st.sampled_from(["create", "reserve", "free"]), st.integers(0, 6),
                          st.integers(0, 200)), max_size=80))
def test_block_manager_bit_exact_vs_oracle(ops):
    ctx = _host_ctx(30)
    ref = paging.BlockManager(30, 16)
    live = set()
    for op, sid, n in ops:
        if op == "create":
            if sid in live:
                with pytest.raises(api.SloweaveError):
                    ctx.seq_create(sid)
                continue
            ctx.seq_create(sid)
            ref.create(sid)
            live.add(sid)
        elif op == "reserve" and sid in live:
            try:
                ref.reserve(sid, n)
                ctx.seq_reserve(sid, n)
            except paging.OutOfBlocks:
                with pytest.raises(api.SloweaveError) as e:
                    ctx.seq_reserve(sid, n)
                assert e.value.code == api.ENOMEM
        elif op == "free" and sid in live:
            ctx.seq_free(sid)
            ref.free(sid)
            live.discard(sid)
        for s in live:
            assert ctx.block_table(s) == ref.block_table(s)
        assert ctx.free_blocks() == ref.free_count()


def test_block_manager_hand_worked_scenario_through_abi():
    ctx = _host_ctx(8)
    ctx.seq_create(1)
    ctx.seq_create(2)
    ctx.seq_reserve(1, 20)
    ctx.seq_reserve(2, 16)
    ctx.seq_reserve(1, 33)
    ctx.seq_reserve(2, 17)
    assert ctx.block_table(1) == [0, 1, 3] and ctx.block_table(2) == [2, 4]
    ctx.seq_free(1)
    ctx.seq_create(3)
    ctx.seq_reserve(3, 40)
    assert ctx.block_table(3) == [0, 1, 3]
    with pytest.raises(api.SloweaveError) as e:
        ctx.seq_reserve(2, 100)
    assert e.value.code == api.ENOMEM and ctx.block_table(2) == [2, 4]


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, api.EUNSUPPORTED), ("n_kv_heads", 3, api.EINVAL), ("block_size", 32, api.EUNSUPPORTED),
    ("d_model", 200, api.EUNSUPPORTED), ("n_layers", 0, api.EINVAL)])
def test_create_rejects_unsupported_shapes(field, value, code):
    kw = dict(n_layers=1, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=704,
              rms_eps=1e-5, rope_theta=1e4, max_pos=4096, block_size=16)
    kw[field] = value
    with pytest.raises(api.SloweaveError) as e:
        api.Context(**kw)
    assert e.value.code == code


def test_workspace_size_grows_with_batch():
    ctx = api.Context.from_shape(synth.LLAMA8B_LAYER)
    a = ctx.workspace_size(64, 32)
    b = ctx.workspace_size(2048, 32)
    c = ctx.workspace_size(2048, 256)
    assert 0 < a < b < c
    off, nb = ctx.workspace_view(api.VIEW_ATTN, 100, 7)
    assert nb == 107 * 32 * 128 * 2 and off % 256 == 0


def _ctx_tables(seed=0):
    rng = np.random.default_rng(seed)
    c_grid, b_grid, p_grid = [0, 32, 64, 256, 1024], [0, 1, 4, 16], [0, 2048, 8192, 16384]
    samples = rng.integers(1_000_000, 60_000_000, size=(len(p_grid), len(b_grid), len(c_grid), 5))
    return (api.CostTable.from_samples(c_grid, b_grid, samples, p_grid=p_grid),
            S.CostTable(c_grid, b_grid, samples.tolist(), p_grid), c_grid, b_grid, p_grid)


def test_context_table_statistics_and_lookup_bit_exact(tmp_path):
    ct, ot, c_grid, b_grid, p_grid = _ctx_tables(1)
    assert ct.prefixes().tolist() == p_grid
    assert ct.values(api.TABLE_P99).tolist() == ot.p99
    assert ct.values(api.TABLE_THAT).tolist() == ot.t_hat
    assert ct.monotone() == ot.monotone_violations()
    rng = np.random.default_rng(2)
    for _ in range(400):
        n, c, p = int(rng.integers(0, 17)), int(rng.integers(0, 1025)), int(rng.integers(0, 16385))
        assert ct.lookup(n, c, p) == ot.lookup(n, c, p)
    with pytest.raises(api.SloweaveError) as e:
        ct.lookup(1, 32, 16385)
    assert e.value.code == api.ERANGE
    path = str(tmp_path / "ctx.txt")
    ct.save(path)
    back = api.CostTable.load(path)
    assert back.prefixes().tolist() == p_grid
    assert back.values(api.TABLE_SAMPLES).tolist() == ct.values(api.TABLE_SAMPLES).tolist()
    flat = api.CostTable.from_samples(c_grid, b_grid, np.ones((4, 5), np.int64))
    assert flat.prefixes() is None


def test_select_chunk_ctx_bit_exact_vs_oracle():
    ct, ot, *_ = _ctx_tables(3)
    rng = np.random.default_rng(4)
    for _ in range(500):
        n = int(rng.integers(0, 17))
        now = int(rng.integers(0, 10**9))
        dl = (now + rng.integers(0, 80_000_000, size=n)).tolist()
        rem, cmax, margin = int(rng.integers(-1, 1500)), int(rng.integers(0, 1500)), int(rng.integers(0, 10**6))
        prefix = int(rng.integers(0, 16385))
        assert api.select_chunk(ct, dl, now, rem, cmax, margin, prefix=prefix)[:2] == \
            S.select_chunk_table(ot, dl, now, rem, cmax, margin, prefix=prefix)[:2]


def test_cost_table_statistics_match_hand_worked_golden():
    """The library's P50, P99, running max and monotonicity report on the
    hand-worked table of tests/golden/monotone_table.txt."""
    from tests.test_oracle_schedule import _golden_monotone
    g, samples = _golden_monotone()
    ct = api.CostTable.from_samples(g["c_grid"], g["b_grid"], np.asarray(samples, dtype=np.int64))
    assert ct.values(api.TABLE_P50).tolist() == [g["p50"][b] for b in g["b_grid"]]
    assert ct.values(api.TABLE_P99).tolist() == [g["p99"][b] for b in g["b_grid"]]
    assert ct.values(api.TABLE_THAT).tolist() == [g["that"][b] for b in g["b_grid"]]
    assert ct.monotone() == g["violations"]
    ct2 = api.CostTable.from_samples(g["c_grid"], g["b_grid"], np.asarray([samples, samples], dtype=np.int64),
                                     p_grid=[0, 4096])
    assert ct2.monotone() == (2 * g["violations"][0], g["violations"][1])


def test_batched_prefill_validation_through_abi():
    """Several prefills in one iteration: malformed batches are refused on the
    host before anything is reserved (no device pointer is ever touched, so
    placeholder addresses serve)."""
    ctx = api.Context.from_shape(synth.TINY)
    fake = 1 << 20
    ctx.set_layer_weights(0, *([fake] * 6))
    ctx.kv_init(fake, fake, 64)
    for sid in (1, 2, 3):
        ctx.seq_create(sid)
    ctx.seq_reserve(1, 20)
    free = ctx.free_blocks()

    def run(batch):
        ctx.mixed_iteration(batch, fake, fake, fake, 1 << 30)

    cases = [
        (api.Batch(30, -1, 0, [], [], ((1, 20, 10), (1, 30, 20))), api.EINVAL),       # sequence twice
        (api.Batch(30, -1, 0, [2], [0], ((1, 20, 10), (2, 0, 20))), api.EINVAL),      # prefill and decode
        (api.Batch(31, -1, 0, [], [], ((1, 20, 10), (2, 0, 20))), api.EINVAL),       # rows do not add up
        (api.Batch(10, -1, 0, [], [], ((1, 20, 10), (2, 0, 0))), api.EINVAL),        # empty chunk
        (api.Batch(30, -1, 0, [], [], ((1, 21, 10), (2, 0, 20))), api.EINVAL),       # prefix not cached
        (api.Batch(17, -1, 0, [], [], tuple((100 + i, 0, 1) for i in range(17))), api.ERANGE),  # > 16
    ]
    for b, code in cases:
        with pytest.raises(api.SloweaveError) as e:
            run(b)
        assert e.value.code == code, (b, e.value)
        assert ctx.free_blocks() == free
    assert api.Batch.batched([(1, 20, 5)]) == api.Batch(5, 1, 20, [], [])
    assert api.Batch.batched([(1, 20, 5), (2, 0, 3)]).chunk == 8


@pytest.mark.parametrize("shape", ["8b", "tiny"])
def test_gemm_plan_is_valid_for_every_row_count(shape):
    """The planner's choice for every row count is a launchable plan: tile
    widths divide n, the k split divides k into whole 64-deep steps, stream-K
    only with whole tiles counted in rounds of 8 XCDs, the weight-streaming
    kernel only up to 32 rows, the narrow kernel only up to 24 with k split
    into whole 32-wide slices over at most eight waves."""
    sh = synth.LLAMA8B_LAYER if shape == "8b" else synth.TINY
    d, F = sh.d_model, sh.ffn_dim
    qkv = (sh.n_q_heads + 2 * sh.n_kv_heads) * sh.head_dim
    seen = set()
    for n, k in [(qkv, d), (d, sh.n_q_heads * sh.head_dim), (2 * F, d), (d, F)]:
        if n % 128:
            continue
        for m in list(range(1, 600)) + list(range(600, 9000, 37)):
            p = api.gemm_plan(m, n, k)
            if p["cfg"] == api.GEMM_SKINNY:
                assert m <= 32
                continue
            if p["cfg"] == api.GEMM_NARROW:
                assert m <= 24 and n % 64 == 0 and k % 32 == 0 and p["bn"] == 16 and p["splits"] == 1
                seen.add(p["cfg"])
                continue
            assert n % p["bn"] == 0 and p["bm"] % 32 == 0
            assert p["splits"] in (1, 2, 4, 8) and k % (64 * p["splits"]) == 0
            if p["sk_workers"]:
                assert p["splits"] == 1 and p["dp_tiles"] % 8 == 0 and 0 < p["sk_workers"] <= 512
            seen.add(p["cfg"])
    assert len(seen) >= 2
    with pytest.raises(api.SloweaveError):
        api.gemm_plan(0, 4096, 4096)
    with pytest.raises(api.SloweaveError):
        api.gemm_plan(64, 4000, 4096)


def _share(total, slots, quantum):
    return -(-(-(-total // slots)) // quantum) * quantum


@settings(max_examples=300, deadline=None)
@given(ctx=st.lists(st.integers(0, 32766), max_size=300),
       pre=st.lists(st.tuples(st.integers(0, 28000), st.integers(1, 4096)), max_size=4),
       shape=st.sampled_from(["8b", "tiny"]))
def test_attention_plans_cover_every_key_once_and_balance(ctx, pre, shape):
    """The executor's attention work lists (the same code, run on the host):
    every decode's keys and every query tile's keys are covered exactly once
    (the call fails otherwise), the decode runs are equal shares of the
    padded keys, the chunk work-groups take equal runs of 64-key tiles or,
    when whole tiles balance, at most 1.1 equal shares each."""
    sh = synth.LLAMA8B_LAYER if shape == "8b" else synth.TINY
    ctx = [min(c, sh.max_pos - 1) for c in ctx]
    pre = [(min(p, sh.max_pos - c), c) for p, c in pre if c <= sh.max_pos]
    p = api.attention_plan(sh, ctx, pre)
    B = len(ctx)
    slots_cap = max(1, 2048 // sh.n_kv_heads)
    if B:
        padded = sum(-(-(c + 1) // 64) * 64 for c in ctx)
        want = min(slots_cap, max(1, padded // 128))
        assert 1 <= p["decode_slots"] <= slots_cap
        assert B <= p["decode_items"] <= p["decode_slots"] + B
        assert p["decode_max_keys"] <= _share(padded, want, 64)
    else:
        assert p["decode_items"] == p["decode_slots"] == 0
    group = sh.n_q_heads // sh.n_kv_heads
    pwg = 256 // group
    tiles = [-(-(pp + min(pwg, cc - j) + j) // 64) for pp, cc in pre for j in range(0, cc, pwg)]
    assert p["query_tiles"] == len(tiles) and p["chunk_tiles"] == sum(tiles)
    if tiles:
        total = sum(tiles)
        want = min(max(1, 256 // sh.n_kv_heads), max(1, total // 4))
        share = -(-total // want)
        assert p["chunk_items"] >= len(tiles)
        if p["chunk_whole"]:
            assert p["chunk_items"] == len(tiles) and len(tiles) >= want
            assert p["chunk_max_tiles"] * 10 <= share * 11
        else:
            assert p["chunk_max_tiles"] <= share


def test_attention_plan_examples():
    """Long prompts take whole query tiles (nothing to merge); the start of a
    prompt, whose tiles grow with their position, is cut into runs; one
    short decode is one item."""
    sh = synth.LLAMA8B_LAYER
    long = api.attention_plan(sh, [20000] * 8, [(28672, 4096)])
    assert long["chunk_whole"] == 1 and long["chunk_items"] == long["query_tiles"] == 64
    assert long["chunk_max_tiles"] == long["chunk_min_tiles"] == 961   # 64 tiles of 449..512 paired to 961
    first = api.attention_plan(sh, [], [(0, 2048)])
    assert first["chunk_whole"] == 0 and first["chunk_tiles"] == 528 and first["chunk_max_tiles"] == 17
    one = api.attention_plan(sh, [0], [])
    assert (one["decode_items"], one["decode_slots"], one["decode_max_keys"]) == (1, 1, 1)
    with pytest.raises(api.SloweaveError):
        api.attention_plan(sh, [sh.max_pos], [])
    with pytest.raises(api.SloweaveError):
        api.attention_plan(sh, [], [(0, 1)] * 17)

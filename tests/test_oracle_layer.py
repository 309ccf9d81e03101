"""Pins for the layer oracle (CPU only).

The oracle is checked against things other than itself:
  * transformers' LlamaDecoderLayer (an independent library implementation
    of the pre-norm RMSNorm / rotate-half RoPE / GQA / SwiGLU block), run in
    float64 over the whole causal sequence;
  * torch's scaled_dot_product_attention for the chunk-vs-prefix mask;
  * the complex-exponential form of RoPE and torch's rms_norm / silu;
  * the invariants that define chunked prefill on a paged cache: any chunk
    split gives the same K/V and outputs, decode equals the last row of the
    full sequence, and rows of a mixed batch do not interact.
"""
import numpy as np
import pytest
import torch

from oracle import layer as L
from paper_2609_07883_amd import synth
from tests.oracle_fixtures import TINY_GQA, oracle_shape, oracle_weights, x_rows


def _hf_layer(s: synth.ModelShape, w: L.LayerWeights):
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer, LlamaRotaryEmbedding
    cfg = LlamaConfig(hidden_size=s.d_model, intermediate_size=s.ffn_dim,
                      num_attention_heads=s.n_q_heads, num_key_value_heads=s.n_kv_heads,
                      head_dim=s.head_dim, rope_theta=s.rope_theta, rms_norm_eps=s.rms_eps,
                      max_position_embeddings=s.max_pos, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "sdpa"
    lay = LlamaDecoderLayer(cfg, 0).double().eval()
    hq, hkv, hd, f = s.n_q_heads, s.n_kv_heads, s.head_dim, s.ffn_dim
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        lay.self_attn.q_proj.weight.copy_(t(w.wqkv[: hq * hd]))
        lay.self_attn.k_proj.weight.copy_(t(w.wqkv[hq * hd: (hq + hkv) * hd]))
        lay.self_attn.v_proj.weight.copy_(t(w.wqkv[(hq + hkv) * hd:]))
        lay.self_attn.o_proj.weight.copy_(t(w.wo))
        lay.mlp.gate_proj.weight.copy_(t(w.wgu[:f]))
        lay.mlp.up_proj.weight.copy_(t(w.wgu[f:]))
        lay.mlp.down_proj.weight.copy_(t(w.wd))
        lay.input_layernorm.weight.copy_(t(w.g1))
        lay.post_attention_layernorm.weight.copy_(t(w.g2))
    rot = LlamaRotaryEmbedding(cfg).double()
    return lay, rot


def _hf_forward(lay, rot, x: np.ndarray) -> np.ndarray:
    n = x.shape[0]
    hs = torch.from_numpy(x)[None]
    pos = torch.arange(n)[None]
    cos, sin = rot(hs, pos)
    mask = torch.full((n, n), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    with torch.no_grad():
        out = lay(hs, attention_mask=mask, position_ids=pos, position_embeddings=(cos, sin))
    if isinstance(out, tuple):
        out = out[0]
    return out[0].numpy()


def _prefill(shape, w, x, chunks, seq=7):
    kv = L.KVState()
    ys = []
    p = 0
    for c in chunks:
        b = L.MixedBatch(chunk=c, prefill_seq=seq, prefix_len=p, decode_seqs=[], context_lens=[])
        ys.append(L.mixed_iteration(shape, w, x[p:p + c], kv, b))
        p += c
    return np.concatenate(ys), kv


@pytest.mark.parametrize("model,qk_std", [(synth.TINY, None), (synth.TINY, 0.16), (TINY_GQA, None)])
def test_layer_matches_transformers_llama(model, qk_std):
    bits = synth.layer_weights(model, weight_seed=0, qk_std=qk_std)
    w = oracle_weights(bits)
    shape = oracle_shape(model)
    n = 200
    x = x_rows(n, model.d_model)
    lay, rot = _hf_layer(model, w)
    ref = _hf_forward(lay, rot, x)
    y, _ = _prefill(shape, w, x, [64, 100, 36])
    # transformers derives its RoPE inverse frequencies in float32 (about 1e-7
    # relative); any structural mistake shows up at O(1)
    assert np.max(np.abs(y - ref)) <= 1e-6 * np.max(np.abs(ref))


def test_decode_equals_last_row_of_transformers_forward():
    model = TINY_GQA
    w = oracle_weights(synth.layer_weights(model, weight_seed=3, qk_std=0.16))
    shape = oracle_shape(model)
    n = 97
    x = x_rows(n + 1, model.d_model, stream=5)
    lay, rot = _hf_layer(model, w)
    ref = _hf_forward(lay, rot, x)
    _, kv = _prefill(shape, w, x[:n], [n], seq=11)
    b = L.MixedBatch(chunk=0, prefill_seq=-1, prefix_len=0, decode_seqs=[11], context_lens=[n])
    y = L.mixed_iteration(shape, w, x[n:], kv, b)
    np.testing.assert_allclose(y[0], ref[n], rtol=0, atol=1e-6 * np.max(np.abs(ref)))


def test_chunk_attention_matches_sdpa_bottom_right_mask():
    """Queries at P..P+C-1 over keys 0..P+C-1 under the causal mask (torch SDPA in fp64)."""
    model = TINY_GQA
    w = oracle_weights(synth.layer_weights(model, weight_seed=4, qk_std=0.16))
    shape = oracle_shape(model)
    P, C = 150, 37
    x = x_rows(P + C, model.d_model, stream=2)
    _, kv = _prefill(shape, w, x[:P], [P], seq=1)
    b = L.MixedBatch(chunk=C, prefill_seq=1, prefix_len=P, decode_seqs=[], context_lens=[])
    o = L.attention_outputs(shape, w, x[P:], kv, b)            # [C][Hq][hd]
    q, _, _ = L.qkv_rope(shape, w, x[P:], np.arange(P, P + C))
    k = torch.from_numpy(kv.seqs[1].k).permute(1, 0, 2)        # [Hkv][n][hd]
    v = torch.from_numpy(kv.seqs[1].v).permute(1, 0, 2)
    rep = model.n_q_heads // model.n_kv_heads
    k = k.repeat_interleave(rep, 0)
    v = v.repeat_interleave(rep, 0)
    qq = torch.from_numpy(q).permute(1, 0, 2)
    qpos = torch.arange(P, P + C)[:, None]
    kpos = torch.arange(P + C)[None, :]
    mask = kpos <= qpos
    ref = torch.nn.functional.scaled_dot_product_attention(qq, k, v, attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)


def test_rope_equals_complex_rotation():
    rng = np.random.default_rng(0)
    hd = 64
    x = rng.standard_normal((5, 3, hd))
    pos = np.array([0, 1, 17, 1000, 32767])
    got = L.apply_rope(x, pos, 10000.0)
    z = x[..., : hd // 2] + 1j * x[..., hd // 2:]
    ang = pos[:, None] * 10000.0 ** (-np.arange(hd // 2) * 2.0 / hd)
    zr = z * np.exp(1j * ang)[:, None, :]
    np.testing.assert_allclose(got[..., : hd // 2], zr.real, atol=1e-12)
    np.testing.assert_allclose(got[..., hd // 2:], zr.imag, atol=1e-12)
    np.testing.assert_array_equal(got[0], x[0])                 # position 0 is the identity


def test_rms_norm_and_silu_match_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 48))
    g = rng.standard_normal(48)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), eps=1e-5)
    np.testing.assert_allclose(L.rms_norm(x, g, 1e-5), ref.numpy(), atol=1e-13)
    np.testing.assert_allclose(L.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               atol=1e-14)


@pytest.mark.parametrize("splits", [[512], [128] * 4, [1, 511], [16] * 32, "random"])
def test_chunk_split_invariance(splits):
    model = synth.TINY
    w = oracle_weights(synth.layer_weights(model, weight_seed=0, qk_std=0.16))
    shape = oracle_shape(model)
    x = x_rows(512, model.d_model)
    if splits == "random":
        rng = np.random.default_rng(9)
        cuts = np.sort(rng.choice(np.arange(1, 512), size=9, replace=False))
        splits = list(np.diff(np.concatenate([[0], cuts, [512]])))
    ref, kv_ref = _prefill(shape, w, x, [512])
    y, kv = _prefill(shape, w, x, splits)
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(kv.seqs[7].k, kv_ref.seqs[7].k, rtol=0, atol=1e-13)
    np.testing.assert_allclose(kv.seqs[7].v, kv_ref.seqs[7].v, rtol=0, atol=1e-13)


def test_mixed_batch_rows_do_not_interact():
    model = TINY_GQA
    w = oracle_weights(synth.layer_weights(model, weight_seed=2, qk_std=0.16))
    shape = oracle_shape(model)
    kv = L.KVState()
    ctx = [1, 16, 33, 70]
    for i, n in enumerate(ctx):
        _prefill_into(shape, w, kv, 100 + i, x_rows(n, model.d_model, stream=10 + i))
    _prefill_into(shape, w, kv, 5, x_rows(40, model.d_model, stream=20))
    xc = x_rows(23, model.d_model, stream=30)
    xd = x_rows(len(ctx), model.d_model, stream=31)
    kv_sep = kv.copy()
    batch = L.MixedBatch(chunk=23, prefill_seq=5, prefix_len=40,
                         decode_seqs=[100, 101, 102, 103], context_lens=ctx)
    y = L.mixed_iteration(shape, w, np.concatenate([xc, xd]), kv, batch)
    y_c = L.mixed_iteration(shape, w, xc, kv_sep,
                            L.MixedBatch(23, 5, 40, [], []))
    parts = [y_c]
    for i, n in enumerate(ctx):
        parts.append(L.mixed_iteration(shape, w, xd[i:i + 1], kv_sep,
                                       L.MixedBatch(0, -1, 0, [100 + i], [n])))
    np.testing.assert_allclose(y, np.concatenate(parts), rtol=0, atol=1e-12)
    for s in kv.seqs:
        np.testing.assert_allclose(kv.seqs[s].k, kv_sep.seqs[s].k, rtol=0, atol=1e-13)


def _prefill_into(shape, w, kv, seq, x):
    b = L.MixedBatch(chunk=x.shape[0], prefill_seq=seq, prefix_len=0, decode_seqs=[], context_lens=[])
    L.mixed_iteration(shape, w, x, kv, b)


def test_sampled_rows_equal_full_rows():
    model = TINY_GQA
    w = oracle_weights(synth.layer_weights(model, weight_seed=2))
    shape = oracle_shape(model)
    x = x_rows(50, model.d_model)
    kv1, kv2 = L.KVState(), L.KVState()
    b = L.MixedBatch(50, 1, 0, [], [])
    full = L.mixed_iteration(shape, w, x, kv1, b)
    part = L.mixed_iteration(shape, w, x, kv2, b, rows=[0, 13, 49])
    np.testing.assert_allclose(part[[0, 13, 49]], full[[0, 13, 49]], rtol=0, atol=1e-12)
    assert np.isnan(part[1]).all()


def test_rejects_inconsistent_context():
    model = synth.TINY
    w = oracle_weights(synth.layer_weights(model))
    shape = oracle_shape(model)
    kv = L.KVState()
    _prefill_into(shape, w, kv, 1, x_rows(10, model.d_model))
    with pytest.raises(ValueError):
        L.mixed_iteration(shape, w, x_rows(1, model.d_model), kv, L.MixedBatch(0, -1, 0, [1], [9]))


def test_append_kv_equals_row_by_row_writes():
    """Step 4 writes row r's K/V at position pos[r] of its sequence, in row
    order: a row at the current length extends the sequence, one inside it
    overwrites, one beyond it is an error.  The append (one copy per
    sequence) must leave exactly what a row-by-row write does."""
    from oracle.layer import LayerShape
    rng = np.random.default_rng(5)
    hkv, hd = 2, 4
    shape = LayerShape(d_model=8, n_q_heads=2, n_kv_heads=hkv, head_dim=hd, ffn_dim=8, rms_eps=1e-5,
                       rope_theta=10000.0)
    for trial in range(40):
        init = {s: int(rng.integers(0, 5)) for s in range(3)}
        kv = L.KVState({s: L.SeqCache(rng.standard_normal((n, hkv, hd)), rng.standard_normal((n, hkv, hd)))
                        for s, n in init.items()})
        ref = {s: [c.k[i].copy() for i in range(c.length)] for s, c in kv.seqs.items()}
        refv = {s: [c.v[i].copy() for i in range(c.length)] for s, c in kv.seqs.items()}
        seqs, pos = [], []
        length = dict(init)
        for _ in range(int(rng.integers(1, 12))):
            s = int(rng.integers(0, 3))
            p = int(rng.integers(0, length[s] + 1))   # inside or at the end: always valid
            seqs.append(s)
            pos.append(p)
            length[s] = max(length[s], p + 1)
        k = rng.standard_normal((len(seqs), hkv, hd))
        v = rng.standard_normal((len(seqs), hkv, hd))
        for r, (s, p) in enumerate(zip(seqs, pos)):       # row-by-row reference
            if p == len(ref[s]):
                ref[s].append(k[r].copy())
                refv[s].append(v[r].copy())
            else:
                ref[s][p] = k[r].copy()
                refv[s][p] = v[r].copy()
        L.append_kv(shape, kv, seqs, pos, k, v)
        for s in range(3):
            assert kv.seqs[s].length == len(ref[s])
            if ref[s]:
                np.testing.assert_array_equal(kv.seqs[s].k, np.stack(ref[s]))
                np.testing.assert_array_equal(kv.seqs[s].v, np.stack(refv[s]))
    # a row beyond the current length (counting earlier rows) is refused
    kv = L.KVState({0: L.SeqCache(np.zeros((2, hkv, hd)), np.zeros((2, hkv, hd)))})
    with pytest.raises(ValueError):
        L.append_kv(shape, kv, [0, 0], [2, 4], np.zeros((2, hkv, hd)), np.zeros((2, hkv, hd)))


def _hf_kv(lay, rot, x: np.ndarray):
    """K (after RoPE) and V that transformers' attention module forms from a
    layer's input rows x [n][d] at positions 0..n-1: [n][Hkv][hd] each."""
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    n = x.shape[0]
    at = lay.self_attn
    hs = torch.from_numpy(x)[None]
    pos = torch.arange(n)[None]
    cos, sin = rot(hs, pos)
    with torch.no_grad():
        u = lay.input_layernorm(hs)
        hd = at.head_dim
        q = at.q_proj(u).view(1, n, -1, hd).transpose(1, 2)
        k = at.k_proj(u).view(1, n, -1, hd).transpose(1, 2)
        v = at.v_proj(u).view(1, n, -1, hd).transpose(1, 2)
        _, k = apply_rotary_pos_emb(q, k, cos, sin)
    return k[0].transpose(0, 1).numpy(), v[0].transpose(0, 1).numpy()


def test_stack_matches_stacked_transformers_layers():
    """stack_iteration over three layers with their own weights and caches:
    a prompt prefilled in two chunks, then one decode token, against three
    transformers LlamaDecoderLayers applied in turn to the whole sequence.
    Every layer's K/V is compared with the K/V transformers forms from that
    layer's input, so a wrong hand-off between layers or a cache shared
    between layers shows up."""
    model = TINY_GQA
    n_layers, n = 3, 90
    bits = [synth.layer_weights(model, layer=l, weight_seed=6, qk_std=0.16) for l in range(n_layers)]
    ws = [oracle_weights(b) for b in bits]
    shape = oracle_shape(model)
    x = x_rows(n + 1, model.d_model, stream=8)
    # transformers: the whole sequence through each layer in turn
    hf_in, hf_kv = [], []
    h = x
    for w in ws:
        lay, rot = _hf_layer(model, w)
        hf_in.append(h)
        hf_kv.append(_hf_kv(lay, rot, h))
        h = _hf_forward(lay, rot, h)
    ref = h
    # oracle: chunks of 40 and 50, then the decode of position 90
    kvs = [L.KVState() for _ in ws]
    ys = []
    for p, c in ((0, 40), (40, 50)):
        b = L.MixedBatch(chunk=c, prefill_seq=3, prefix_len=p, decode_seqs=[], context_lens=[])
        ys.append(L.stack_iteration(shape, ws, x[p:p + c], kvs, b))
    b = L.MixedBatch(chunk=0, prefill_seq=-1, prefix_len=0, decode_seqs=[3], context_lens=[n])
    ys.append(L.stack_iteration(shape, ws, x[n:], kvs, b))
    y = np.concatenate(ys)
    scale = np.max(np.abs(ref))
    assert np.max(np.abs(y - ref)) <= 1e-6 * scale
    for l in range(n_layers):
        k_ref, v_ref = hf_kv[l]
        c = kvs[l].seqs[3]
        assert c.length == n + 1
        # K carries transformers' float32 RoPE frequencies directly (about
        # 1e-6 relative at these positions); a structural mistake is O(1)
        assert np.max(np.abs(c.k - k_ref)) <= 1e-5 * np.max(np.abs(k_ref))
        assert np.max(np.abs(c.v - v_ref)) <= 1e-6 * np.max(np.abs(v_ref))
    # the layers differ: a stack that reused one layer's weights would not match
    assert np.max(np.abs(hf_kv[0][0] - hf_kv[1][0])) > 0.1 * np.max(np.abs(hf_kv[0][0]))


def test_prefill_batching_equals_each_prompt_alone():
    """Several prompts' chunks in one iteration (Sec. 3.3 prefill batching)
    give every row the output and K/V it gets when its prompt runs alone:
    rows of different sequences do not interact."""
    model = TINY_GQA
    w = oracle_weights(synth.layer_weights(model, weight_seed=7, qk_std=0.16))
    shape = oracle_shape(model)
    base = L.KVState()
    # sequence 1 holds 30 tokens, 3 holds 17, decode 9 holds 40; sequence 2 is new
    for sid, n, st in ((1, 30, 21), (3, 17, 22), (9, 40, 23)):
        b = L.MixedBatch(chunk=n, prefill_seq=sid, prefix_len=0, decode_seqs=[], context_lens=[])
        L.mixed_iteration(shape, w, x_rows(n, model.d_model, stream=st), base, b)
    pre = [(1, 30, 25), (2, 0, 40), (3, 17, 9)]
    x = x_rows(75, model.d_model, stream=24)
    xd = x_rows(1, model.d_model, stream=25)
    kv = base.copy()
    batch = L.MixedBatch(chunk=74, prefill_seq=-1, prefix_len=0, decode_seqs=[9], context_lens=[40], prefills=pre)
    y = L.mixed_iteration(shape, w, np.concatenate([x[:74], xd]), kv, batch)
    r0 = 0
    scale = np.max(np.abs(y))
    for sid, p0, c in pre:
        alone = base.copy()
        b = L.MixedBatch(chunk=c, prefill_seq=sid, prefix_len=p0, decode_seqs=[], context_lens=[])
        ya = L.mixed_iteration(shape, w, x[r0:r0 + c], alone, b)
        np.testing.assert_allclose(y[r0:r0 + c], ya, rtol=0, atol=1e-12 * scale)
        np.testing.assert_allclose(kv.seqs[sid].k, alone.seqs[sid].k, rtol=0, atol=1e-12)
        np.testing.assert_allclose(kv.seqs[sid].v, alone.seqs[sid].v, rtol=0, atol=1e-12)
        r0 += c
    alone = base.copy()
    yd = L.mixed_iteration(shape, w, xd, alone, L.MixedBatch(0, -1, 0, [9], [40]))
    np.testing.assert_allclose(y[74:], yd, rtol=0, atol=1e-12 * scale)
    with pytest.raises(ValueError):      # a sequence listed twice
        L.mixed_iteration(shape, w, x[:20], base.copy(),
                          L.MixedBatch(20, -1, 0, [], [], prefills=[(1, 30, 10), (1, 40, 10)]))

"""GPU parity of multi-layer iterations against the oracle's stacked layers.

A stack of n layers passes each layer's bf16 output rows to the next layer,
keeps one KV pool region per layer and one set of weights per layer.  Every
output row of the last layer and the K/V that every layer appended are
compared with the oracle (each layer of the oracle reads the previous one's
float64 output and its own dense cache); slots and block tables must match
the oracle's block manager bit-exactly.

Shapes:
  * Tiny stack, 3 layers (d 256, 4 MHA heads of 64, FFN 704, sharp q/k
    weights so attention is far from uniform): decode contexts built by
    prefill iterations through all three layers, then a 512-token prompt in
    four chunks of 128 next to the four decodes, element-wise on every row;
  * 8B-shaped stack, 2 layers (d 4096, 32/8 heads of 128, FFN 14336) at
    small ragged batches: chunk rows at a non-zero prefix with decodes whose
    contexts cross block boundaries, a decode-only batch and a prefill-only
    batch, all rows compared.
"""
import numpy as np
import pytest

from paper_2609_07883_amd import api, synth
from tests.parity import TOL, Mirror, check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _kv_all_layers(mir, batch):
    return max(mir.kv_error(batch, layer=l) for l in range(len(mir.w)))


def test_tiny_three_layer_stack():
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    shape = synth.with_layers(synth.TINY, 3)
    sess = Session(shape, num_blocks=256, max_c=256, max_b=4, qk_std=0.16)
    mir = Mirror(sess)
    ctx_lens = synth.uniform_lengths(4, 64, 256, seed=2).tolist()
    dec = [11, 12, 13, 14]
    for sid, L in zip(dec, ctx_lens):
        mir.create(sid)
        b = api.Batch(L, sid, 0, [], [])
        x = synth.embeddings(L, shape.d_model, seed=1, stream=300 + sid)
        y, yr, sg, sr = mir.step(b, x)
        assert sg == sr
        check(y, yr, f"3-layer context prefill of seq {sid}", layers=3)
        assert _kv_all_layers(mir, b) <= TOL
    prompt = 99
    mir.create(prompt)
    xp = synth.embeddings(512, shape.d_model, seed=1, stream=31)
    lens = list(ctx_lens)
    for it in range(4):
        xd = synth.embeddings(4, shape.d_model, seed=1, stream=400 + it)
        b = api.Batch(128, prompt, 128 * it, dec, lens)
        y, yr, sg, sr = mir.step(b, np.concatenate([xp[128 * it: 128 * (it + 1)], xd]))
        assert sg == sr, f"slots differ at iteration {it}"
        e = check(y, yr, f"3-layer iteration {it}", layers=3)
        kv = _kv_all_layers(mir, b)
        print(f"3-layer iteration {it}: out {e} kv {kv:.3e}", flush=True)
        assert kv <= TOL
        for sid in dec + [prompt]:
            assert sess.ctx.block_table(sid) == mir.mgr.block_table(sid)
        lens = [L + 1 for L in lens]


@pytest.fixture(scope="module")
def stack8b():
    _require_gpu()
    from paper_2609_07883_amd.runtime import Session
    return Session(synth.with_layers(synth.LLAMA8B_LAYER, 2), num_blocks=512, max_c=160, max_b=6)


STACK_CASES = [
    # (C, P, decode contexts)
    (37, 50, [1, 16, 33, 300]),
    (0, 0, [0, 15, 17, 130, 999, 64]),
    (150, 0, []),
    (1, 31, [2]),
]


@pytest.mark.parametrize("case", STACK_CASES, ids=[f"C{c}_P{p}_B{len(d)}" for c, p, d in STACK_CASES])
def test_8b_two_layer_stack(stack8b, case):
    C, P, ctx = case
    sess = stack8b
    sess.ctx.kv_init(sess.k_pool.data_ptr(), sess.v_pool.data_ptr(), sess.num_blocks)
    mir = Mirror(sess, seed=5)
    pre = 70
    mir.create(pre)
    mir.install_context(pre, P)
    dec = list(range(700, 700 + len(ctx)))
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, L)
    b = api.Batch(C, pre, P, dec, ctx)
    x = synth.embeddings(b.rows, sess.shape.d_model, seed=1, stream=11 * C + len(ctx))
    y, yr, sg, sr = mir.step(b, x)
    assert sg == sr
    for sid in dec + ([pre] if C else []):
        assert sess.ctx.block_table(sid) == mir.mgr.block_table(sid)
    e = check(y, yr, f"2-layer case {case}", layers=2)
    kv = [mir.kv_error(b, layer=l) for l in range(2)]
    print(f"2-layer case {case}: out {e} kv per layer {kv}", flush=True)
    assert max(kv) <= TOL

"""The allocation-free entry point against the ordinary one (GPU, through the C ABI).

slw_mixed_iteration_static runs the same iteration on the library's static
workspace array instead of a caller workspace.  Two sessions with the same
weights and the same pre-existing K/V run the same calls, one through each
entry point: two iterations in a row, the second with fewer rows than the
first, so the second call reuses an array that still holds the first call's
values.  Outputs, slots, block tables and every appended K/V row must be
identical, and both must meet the parity bar against the oracle.  An
iteration whose workspace exceeds the array is refused with SLW_ENOMEM and
leaves the block manager as it was.
"""
import numpy as np
import pytest

from paper_2609_07883_amd import api, synth
from tests.parity import Mirror, check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _pair(shape, **kw):
    from paper_2609_07883_amd.runtime import Session
    a = Session(shape, **kw)
    b = Session(shape, layers=a.layer_bits, **{k: v for k, v in kw.items() if k != "qk_std"})
    return a, b


def _run_static(sess, batch, x_bits):
    m = batch.rows
    sess.x_in[:m].copy_(torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(sess.dev)
                        .view(torch.bfloat16))
    sess.ctx.mixed_iteration_static(batch, sess.x_in.data_ptr(), sess.x_out.data_ptr(), sess.stream())
    return sess.output(m)


@pytest.mark.parametrize("shape_name", ["tiny2", "gqa8b"])
def test_static_entry_matches_workspace_entry(shape_name):
    _require_gpu()
    if shape_name == "tiny2":
        shape = synth.with_layers(synth.TINY, 2)
        a, b = _pair(shape, num_blocks=256, max_c=320, max_b=4, qk_std=0.16)
        calls = [  # (C, prefix, decode contexts): the second call is smaller
            (300, 40, [33, 130, 17]),
            (21, 340, [34]),
        ]
    else:
        shape = synth.LLAMA8B_LAYER
        a, b = _pair(shape, num_blocks=256, max_c=96, max_b=4)
        calls = [(90, 20, [100, 7, 64]), (5, 110, [101])]
    ma, mb = Mirror(a, seed=9), Mirror(b, seed=9)
    pre = 5
    dec = [61, 62, 63]
    for mir in (ma, mb):
        mir.create(pre)
        mir.install_context(pre, calls[0][1])
        for sid, L in zip(dec, calls[0][2]):
            mir.create(sid)
            mir.install_context(sid, L)
    for i, (C, P, ctx) in enumerate(calls):
        batch = api.Batch(C, pre, P, dec[:len(ctx)], ctx)
        x = synth.embeddings(batch.rows, shape.d_model, seed=1, stream=77 + i)
        print(f"{shape_name} call {i}: C={C} P={P} B={len(ctx)}", flush=True)
        y_ref_gpu, y_oracle, sg, sr = ma.step(batch, x)        # the workspace entry point
        y_static = _run_static(b, batch, x)
        assert b.ctx.last_slots() == sg == sr
        np.testing.assert_array_equal(y_static, y_ref_gpu)
        e = check(y_static, y_oracle, f"{shape_name} static call {i}", layers=shape.n_layers)
        print(f"{shape_name} call {i}: identical to the workspace entry point; oracle {e}", flush=True)
        for sid in [pre] + dec:
            assert b.ctx.block_table(sid) == a.ctx.block_table(sid)
        seqs = [pre] * C + dec[:len(ctx)]
        pos = list(range(P, P + C)) + list(ctx)
        for layer in range(shape.n_layers):
            for sid in set(seqs):
                ps = [p for s, p in zip(seqs, pos) if s == sid]
                ka, va = a.read_kv(layer, sid, ps)
                kb, vb = b.read_kv(layer, sid, ps)
                np.testing.assert_array_equal(kb, ka)
                np.testing.assert_array_equal(vb, va)


def test_static_entry_refuses_iterations_beyond_its_array():
    """An 8B-shaped iteration of 2048 chunk rows needs more than the array
    holds: refused before any reservation or launch.  The buffers are full
    size all the same (uninitialised weights), so that nothing could read
    outside them."""
    _require_gpu()
    shape = synth.LLAMA8B_LAYER
    ctx = api.Context.from_shape(shape)
    dev = torch.device("cuda", torch.cuda.current_device())
    need = ctx.workspace_size(2048, 0)
    assert need > api.STATIC_WS_BYTES
    d, f, qw = shape.d_model, shape.ffn_dim, (shape.n_q_heads + 2 * shape.n_kv_heads) * shape.head_dim
    w = [torch.empty(n, dtype=torch.bfloat16, device=dev)
         for n in (qw * d, d * shape.n_q_heads * shape.head_dim, 2 * f * d, d * f, d, d)]
    for layer in range(shape.n_layers):
        ctx.set_layer_weights(layer, *(t.data_ptr() for t in w))
    blocks = 200
    page = shape.n_kv_heads * shape.head_dim * 16
    kpool = torch.zeros(shape.n_layers * blocks * page, dtype=torch.bfloat16, device=dev)
    vpool = torch.zeros_like(kpool)
    ctx.kv_init(kpool.data_ptr(), vpool.data_ptr(), blocks)
    ctx.seq_create(1)
    free = ctx.free_blocks()
    x = torch.zeros((2048, shape.d_model), dtype=torch.bfloat16, device=dev)
    with pytest.raises(api.SloweaveError) as e:
        ctx.mixed_iteration_static(api.Batch(2048, 1, 0, [], []), x.data_ptr(), x.data_ptr(),
                                   torch.cuda.current_stream(dev).cuda_stream)
    assert e.value.code == api.ENOMEM and "static workspace" in str(e.value)
    assert ctx.free_blocks() == free and ctx.block_table(1) == []

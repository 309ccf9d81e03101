"""GPU parity with every KV-pool slot that no token owns holding NaN.

Attention reads whole 16-token pages (and, past a key range's last page, that
page again in place of the next ones), so the slots after a sequence's last
token are read too.  Their keys must get probability 0 and their values must
not reach the output: chunk attention zeroes them in LDS on an item's last
tile, decode attention masks them per lane.  The pools are filled with NaN
before any context is installed, so a slot that leaks turns its row into NaN
and fails the comparison with the float64 oracle.

Steps, for MHA at head dim 64 and a group of 4 at head dim 128: a 50-row chunk
after a 45-token prefix beside decodes at contexts 0, 5, 37 and 100 (chunk and
decode attention in one launch), the next 30 rows of that prompt alone (chunk
attention alone), and a decode-only iteration (the decode kernel alone).
"""
import numpy as np
import pytest

from paper_2609_07883_amd import api, synth
from paper_2609_07883_amd.synth import ModelShape
from tests.parity import TOL, Mirror, check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SHAPES = {
    "mha_hd64": synth.TINY,
    "gqa4_hd128": ModelShape(n_layers=1, d_model=512, n_q_heads=4, n_kv_heads=1, head_dim=128, ffn_dim=512,
                             rms_eps=1e-5, rope_theta=10000.0, max_pos=4096),
}


@pytest.mark.parametrize("name", list(SHAPES))
def test_nan_in_unowned_slots_never_reaches_the_output(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_07883_amd.runtime import Session
    shape = SHAPES[name]
    qk_std = 0.16 * (256 / shape.d_model) ** 0.5 * (64 / shape.head_dim) ** 0.25
    sess = Session(shape, num_blocks=128, max_c=64, max_b=4, qk_std=qk_std)
    sess.k_pool.fill_(float("nan"))
    sess.v_pool.fill_(float("nan"))
    torch.cuda.synchronize()
    mir = Mirror(sess, seed=5)
    dec, ctx = [21, 22, 23, 24], [0, 5, 37, 100]
    for sid, L in zip(dec, ctx):
        mir.create(sid)
        mir.install_context(sid, L)
    pre = 3
    mir.create(pre)
    mir.install_context(pre, 45)
    steps = [api.Batch(50, pre, 45, dec, ctx),
             api.Batch(30, pre, 95, [], []),
             api.Batch(0, 0, 0, dec, [L + 1 for L in ctx])]
    for i, b in enumerate(steps):
        x = synth.embeddings(b.rows, shape.d_model, seed=1, stream=400 + i)
        y, yr, sg, sr = mir.step(b, x)
        assert sg == sr, f"{name}: slots differ at step {i}"
        assert np.isfinite(np.asarray(y, dtype=np.float64)).all(), f"{name}: NaN in step {i}"
        check(y, yr, f"{name} step {i}")
        assert mir.kv_error(b) <= TOL

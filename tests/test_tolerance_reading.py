"""Pin of the parity bar's reading against an exact bf16-storage emulation (CPU).

The stated bar is a maximum relative error of 2e-2 for bf16 inputs with fp32
accumulation, with no denominator given.  Two readings:

  elementwise   max_i |g_i - r_i| / (|r_i| + rms(r)) over a whole tensor;
  per vector    max over output vectors v of max_i |g_vi - r_vi| / max_i |r_vi|
                (a token's output row, one head of an appended K/V row),
                together with the rms error ||g - r|| / ||r||.

This test runs the 8B-shaped layer (d 4096, 32/8 heads of 128, FFN 14336)
over a 200-token prefill chunk twice on the CPU: exactly (the float64 oracle)
and with every value that a bf16 matrix-core pipeline stores in bf16 rounded
to bf16 (round to nearest even) at the point where it is stored, everything
else in float64.  Such a pipeline has no error source besides those
roundings, so its errors are a floor for any bf16 implementation.  The test
pins three facts the parity harness relies on:

  * with the residual stream stored in bf16 (the usual bf16 pipeline) the
    elementwise reading exceeds 2e-2, so no bf16 implementation can be held
    to it reliably;
  * the per-vector reading stays below 1e-2 and the rms error below 6e-3
    for the same pipeline, well inside 2e-2;
  * with the residual stream kept in fp32 inside the layer (as the HIP path
    keeps it), the elementwise figure still sits near 2e-2 but below
    ELEMENTWISE_TOL, the bound the harness asserts on top of the per-vector
    bar for every GPU case;
  * over two stacked layers (bf16 rows handed from one layer to the next)
    the elementwise floor grows about as sqrt(2), to which the harness scales
    its bound for stacks, while the per-vector reading stays near 1e-2.
"""
import numpy as np

from oracle import layer as OL
from paper_2609_07883_amd import synth
from tests.oracle_fixtures import oracle_shape, oracle_weights
from tests.parity import ELEMENTWISE_TOL, elementwise_err, rel_err, rms_err


def _bf(a):
    return synth.bf16_to_f64(synth.bf16_bits(np.asarray(a, dtype=np.float32)))


def _keep(a):
    return np.asarray(a, dtype=np.float64)


def _layer(sh, w, x, pos, rnd, resid_rnd):
    """One prefill chunk at positions `pos` (the whole sequence) with rounding
    `rnd` applied where a bf16 pipeline stores a value: the normed rows, q/k/v
    after RoPE (also the cached K/V), the softmax weights fed to the P.V
    product, the attention output, the SwiGLU activation and the layer
    output; `resid_rnd` is applied to the residual stream after attention."""
    m = x.shape[0]
    hq, hkv, hd, f = sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.ffn_dim
    u = rnd(OL.rms_norm(x, w.g1, sh.rms_eps))
    qkv = u @ w.wqkv.T
    q = rnd(OL.apply_rope(qkv[:, : hq * hd].reshape(m, hq, hd), pos, sh.rope_theta))
    k = rnd(OL.apply_rope(qkv[:, hq * hd: (hq + hkv) * hd].reshape(m, hkv, hd), pos, sh.rope_theta))
    v = rnd(qkv[:, (hq + hkv) * hd:].reshape(m, hkv, hd))
    o = np.empty((m, hq, hd))
    g = sh.group
    for r in range(m):
        for h in range(hq):
            s = k[: r + 1, h // g] @ q[r, h] / np.sqrt(hd)
            p = np.exp(s - np.max(s))
            o[r, h] = (rnd(p) @ v[: r + 1, h // g]) / np.sum(p)
    o = rnd(o)
    hres = resid_rnd(x + o.reshape(m, -1) @ w.wo.T)
    wn = rnd(OL.rms_norm(hres, w.g2, sh.rms_eps))
    gu = wn @ w.wgu.T
    a = rnd(OL.silu(gu[:, :f]) * gu[:, f:])
    return rnd(hres + a @ w.wd.T), k, v


def test_elementwise_reading_is_unreachable_for_bf16_storage():
    s = synth.LLAMA8B_LAYER
    sh = oracle_shape(s)
    w = oracle_weights(synth.layer_weights(s, weight_seed=0))
    C = 200
    x = synth.bf16_to_f64(synth.embeddings(C, s.d_model, seed=1, stream=7 * C))
    pos = np.arange(C)
    # exact: the oracle itself (its own chunked-prefill entry point)
    kv = OL.KVState()
    y_ref = OL.mixed_iteration(sh, w, x, kv, OL.MixedBatch(C, 1, 0, [], []))
    k_ref, v_ref = kv.seqs[1].k, kv.seqs[1].v
    # the emulation with every rounding off reproduces the oracle
    y0, _, _ = _layer(sh, w, x, pos, _keep, _keep)
    assert np.max(np.abs(y0 - y_ref)) <= 1e-12 * np.max(np.abs(y_ref))

    y_bf, k_bf, v_bf = _layer(sh, w, x, pos, _bf, _bf)        # residual stored in bf16
    y_f32, _, _ = _layer(sh, w, x, pos, _bf, _keep)            # residual kept wide
    e_bf = elementwise_err(y_bf, y_ref)
    e_f32 = elementwise_err(y_f32, y_ref)
    print(f"bf16 residual: elementwise {e_bf:.4f} per-vector {rel_err(y_bf, y_ref):.4f} "
          f"rms {rms_err(y_bf, y_ref):.5f}; fp32 residual: elementwise {e_f32:.4f} "
          f"per-vector {rel_err(y_f32, y_ref):.4f} rms {rms_err(y_f32, y_ref):.5f}")
    assert e_bf > 2e-2
    assert rel_err(y_bf, y_ref) <= 1e-2 and rms_err(y_bf, y_ref) <= 6e-3
    assert rel_err(k_bf.reshape(-1, s.head_dim), k_ref.reshape(-1, s.head_dim)) <= 1e-2
    assert rel_err(v_bf.reshape(-1, s.head_dim), v_ref.reshape(-1, s.head_dim)) <= 1e-2
    assert 1.5e-2 < e_f32 <= ELEMENTWISE_TOL
    assert rel_err(y_f32, y_ref) <= 1e-2 and rms_err(y_f32, y_ref) <= 6e-3


def test_elementwise_floor_of_a_two_layer_stack():
    """The 2-layer case of the GPU stack test (150-token chunk at prefix 0):
    the emulated floor with the residual in fp32 inside each layer and bf16
    rows between layers."""
    s = synth.LLAMA8B_LAYER
    sh = oracle_shape(s)
    ws = [oracle_weights(synth.layer_weights(s, layer=l, weight_seed=0)) for l in range(2)]
    C = 150
    x = synth.bf16_to_f64(synth.embeddings(C, s.d_model, seed=1, stream=11 * C))
    pos = np.arange(C)
    y_ref = OL.stack_iteration(sh, ws, x, [OL.KVState(), OL.KVState()], OL.MixedBatch(C, 1, 0, [], []))
    y = x
    for w in ws:
        y, _, _ = _layer(sh, w, y, pos, _bf, _keep)
    e = elementwise_err(y, y_ref)
    print(f"2-layer floor: elementwise {e:.4f} per-vector {rel_err(y, y_ref):.4f} rms {rms_err(y, y_ref):.5f}")
    assert 2.5e-2 < e <= ELEMENTWISE_TOL * np.sqrt(2)
    assert rel_err(y, y_ref) <= 1e-2 and rms_err(y, y_ref) <= 7e-3


def test_elementwise_floor_grows_with_the_score_spread():
    """The floor depends on how sharp attention is, not only on the shapes:
    with 16 q heads per kv head at d_model 1024 and the q/k weights at
    std 0.16, scores reach tens of units, softmax is nearly hard, and the
    bf16 rounding of the normed rows and of q/k alone moves the output past
    ELEMENTWISE_TOL; at the scale 0.16 sqrt(256 / d_model) (the spread of the
    d_model-256 cases) the same pipeline stays far inside it.  GPU cases of
    other widths scale their q/k weights that way, and those at head dim 128
    also by (64 / head_dim)^(1/4), since the scores grow with sqrt(head_dim)
    after the 1/sqrt(head_dim) scaling."""
    from tests.test_gpu_gqa import SHAPES
    s = SHAPES["gqa16_hd64"]
    sh = oracle_shape(s)
    C = 150
    x = synth.bf16_to_f64(synth.embeddings(C, s.d_model, seed=1, stream=3))
    pos = np.arange(C)
    errs = {}
    for qk in (0.16, 0.16 * (256 / s.d_model) ** 0.5):
        w = oracle_weights(synth.layer_weights(s, weight_seed=0, qk_std=qk))
        ref, _, _ = _layer(sh, w, x, pos, _keep, _keep)
        em, _, _ = _layer(sh, w, x, pos, _bf, _keep)
        errs[qk] = elementwise_err(em, ref)
    sharp, spread = errs.values()
    assert sharp > ELEMENTWISE_TOL
    assert spread < 0.5 * ELEMENTWISE_TOL

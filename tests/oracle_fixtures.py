"""Shared helpers for the oracle tests: shapes and seeded float64 weights."""
from __future__ import annotations

import numpy as np

from oracle.layer import LayerShape, LayerWeights
from paper_2609_07883_amd import synth


def oracle_shape(s: synth.ModelShape) -> LayerShape:
    return LayerShape(d_model=s.d_model, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                      head_dim=s.head_dim, ffn_dim=s.ffn_dim, rms_eps=s.rms_eps,
                      rope_theta=s.rope_theta)


def oracle_weights(bits: synth.LayerBits) -> LayerWeights:
    return LayerWeights(**bits.as_f64())


TINY_GQA = synth.ModelShape(n_layers=1, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=32,
                            ffn_dim=384, rms_eps=1e-5, rope_theta=10000.0, max_pos=4096)


def x_rows(rows: int, d: int, stream: int = 0) -> np.ndarray:
    return synth.bf16_to_f64(synth.embeddings(rows, d, seed=1, stream=stream))

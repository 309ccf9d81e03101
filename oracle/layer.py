"""Oracle for one decoder layer of a mixed prefill+decode iteration.

Test infrastructure only (see ``oracle/__init__``).

What is computed
----------------
The paper schedules an unmodified model: "model kernels require no semantic
changes" (Sec. 5.1) and the executor needs no new operator (Table 1).  Its
GPU study runs an "8B dense decoder" (Sec. 5.2) without defining it further,
so the layer here is the standard Llama-style pre-norm block:

    u  = RMSNorm(x; g1)
    q, k, v = u Wq^T, u Wk^T, u Wv^T
    q, k    = RoPE(q, pos), RoPE(k, pos)        (rotate-half form)
    K[seq, pos], V[seq, pos] = k, v             (append to the sequence's cache)
    o_h = sum_{p' <= pos} softmax_p'(q_h . K[g(h), p'] / sqrt(hd)) V[g(h), p']
    h  = x + o Wo^T
    y  = h + (silu(w Wg^T) * (w Wu^T)) Wd^T,    w = RMSNorm(h; g2)

with g(h) = h // (Hq / Hkv) (grouped-query attention).  A mixed iteration
holds C rows of one prefill sequence at positions P..P+C-1 followed by B
decode rows, decode b at position L_b (its cached length before the
iteration).  Every row attends over its own sequence's keys 0..pos,
including the keys written in this same iteration.  Chunked prefill
(Sec. 2.2) and the paged layout (Table 1) only change where and when these
values are computed, not the values, so K/V are held here as one dense
array per sequence and no paging appears.

Precision: float64 throughout.  The paper fixes no precision; the GPU path
runs bf16 storage with fp32 accumulation and is compared to this within a
tolerance.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class LayerShape:
    """Dimensions and constants of one layer (no defaults: callers state them)."""

    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    rms_eps: float
    rope_theta: float

    @property
    def group(self) -> int:
        assert self.n_q_heads % self.n_kv_heads == 0
        return self.n_q_heads // self.n_kv_heads


@dataclass
class LayerWeights:
    """Weights as float64 arrays, row-major [out][in].

    wqkv: [(Hq + 2 Hkv) * hd][d]  (q rows, then k rows, then v rows)
    wo:   [d][Hq * hd]
    wgu:  [2 F][d]                 (gate rows, then up rows)
    wd:   [d][F]
    g1, g2: [d]                    RMSNorm gains
    """

    wqkv: np.ndarray
    wo: np.ndarray
    wgu: np.ndarray
    wd: np.ndarray
    g1: np.ndarray
    g2: np.ndarray


@dataclass
class SeqCache:
    """Dense K/V of one sequence: k, v are [len][Hkv][hd] float64."""

    k: np.ndarray
    v: np.ndarray

    @property
    def length(self) -> int:
        return self.k.shape[0]


@dataclass
class KVState:
    """All sequences' caches for one layer, keyed by sequence id."""

    seqs: dict = field(default_factory=dict)

    def copy(self) -> "KVState":
        return KVState({s: SeqCache(c.k.copy(), c.v.copy()) for s, c in self.seqs.items()})


# ---------------------------------------------------------------------------
# Elementwise pieces
# ---------------------------------------------------------------------------

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm (Zhang & Sennrich 2019): x / sqrt(mean(x^2) + eps) * g, per row."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, dtype=np.float64)


def rope_angles(pos: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """Angles a[p, i] = p * theta^(-2 i / hd) for i < hd/2 (Su et al. 2021)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = float(theta) ** (-2.0 * i / head_dim)
    return np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]


def apply_rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE on x[n][heads][hd] at absolute positions pos[n].

    Pairs (i, i + hd/2) are rotated by a_i:
        x_i'        = x_i cos a_i - x_{i+hd/2} sin a_i
        x_{i+hd/2}' = x_{i+hd/2} cos a_i + x_i sin a_i
    """
    x = np.asarray(x, dtype=np.float64)
    hd = x.shape[-1]
    half = hd // 2
    a = rope_angles(pos, hd, theta)[:, None, :]          # [n][1][hd/2]
    c, s = np.cos(a), np.sin(a)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU (Shazeer 2020): z / (1 + exp(-z))."""
    return z / (1.0 + np.exp(-z))


def attend_row(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_keys: int,
               group: int) -> np.ndarray:
    """Softmax attention of one query row over the first n_keys keys.

    q: [Hq][hd]; k, v: [>= n_keys][Hkv][hd].  q-head h uses kv-head h // group
    and scale 1/sqrt(hd).  Returns [Hq][hd].
    """
    hq, hd = q.shape
    out = np.empty((hq, hd), dtype=np.float64)
    scale = 1.0 / np.sqrt(hd)
    for h in range(hq):
        g = h // group
        kk = k[:n_keys, g, :]
        vv = v[:n_keys, g, :]
        s = (kk @ q[h]) * scale
        w = np.exp(s - np.max(s))
        w /= np.sum(w)
        out[h] = w @ vv
    return out


# ---------------------------------------------------------------------------
# The mixed iteration
# ---------------------------------------------------------------------------

@dataclass
class MixedBatch:
    """One iteration's batch (the chunk rides in ordinary sequence metadata, Sec. 5.1).

    Rows 0..C-1 are the prefill chunk of ``prefill_seq`` at positions
    prefix_len..prefix_len+C-1; rows C..C+B-1 are one decode token each for
    ``decode_seqs[b]`` at position ``context_lens[b]`` (tokens cached before
    this iteration).  With prefill batching (Sec. 3.3) ``prefills`` lists
    several (sequence, prefix, chunk) triples instead: the chunk rows are
    those of each triple in turn and ``chunk`` is their total.
    """

    chunk: int
    prefill_seq: int
    prefix_len: int
    decode_seqs: list
    context_lens: list
    prefills: list | None = None

    @property
    def prefill_list(self):
        """The (sequence, prefix, chunk) triples whose rows come first."""
        if self.prefills is not None:
            return [tuple(p) for p in self.prefills if p[2] > 0]
        return [(self.prefill_seq, self.prefix_len, self.chunk)] if self.chunk > 0 else []

    @property
    def rows(self) -> int:
        return self.chunk + len(self.decode_seqs)

    def row_seq_pos(self):
        seqs, pos = [], []
        for sid, p0, c in self.prefill_list:
            seqs += [sid] * c
            pos += list(range(p0, p0 + c))
        return seqs + list(self.decode_seqs), pos + list(self.context_lens)


def qkv_rope(shape: LayerShape, w: LayerWeights, x: np.ndarray, pos):
    """Steps 1-3: RMSNorm, QKV projection, RoPE.  Returns q [M][Hq][hd], k, v [M][Hkv][hd]."""
    m = x.shape[0]
    hq, hkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    u = rms_norm(x, w.g1, shape.rms_eps)
    qkv = u @ w.wqkv.T
    q = qkv[:, : hq * hd].reshape(m, hq, hd)
    k = qkv[:, hq * hd: (hq + hkv) * hd].reshape(m, hkv, hd)
    v = qkv[:, (hq + hkv) * hd:].reshape(m, hkv, hd)
    pos = np.asarray(pos, dtype=np.int64)
    return apply_rope(q, pos, shape.rope_theta), apply_rope(k, pos, shape.rope_theta), v


def append_kv(shape: LayerShape, kv: KVState, seqs, pos, k, v) -> None:
    """Step 4: write k[r], v[r] at position pos[r] of sequence seqs[r].

    A row at position p requires the sequence to hold at least p cached
    tokens before this iteration's rows are written (positions are dense).
    """
    hkv, hd = shape.n_kv_heads, shape.head_dim
    grown = {}      # sequence -> rows that extend it, in position order
    for r, (s, p) in enumerate(zip(seqs, pos)):
        if s not in kv.seqs:
            kv.seqs[s] = SeqCache(np.zeros((0, hkv, hd)), np.zeros((0, hkv, hd)))
        c = kv.seqs[s]
        new = grown.setdefault(s, [])
        if p > c.length + len(new):
            raise ValueError(f"seq {s}: row at position {p} but only {c.length + len(new)} cached")
        if p == c.length + len(new):
            new.append(r)
        elif p >= c.length:
            new[p - c.length] = r
        else:
            c.k[p] = k[r]
            c.v[p] = v[r]
    for s, new in grown.items():     # one copy per sequence, not one per row
        if new:
            c = kv.seqs[s]
            c.k = np.concatenate([c.k, np.asarray(k)[new]])
            c.v = np.concatenate([c.v, np.asarray(v)[new]])


def mlp_rows(shape: LayerShape, w: LayerWeights, x: np.ndarray, o: np.ndarray) -> np.ndarray:
    """Steps 6-7: output projection plus residual, then the SwiGLU MLP plus residual."""
    f = shape.ffn_dim
    h = x + o.reshape(o.shape[0], -1) @ w.wo.T
    wn = rms_norm(h, w.g2, shape.rms_eps)
    gu = wn @ w.wgu.T
    a = silu(gu[:, :f]) * gu[:, f:]
    return h + a @ w.wd.T


def mixed_iteration(shape: LayerShape, w: LayerWeights, x: np.ndarray,
                    kv: KVState, batch: MixedBatch, rows=None) -> np.ndarray:
    """One layer over a mixed batch; updates ``kv`` in place and returns y [M][d].

    If ``rows`` is given, only those output rows are computed (the others are
    returned as NaN); the K/V of every row are still appended, since every
    row's keys feed later rows of its sequence.
    """
    x = np.asarray(x, dtype=np.float64)
    m = batch.rows
    assert x.shape == (m, shape.d_model)
    seqs, pos = batch.row_seq_pos()
    pre = batch.prefill_list
    if sum(c for _, _, c in pre) != batch.chunk:
        raise ValueError("the prefills' chunks must add up to the chunk rows")
    listed = [sid for sid, _, _ in pre] + list(batch.decode_seqs)
    if len(set(listed)) != len(listed):
        raise ValueError("a sequence may appear at most once per iteration")
    for s, p in zip(batch.decode_seqs, batch.context_lens):
        have = kv.seqs[s].length if s in kv.seqs else 0
        if have != p:
            raise ValueError(f"decode seq {s}: context_len {p} but {have} cached")
    for sid, p0, _ in pre:
        have = kv.seqs[sid].length if sid in kv.seqs else 0
        if have != p0:
            raise ValueError(f"prefill seq {sid}: prefix_len {p0} but {have} cached")

    q, k, v = qkv_rope(shape, w, x, pos)
    append_kv(shape, kv, seqs, pos, k, v)

    want = range(m) if rows is None else sorted(set(int(r) for r in rows))
    y = np.full((m, shape.d_model), np.nan)
    if len(want) == 0:
        return y
    want = np.asarray(list(want), dtype=np.int64)
    o = np.empty((len(want), shape.n_q_heads, shape.head_dim))
    for i, r in enumerate(want):
        c = kv.seqs[seqs[r]]
        o[i] = attend_row(q[r], c.k, c.v, pos[r] + 1, shape.group)
    y[want] = mlp_rows(shape, w, x[want], o)
    return y


def attention_outputs(shape: LayerShape, w: LayerWeights, x: np.ndarray,
                      kv: KVState, batch: MixedBatch) -> np.ndarray:
    """Attention output o [M][Hq][hd] of the mixed iteration (updates ``kv``).

    The same steps as ``mixed_iteration`` stopped before the output
    projection; used to compare the attention stage on its own.
    """
    seqs, pos = batch.row_seq_pos()
    q, k, v = qkv_rope(shape, w, np.asarray(x, dtype=np.float64), pos)
    append_kv(shape, kv, seqs, pos, k, v)
    o = np.empty((batch.rows, shape.n_q_heads, shape.head_dim))
    for r in range(batch.rows):
        c = kv.seqs[seqs[r]]
        o[r] = attend_row(q[r], c.k, c.v, pos[r] + 1, shape.group)
    return o


def stack_iteration(shape: LayerShape, layers, x: np.ndarray, kvs, batch: MixedBatch) -> np.ndarray:
    """A stack of layers: layer l reads layer l-1's output and its own cache kvs[l]."""
    for w, kv in zip(layers, kvs):
        x = mixed_iteration(shape, w, x, kv, batch)
    return x

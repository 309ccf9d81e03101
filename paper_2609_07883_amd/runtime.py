"""Device-memory plumbing around the C ABI (PyTorch for allocation and streams only).

``Session`` allocates the caller-owned buffers the library needs (weights,
paged KV pools, input/output rows, workspace) as torch tensors on the GPU and
hands their addresses to ``api.Context``.  It also writes and reads cached
K/V pages in the library's documented pool layout, which tests and benchmarks
use to install pre-existing contexts and to inspect what an iteration
appended; that is set-up and inspection, not a step of the iteration.
"""
from __future__ import annotations

import numpy as np
import torch

from . import api, synth


def _dev():
    if not torch.cuda.is_available():
        raise RuntimeError("a ROCm GPU is required")
    return torch.device("cuda", torch.cuda.current_device())


def bits_to_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns -> torch.bfloat16 tensor on device."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def tensor_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


class Session:
    """One context with its device buffers for iterations up to (max_c, max_b)."""

    def __init__(self, shape: synth.ModelShape, num_blocks: int, max_c: int, max_b: int,
                 layers=None, weight_seed: int = 0, qk_std=None, device_weights: bool = False):
        """device_weights draws the weights on the GPU (the library's Philox
        generator, seeds derived from weight_seed + 1000 * layer; N(0, 0.02)
        matrices, 1 + N(0, 0.02) gains) instead of the host recipe of
        ``synth.layer_weights``: for deep stacks whose outputs are timed but
        never compared with the oracle."""
        self.shape = shape
        self.dev = _dev()
        self.ctx = api.Context.from_shape(shape)
        self.num_blocks = num_blocks
        s = shape
        self.k_pool = torch.zeros((s.n_layers, num_blocks, s.n_kv_heads, s.head_dim // 32, 16, 32),
                                  dtype=torch.bfloat16, device=self.dev)
        self.v_pool = torch.zeros((s.n_layers, num_blocks, s.n_kv_heads, s.head_dim, 16),
                                  dtype=torch.bfloat16, device=self.dev)
        self.ctx.kv_init(self.k_pool.data_ptr(), self.v_pool.data_ptr(), num_blocks)
        self.weights = []
        self.layer_bits = []
        for layer in range(s.n_layers):
            if device_weights:
                w = self._device_layer(weight_seed + 1000 * layer)
                self.layer_bits.append(None)
            else:
                bits = layers[layer] if layers is not None else synth.layer_weights(
                    s, layer=layer, weight_seed=weight_seed, qk_std=qk_std)
                self.layer_bits.append(bits)
                w = {k: bits_to_tensor(getattr(bits, k), self.dev)
                     for k in ("wqkv", "wo", "wgu", "wd", "g1", "g2")}
            self.weights.append(w)
            self.ctx.set_layer_weights(layer, *(w[k].data_ptr() for k in
                                                ("wqkv", "wo", "wgu", "wd", "g1", "g2")))
        self.max_c, self.max_b = max_c, max_b
        rows = max(1, max_c + max_b)
        self.x_in = torch.zeros((rows, s.d_model), dtype=torch.bfloat16, device=self.dev)
        self.x_out = torch.zeros_like(self.x_in)
        self.ws_bytes = self.ctx.workspace_size(max_c, max_b)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)

    def _device_layer(self, seed: int) -> dict:
        """One layer drawn on the device by the library's seeded generator:
        matrix j of the layer (wqkv, wo, wgu, wd, g1, g2) from the stream
        keyed by seed * 16 + j; N(0, 0.02) matrices, 1 + N(0, 0.02) gains."""
        s = self.shape
        nqkv = (s.n_q_heads + 2 * s.n_kv_heads) * s.head_dim
        shapes = {"wqkv": (nqkv, s.d_model), "wo": (s.d_model, s.n_q_heads * s.head_dim),
                  "wgu": (2 * s.ffn_dim, s.d_model), "wd": (s.d_model, s.ffn_dim),
                  "g1": (s.d_model,), "g2": (s.d_model,)}
        stream = self.stream()
        w = {}
        for j, (k, shp) in enumerate(shapes.items()):
            t = torch.empty(shp, dtype=torch.bfloat16, device=self.dev)
            api.fill_normal(t.data_ptr(), t.numel(), seed * 16 + j, 1.0 if k in ("g1", "g2") else 0.0, 0.02, stream)
            w[k] = t
        return w

    # -- iteration ------------------------------------------------------------
    def stream(self) -> int:
        return torch.cuda.current_stream(self.dev).cuda_stream

    def run(self, batch: api.Batch, x_bits=None) -> None:
        """Enqueue one iteration on the current stream (x_bits: uint16 [rows][d] or None)."""
        m = batch.rows
        if m > self.x_in.shape[0] or batch.chunk > self.max_c or len(batch.decode_seqs) > self.max_b:
            raise ValueError(f"batch of C={batch.chunk}, B={len(batch.decode_seqs)} exceeds this session's "
                             f"buffers (C<={self.max_c}, B<={self.max_b})")
        if x_bits is not None:
            self.x_in[:m].copy_(bits_to_tensor(x_bits, self.dev))
        self.ctx.mixed_iteration(batch, self.x_in.data_ptr(), self.x_out.data_ptr(),
                                 self.ws.data_ptr(), self.ws_bytes, self.stream())

    def output(self, rows: int) -> np.ndarray:
        torch.cuda.synchronize(self.dev)
        return tensor_to_f64(self.x_out[:rows])

    def view(self, which: int, c: int, b: int, cols: int, fp32: bool = False) -> np.ndarray:
        """A workspace intermediate of the last iteration (see slw_workspace_view)."""
        torch.cuda.synchronize(self.dev)
        off, nbytes = self.ctx.workspace_view(which, c, b)
        t = self.ws[off: off + nbytes].view(torch.float32 if fp32 else torch.bfloat16).view(c + b, cols)
        return tensor_to_f64(t)

    # -- cached K/V in the pool layout ---------------------------------------------
    def _index(self, sid: int, positions):
        bt = np.asarray(self.ctx.block_table(sid), dtype=np.int64)
        pos = np.asarray(positions, dtype=np.int64)
        blk = torch.from_numpy(bt[pos // 16]).to(self.dev)
        t = torch.from_numpy(pos % 16).to(self.dev)
        return blk, t

    def write_kv(self, layer: int, sid: int, k_bits: np.ndarray, v_bits: np.ndarray, start: int = 0):
        """Install K/V (uint16 [n][Hkv][hd]) at positions start..start+n-1 of sequence sid."""
        s = self.shape
        n = k_bits.shape[0]
        blk, t = self._index(sid, np.arange(start, start + n))
        k = bits_to_tensor(k_bits, self.dev).view(n, s.n_kv_heads, s.head_dim // 32, 32)
        v = bits_to_tensor(v_bits, self.dev).view(n, s.n_kv_heads, s.head_dim)
        self.k_pool[layer].permute(0, 3, 1, 2, 4)[blk, t] = k
        self.v_pool[layer].permute(0, 3, 1, 2)[blk, t] = v

    def read_kv(self, layer: int, sid: int, positions):
        """(K, V) float64 [n][Hkv][hd] at the given positions of sequence sid."""
        s = self.shape
        torch.cuda.synchronize(self.dev)
        blk, t = self._index(sid, positions)
        k = self.k_pool[layer].permute(0, 3, 1, 2, 4)[blk, t].reshape(len(positions), s.n_kv_heads, s.head_dim)
        v = self.v_pool[layer].permute(0, 3, 1, 2)[blk, t]
        return tensor_to_f64(k), tensor_to_f64(v)

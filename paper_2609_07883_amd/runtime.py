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
    """A bf16 (or fp32) tensor as float64 numbers: copied to the host first,
    converted there."""
    return t.detach().cpu().float().numpy().astype(np.float64)


def _page_bits(page: torch.Tensor) -> np.ndarray:
    """One pool page (bf16, any device) as a writable host uint16 array."""
    return page.view(torch.int16).cpu().numpy().view(np.uint16).copy()


def write_pages(k_pool: torch.Tensor, v_pool: torch.Tensor, blk: np.ndarray, tok: np.ndarray,
                k_bits: np.ndarray, v_bits: np.ndarray) -> None:
    """Write K/V rows into one layer's pools, page by page through host copies.

    k_pool is [blocks][Hkv][hd/32][16][32], v_pool [blocks][Hkv][hd][16]
    (bf16); row i (k_bits/v_bits uint16 [n][Hkv][hd]) goes to token tok[i] of
    block blk[i], and rows of one block are consecutive.  A page the rows fill
    is written whole; one they cover in part is read, updated and written
    back, so its other tokens keep what they held.  torch only moves memory.
    """
    n = len(blk)
    hkv, slabs = k_pool.shape[1], k_pool.shape[2]
    k = np.ascontiguousarray(k_bits, dtype=np.uint16).reshape(n, hkv, slabs, 32)
    v = np.ascontiguousarray(v_bits, dtype=np.uint16).reshape(n, hkv, slabs * 32)
    i = 0
    while i < n:
        b = int(blk[i])
        j = i + 1
        while j < n and blk[j] == b:
            j += 1
        t = np.asarray(tok[i:j], dtype=np.int64)
        if j - i == 16 and np.array_equal(np.sort(t), np.arange(16)):
            kpage = np.empty(tuple(k_pool.shape[1:]), dtype=np.uint16)
            vpage = np.empty(tuple(v_pool.shape[1:]), dtype=np.uint16)
        else:
            kpage, vpage = _page_bits(k_pool[b]), _page_bits(v_pool[b])
        kpage[:, :, t, :] = k[i:j].transpose(1, 2, 0, 3)
        vpage[:, :, t] = v[i:j].transpose(1, 2, 0)
        k_pool[b].copy_(torch.from_numpy(kpage.view(np.int16)).view(torch.bfloat16))
        v_pool[b].copy_(torch.from_numpy(vpage.view(np.int16)).view(torch.bfloat16))
        i = j


def read_pages(k_pool: torch.Tensor, v_pool: torch.Tensor, blk: np.ndarray, tok: np.ndarray):
    """(K, V) uint16 [n][Hkv][hd]: the rows at token tok[i] of block blk[i] of
    one layer's pools (layouts as in write_pages), read page by page."""
    n = len(blk)
    hkv, slabs = k_pool.shape[1], k_pool.shape[2]
    k = np.empty((n, hkv, slabs * 32), dtype=np.uint16)
    v = np.empty((n, hkv, slabs * 32), dtype=np.uint16)
    blk = np.asarray(blk, dtype=np.int64)
    tok = np.asarray(tok, dtype=np.int64)
    for b in np.unique(blk):
        sel = np.nonzero(blk == b)[0]
        kpage, vpage = _page_bits(k_pool[int(b)]), _page_bits(v_pool[int(b)])
        k[sel] = kpage[:, :, tok[sel], :].transpose(2, 0, 1, 3).reshape(len(sel), hkv, slabs * 32)
        v[sel] = vpage[:, :, tok[sel]].transpose(2, 0, 1)
    return k, v


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
    def _pages(self, sid: int, positions):
        """(block id, token in the block) of each position of sequence sid."""
        bt = np.asarray(self.ctx.block_table(sid), dtype=np.int64)
        pos = np.asarray(positions, dtype=np.int64)
        return bt[pos // 16], pos % 16

    def write_kv(self, layer: int, sid: int, k_bits: np.ndarray, v_bits: np.ndarray, start: int = 0):
        """Install K/V (uint16 [n][Hkv][hd]) at positions start..start+n-1 of sequence sid."""
        blk, tok = self._pages(sid, np.arange(start, start + k_bits.shape[0]))
        write_pages(self.k_pool[layer], self.v_pool[layer], blk, tok, k_bits, v_bits)

    def read_kv(self, layer: int, sid: int, positions):
        """(K, V) float64 [n][Hkv][hd] at the given positions of sequence sid."""
        torch.cuda.synchronize(self.dev)
        blk, tok = self._pages(sid, positions)
        k, v = read_pages(self.k_pool[layer], self.v_pool[layer], blk, tok)
        return synth.bf16_to_f64(k), synth.bf16_to_f64(v)

"""ctypes binding of libsloweave.so (argument marshalling only).

Every computation happens in the library: the mixed iteration in its gfx950
kernels, the block manager, profiler and controller in its host code.  This
module converts Python values to the C ABI of ``include/sloweave.h`` and
raises ``SloweaveError`` for every negative return code.  Device buffers are
passed as integer addresses (``tensor.data_ptr()``) and streams as integer
handles (``torch.cuda.current_stream().cuda_stream``).

A missing library is an error, never a fallback: build it with
``python -m paper_2609_07883_amd.build``.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsloweave.so")

OK, EINVAL, ERANGE, ENOMEM, EHIP, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
FLAG_NO_PENDING, FLAG_NO_ACTIVE, FLAG_DECODE_INFEASIBLE, FLAG_CAPPED_BY_GRID = 1, 2, 4, 8
VIEW_QKV, VIEW_ATTN, VIEW_H, VIEW_ACT = 0, 1, 2, 3
TABLE_SAMPLES, TABLE_P50, TABLE_P99, TABLE_THAT = 0, 1, 2, 3

EXPORTS = (
    "slw_last_error", "slw_create", "slw_destroy", "slw_set_layer_weights", "slw_kv_init",
    "slw_kv_free_blocks", "slw_seq_create", "slw_seq_free", "slw_seq_reserve",
    "slw_seq_block_table", "slw_workspace_size", "slw_mixed_iteration", "slw_last_slots",
    "slw_workspace_view", "slw_build_cost_table", "slw_cost_table_from_samples",
    "slw_cost_table_free", "slw_cost_table_dims", "slw_cost_table_grids", "slw_cost_table_values",
    "slw_cost_table_lookup", "slw_cost_table_monotone", "slw_cost_table_save",
    "slw_cost_table_load", "slw_select_chunk", "slw_set_stage_timing", "slw_stage_times",
    "slw_serve", "slw_cost_table_analytic", "slw_build_cost_table_ctx", "slw_cost_table_from_samples_ctx",
    "slw_cost_table_prefixes", "slw_cost_table_lookup_ctx", "slw_select_chunk_ctx",
    "slw_mixed_iteration_static", "slw_flush_cache", "slw_fill_normal", "slw_gemm_plan",
    "slw_attention_plan",
)
STATIC_WS_BYTES = 128 << 20
STAGES = ("rmsnorm_attn", "rope_table", "qkv_gemm", "chunk_attn", "decode_attn", "attn_merge",
          "o_gemm", "rmsnorm_mlp", "gateup_gemm", "down_gemm")


class SloweaveError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"sloweave error {code}: {msg}")
        self.code = code


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float), ("block_size", C.c_int32),
                ("max_pos", C.c_int32)]


class LayerWeightsC(C.Structure):
    _fields_ = [("wqkv", C.c_void_p), ("wo", C.c_void_p), ("wgu", C.c_void_p), ("wd", C.c_void_p),
                ("g1", C.c_void_p), ("g2", C.c_void_p)]


class BatchC(C.Structure):
    _fields_ = [("C", C.c_int32), ("prefill_seq", C.c_int64), ("prefix_len", C.c_int32),
                ("B", C.c_int32), ("decode_seqs", C.POINTER(C.c_int64)),
                ("context_lens", C.POINTER(C.c_int32)), ("n_prefill", C.c_int32),
                ("prefill_seqs", C.POINTER(C.c_int64)), ("prefix_lens", C.POINTER(C.c_int32)),
                ("chunk_lens", C.POINTER(C.c_int32))]


MAX_PREFILLS = 16


class ProfileOpts(C.Structure):
    _fields_ = [("prefix_len", C.c_int32), ("ctx_lo", C.c_int32), ("ctx_hi", C.c_int32),
                ("seed", C.c_uint64), ("warmup", C.c_int32), ("repeats", C.c_int32),
                ("flush_buf", C.c_void_p), ("flush_bytes", C.c_size_t), ("x_in", C.c_void_p),
                ("x_out", C.c_void_p), ("ws", C.c_void_p), ("ws_bytes", C.c_size_t),
                ("stream", C.c_void_p)]


class RequestC(C.Structure):
    _fields_ = [("id", C.c_int64), ("arrival_ns", C.c_int64), ("prompt_len", C.c_int32),
                ("output_len", C.c_int32)]


class ServeOpts(C.Structure):
    _fields_ = [("policy", C.c_int32), ("fixed_chunk", C.c_int32), ("c_max", C.c_int32),
                ("max_decode", C.c_int32), ("tpot_ns", C.c_int64), ("margin_ns", C.c_int64),
                ("table", C.c_void_p), ("executor", C.c_int32), ("skip_idle", C.c_int32),
                ("x_in", C.c_void_p), ("x_out", C.c_void_p), ("max_rows", C.c_int32),
                ("ws", C.c_void_p), ("ws_bytes", C.c_size_t), ("stream", C.c_void_p),
                ("residual_window", C.c_int32), ("exec_table", C.c_void_p), ("slo", C.c_void_p),
                ("queue", C.c_int32), ("admit_ppm", C.c_int32), ("aging_ns", C.c_int64),
                ("aging_chunk", C.c_int32), ("max_prefills", C.c_int32), ("fallback_window", C.c_int32),
                ("log_every", C.c_int32)]


class RequestSloC(C.Structure):
    _fields_ = [("tpot_ns", C.c_int64), ("margin_ns", C.c_int64), ("ttft_ns", C.c_int64)]


class IterationRecord(C.Structure):
    _fields_ = [("start_ns", C.c_int64), ("end_ns", C.c_int64), ("budget_ns", C.c_int64),
                ("decide_ns", C.c_int64), ("predicted_ns", C.c_int64), ("prefill_id", C.c_int64),
                ("chunk", C.c_int32), ("n_decode", C.c_int32), ("remaining", C.c_int32),
                ("flags", C.c_uint32), ("rel_margin_ppm", C.c_int64), ("n_prefill", C.c_int32),
                ("reserved", C.c_int32), ("resid_p99_ns", C.c_int64)]


POLICY_SLOWEAVE, POLICY_FIXED = 0, 1
EXEC_GPU, EXEC_ANALYTIC, EXEC_TABLE = 0, 1, 2
SERVE_KV_WAIT, SERVE_DECODE_CAP, SERVE_UNPRICED, SERVE_AGED, SERVE_FALLBACK = 0x100, 0x200, 0x400, 0x800, 0x1000
QUEUES = {"oldest": 0, "srpt": 1, "edf": 2}

_lib = None


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2609_07883_amd.build`")
    L = C.CDLL(LIB_PATH)
    i32, i64, u32, vp, sz = C.c_int32, C.c_int64, C.c_uint32, C.c_void_p, C.c_size_t
    P = C.POINTER
    sig = {
        "slw_last_error": ([], C.c_char_p),
        "slw_create": ([P(ModelCfg), P(vp)], C.c_int),
        "slw_destroy": ([vp], C.c_int),
        "slw_set_layer_weights": ([vp, i32, P(LayerWeightsC)], C.c_int),
        "slw_kv_init": ([vp, vp, vp, i32], C.c_int),
        "slw_kv_free_blocks": ([vp, P(i32)], C.c_int),
        "slw_seq_create": ([vp, i64], C.c_int),
        "slw_seq_free": ([vp, i64], C.c_int),
        "slw_seq_reserve": ([vp, i64, i32], C.c_int),
        "slw_seq_block_table": ([vp, i64, P(i32), i32, P(i32)], C.c_int),
        "slw_workspace_size": ([vp, i32, i32, P(sz)], C.c_int),
        "slw_mixed_iteration": ([vp, P(BatchC), vp, vp, vp, sz, vp], C.c_int),
        "slw_mixed_iteration_static": ([vp, P(BatchC), vp, vp, vp], C.c_int),
        "slw_flush_cache": ([vp, sz, vp], C.c_int),
        "slw_fill_normal": ([vp, sz, C.c_uint64, C.c_float, C.c_float, vp], C.c_int),
        "slw_gemm_plan": ([i32, i32, i32, P(i32)], C.c_int),
        "slw_attention_plan": ([P(ModelCfg), i32, P(i32), i32, P(i32), P(i32), P(i64)], C.c_int),
        "slw_last_slots": ([vp, P(i32), i32, P(i32)], C.c_int),
        "slw_workspace_view": ([vp, i32, i32, i32, P(sz), P(sz)], C.c_int),
        "slw_build_cost_table": ([vp, P(i32), i32, P(i32), i32, P(ProfileOpts), P(vp)], C.c_int),
        "slw_cost_table_from_samples": ([P(i32), i32, P(i32), i32, P(i64), i32, P(vp)], C.c_int),
        "slw_cost_table_analytic": ([P(i32), i32, P(i32), i32, P(vp)], C.c_int),
        "slw_build_cost_table_ctx": ([vp, P(i32), i32, P(i32), i32, P(i32), i32, P(ProfileOpts), P(vp)], C.c_int),
        "slw_cost_table_from_samples_ctx": ([P(i32), i32, P(i32), i32, P(i32), i32, P(i64), i32, P(vp)], C.c_int),
        "slw_cost_table_prefixes": ([vp, P(i32), i32, P(i32)], C.c_int),
        "slw_cost_table_lookup_ctx": ([vp, i32, i32, i32, P(i64)], C.c_int),
        "slw_select_chunk_ctx": ([vp, P(i64), i32, i64, i32, i32, i32, i64, P(i32), P(u32), P(i32)], C.c_int),
        "slw_cost_table_free": ([vp], None),
        "slw_cost_table_dims": ([vp, P(i32), P(i32), P(i32)], C.c_int),
        "slw_cost_table_grids": ([vp, P(i32), P(i32)], C.c_int),
        "slw_cost_table_values": ([vp, i32, P(i64), sz], C.c_int),
        "slw_cost_table_lookup": ([vp, i32, i32, P(i64)], C.c_int),
        "slw_cost_table_monotone": ([vp, P(i32), P(i64)], C.c_int),
        "slw_cost_table_save": ([vp, C.c_char_p], C.c_int),
        "slw_cost_table_load": ([C.c_char_p, P(vp)], C.c_int),
        "slw_select_chunk": ([vp, P(i64), i32, i64, i32, i32, i64, P(i32), P(u32), P(i32)], C.c_int),
        "slw_set_stage_timing": ([vp, i32], C.c_int),
        "slw_stage_times": ([vp, i32, P(C.c_float), i32, P(i32)], C.c_int),
        "slw_serve": ([vp, P(RequestC), i32, P(ServeOpts), P(i64), i64, P(IterationRecord), i64, P(i64)],
                      C.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(rc: int) -> None:
    if rc != OK:
        raise SloweaveError(rc, lib().slw_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _ptr(a: np.ndarray, ct):
    return a.ctypes.data_as(C.POINTER(ct))


# ---------------------------------------------------------------------------
# Cost table and controller
# ---------------------------------------------------------------------------

class CostTable:
    """Owns a slw_cost_table*."""

    def __init__(self, handle: int):
        self._h = C.c_void_p(handle)

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.slw_cost_table_free(self._h)
            self._h = None

    @property
    def handle(self):
        return self._h

    @classmethod
    def from_samples(cls, c_grid, b_grid, samples, p_grid=None) -> "CostTable":
        """samples [nb][nc][repeats] (or [nb][nc]); with p_grid, [np][nb][nc][repeats] (or [np][nb][nc])."""
        cg, bg = _i32(c_grid), _i32(b_grid)
        s = _i64(samples)
        h = C.c_void_p()
        if p_grid is None:
            if s.ndim == 2:
                s = s[:, :, None]
            assert s.shape[:2] == (len(bg), len(cg))
            _check(lib().slw_cost_table_from_samples(_ptr(cg, C.c_int32), len(cg), _ptr(bg, C.c_int32),
                                                     len(bg), _ptr(np.ascontiguousarray(s), C.c_int64), s.shape[2],
                                                     C.byref(h)))
        else:
            pg = _i32(p_grid)
            if s.ndim == 3:
                s = s[:, :, :, None]
            assert s.shape[:3] == (len(pg), len(bg), len(cg))
            _check(lib().slw_cost_table_from_samples_ctx(_ptr(cg, C.c_int32), len(cg), _ptr(bg, C.c_int32), len(bg),
                                                         _ptr(pg, C.c_int32), len(pg),
                                                         _ptr(np.ascontiguousarray(s), C.c_int64), s.shape[3],
                                                         C.byref(h)))
        return cls(h.value)

    @classmethod
    def analytic(cls, c_grid, b_grid) -> "CostTable":
        """The simulator's analytic cost model (Sec. 4.1) at every grid point."""
        cg, bg = _i32(c_grid), _i32(b_grid)
        h = C.c_void_p()
        _check(lib().slw_cost_table_analytic(_ptr(cg, C.c_int32), len(cg), _ptr(bg, C.c_int32), len(bg),
                                             C.byref(h)))
        return cls(h.value)

    @classmethod
    def load(cls, path: str) -> "CostTable":
        h = C.c_void_p()
        _check(lib().slw_cost_table_load(path.encode(), C.byref(h)))
        return cls(h.value)

    def save(self, path: str) -> None:
        _check(lib().slw_cost_table_save(self._h, path.encode()))

    def dims(self):
        nc, nb, r = C.c_int32(), C.c_int32(), C.c_int32()
        _check(lib().slw_cost_table_dims(self._h, C.byref(nc), C.byref(nb), C.byref(r)))
        return nc.value, nb.value, r.value

    def grids(self):
        nc, nb, _ = self.dims()
        cg = np.zeros(nc, np.int32)
        bg = np.zeros(nb, np.int32)
        _check(lib().slw_cost_table_grids(self._h, _ptr(cg, C.c_int32), _ptr(bg, C.c_int32)))
        return cg, bg

    def prefixes(self):
        """Context points, or None for a table without a context axis."""
        n = C.c_int32()
        _check(lib().slw_cost_table_prefixes(self._h, None, 0, C.byref(n)))
        if n.value == 0:
            return None
        pg = np.zeros(n.value, np.int32)
        _check(lib().slw_cost_table_prefixes(self._h, _ptr(pg, C.c_int32), len(pg), C.byref(n)))
        return pg

    def values(self, which: int) -> np.ndarray:
        """A view as [nb][nc] ([nb][nc][repeats] for samples), with a leading [np] on context tables."""
        nc, nb, r = self.dims()
        shape = (nb, nc, r) if which == TABLE_SAMPLES else (nb, nc)
        pg = self.prefixes()
        if pg is not None:
            shape = (len(pg),) + shape
        out = np.zeros(shape, np.int64)
        _check(lib().slw_cost_table_values(self._h, which, _ptr(out, C.c_int64), out.size))
        return out

    def lookup(self, n: int, c: int, prefix: int = 0) -> int:
        t = C.c_int64()
        _check(lib().slw_cost_table_lookup_ctx(self._h, prefix, n, c, C.byref(t)))
        return t.value

    def monotone(self):
        v, w = C.c_int32(), C.c_int64()
        _check(lib().slw_cost_table_monotone(self._h, C.byref(v), C.byref(w)))
        return v.value, w.value


def select_chunk(table: CostTable, deadlines_ns, now_ns: int, remaining: int, c_max: int,
                 margin_ns: int = 0, prefix: int | None = None):
    """(chunk, flags, n_lookups) from slw_select_chunk (Alg. 1); with prefix, slw_select_chunk_ctx."""
    d = _i64(deadlines_ns)
    ch, fl, nl = C.c_int32(), C.c_uint32(), C.c_int32()
    if prefix is None:
        _check(lib().slw_select_chunk(table.handle, _ptr(d, C.c_int64), len(d), int(now_ns), int(remaining),
                                      int(c_max), int(margin_ns), C.byref(ch), C.byref(fl), C.byref(nl)))
    else:
        _check(lib().slw_select_chunk_ctx(table.handle, _ptr(d, C.c_int64), len(d), int(now_ns), int(prefix),
                                          int(remaining), int(c_max), int(margin_ns), C.byref(ch), C.byref(fl),
                                          C.byref(nl)))
    return ch.value, fl.value, nl.value


def fill_normal(dst: int, n: int, seed: int, mean: float, std: float, stream: int = 0) -> None:
    """Enqueue dst[i] = bf16(mean + std z_i), z the Philox4x32-10 normal stream of seed."""
    _check(lib().slw_fill_normal(dst or None, int(n), int(seed), float(mean), float(std), stream or None))


GEMM_SKINNY = 99
GEMM_NARROW = 98


def gemm_plan(m: int, n: int, k: int) -> dict:
    """The GEMM plan an iteration uses for out[m][n] = A[m][k] W^T (host only)."""
    out = np.zeros(6, np.int32)
    _check(lib().slw_gemm_plan(int(m), int(n), int(k), _ptr(out, C.c_int32)))
    return dict(zip(("cfg", "bm", "bn", "splits", "sk_workers", "dp_tiles"), (int(v) for v in out)))


ATTENTION_PLAN_FIELDS = ("decode_items", "decode_slots", "decode_max_keys", "decode_min_keys",
                         "query_tiles", "chunk_items", "chunk_slots", "chunk_whole",
                         "chunk_max_tiles", "chunk_min_tiles", "chunk_tiles")


def attention_plan(shape, context_lens, prefills=()) -> dict:
    """The attention work lists an iteration would build (host only).

    shape: a model shape (synth.ModelShape); context_lens: cached tokens of
    each decode; prefills: (prefix_len, chunk_len) per prompt."""
    cfg = ModelCfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                   shape.ffn_dim, shape.rms_eps, shape.rope_theta, 16, shape.max_pos)
    cl = _i32(context_lens)
    pp = _i32([p for p, _ in prefills])
    pc = _i32([c for _, c in prefills])
    out = np.zeros(12, np.int64)
    _check(lib().slw_attention_plan(C.byref(cfg), len(cl), _ptr(cl, C.c_int32), len(pp), _ptr(pp, C.c_int32),
                                    _ptr(pc, C.c_int32), _ptr(out, C.c_int64)))
    return dict(zip(ATTENTION_PLAN_FIELDS, (int(v) for v in out)))


def flush_cache(buf: int, nbytes: int, stream: int = 0) -> None:
    """Enqueue a read of nbytes of device memory at buf (last-level cache flush)."""
    _check(lib().slw_flush_cache(buf or None, int(nbytes), stream or None))


# ---------------------------------------------------------------------------
# Serving loop
# ---------------------------------------------------------------------------

ITERATION_DTYPE = np.dtype([("start_ns", np.int64), ("end_ns", np.int64), ("budget_ns", np.int64),
                            ("decide_ns", np.int64), ("predicted_ns", np.int64), ("prefill_id", np.int64),
                            ("chunk", np.int32), ("n_decode", np.int32), ("remaining", np.int32),
                            ("flags", np.uint32), ("rel_margin_ppm", np.int64), ("n_prefill", np.int32),
                            ("reserved", np.int32), ("resid_p99_ns", np.int64)])
assert ITERATION_DTYPE.itemsize == C.sizeof(IterationRecord)


def serve(ids, arrival_ns, prompt, output, *, policy: int, tpot_ns: int, max_decode: int,
          fixed_chunk: int = 0, c_max: int = 4096, margin_ns: int = 0, table: CostTable | None = None,
          executor: int = EXEC_ANALYTIC, ctx: "Context | None" = None, skip_idle: bool = True,
          x_in: int = 0, x_out: int = 0, max_rows: int = 0, ws: int = 0, ws_bytes: int = 0,
          stream: int = 0, iter_cap: int | None = None, residual_window: int = 0,
          exec_table: CostTable | None = None, slo_tpot_ns=None, slo_margin_ns=None, slo_ttft_ns=None,
          queue: str = "oldest", admit_ppm: int = 0, aging_ns: int = 0, aging_chunk: int = 0,
          max_prefills: int = 1, fallback_window: int = 0, log_every: int = 0):
    """slw_serve over a trace given as arrays.

    slo_tpot_ns / slo_margin_ns / slo_ttft_ns are optional per-request
    objectives (0 / -1 / 0 entries defer to the run's values).
    Returns (token_ns, iterations): token_ns is a list of int64 arrays, one per
    request in the given order (all -1 for a request refused by admission
    control); iterations is a structured array of ITERATION_DTYPE records.
    """
    n = len(ids)
    reqs = (RequestC * max(n, 1))()
    for k in range(n):
        reqs[k] = RequestC(int(ids[k]), int(arrival_ns[k]), int(prompt[k]), int(output[k]))
    slo = None
    if slo_tpot_ns is not None or slo_margin_ns is not None or slo_ttft_ns is not None:
        slo = (RequestSloC * max(n, 1))()
        for k in range(n):
            slo[k] = RequestSloC(int(slo_tpot_ns[k]) if slo_tpot_ns is not None else 0,
                                 int(slo_margin_ns[k]) if slo_margin_ns is not None else -1,
                                 int(slo_ttft_ns[k]) if slo_ttft_ns is not None else 0)
    out = np.asarray(output, dtype=np.int64)
    tok = np.zeros(max(int(out.sum()), 1), np.int64)
    cap = int(iter_cap if iter_cap is not None else 4 * (int(out.sum()) + int(np.sum(prompt))) + 16)
    its = np.zeros(max(cap, 1), ITERATION_DTYPE)
    o = ServeOpts(policy, fixed_chunk, c_max, max_decode, int(tpot_ns), int(margin_ns),
                  table.handle if table is not None else None, executor, int(skip_idle),
                  x_in or None, x_out or None, max_rows, ws or None, ws_bytes, stream or None,
                  residual_window, exec_table.handle if exec_table is not None else None,
                  C.cast(slo, C.c_void_p) if slo is not None else None, QUEUES[queue], int(admit_ppm),
                  int(aging_ns), int(aging_chunk), int(max_prefills), int(fallback_window), int(log_every))
    nit = C.c_int64()
    _check(lib().slw_serve(ctx._h if ctx is not None else None, reqs, n, C.byref(o), _ptr(tok, C.c_int64),
                           len(tok), its.ctypes.data_as(C.POINTER(IterationRecord)), len(its), C.byref(nit)))
    offs = np.concatenate([[0], np.cumsum(out)])
    return [tok[offs[k]:offs[k + 1]].copy() for k in range(n)], its[: nit.value].copy()


# ---------------------------------------------------------------------------
# Context
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Batch:
    """One iteration's batch.  Immutable: its C struct is built on first use
    and reused by every later call with the same batch.  ``prefills``
    (prefill batching) lists (sequence, prefix, chunk) triples whose rows come
    first, in that order; chunk is then their total and prefill_seq /
    prefix_len are ignored."""
    chunk: int
    prefill_seq: int
    prefix_len: int
    decode_seqs: tuple
    context_lens: tuple
    prefills: tuple | None = None

    def __post_init__(self):
        object.__setattr__(self, "decode_seqs", tuple(int(v) for v in self.decode_seqs))
        object.__setattr__(self, "context_lens", tuple(int(v) for v in self.context_lens))
        if self.prefills is not None:
            object.__setattr__(self, "prefills", tuple((int(s), int(p), int(c)) for s, p, c in self.prefills))

    @classmethod
    def batched(cls, prefills, decode_seqs=(), context_lens=()) -> "Batch":
        """A batch of several prefills (sequence, prefix, chunk) next to decodes."""
        prefills = [tuple(p) for p in prefills if p[2] > 0]
        if len(prefills) == 1:
            (s, p, c), = prefills
            return cls(c, s, p, decode_seqs, context_lens)
        return cls(sum(c for _, _, c in prefills), -1, 0, decode_seqs, context_lens, tuple(prefills))

    @property
    def prefill_list(self):
        """The (sequence, prefix, chunk) triples of the chunk rows, in row order."""
        if self.prefills is not None:
            return list(self.prefills)
        return [(self.prefill_seq, self.prefix_len, self.chunk)] if self.chunk > 0 else []

    @property
    def rows(self) -> int:
        return self.chunk + len(self.decode_seqs)

    def c_struct(self):
        c = self.__dict__.get("_c")
        if c is None:
            ds, cl = _i64(self.decode_seqs), _i32(self.context_lens)
            pre = list(self.prefills) if self.prefills is not None else []
            ps = _i64([p[0] for p in pre])
            pp = _i32([p[1] for p in pre])
            pc = _i32([p[2] for p in pre])
            c = (BatchC(self.chunk, self.prefill_seq, self.prefix_len, len(ds), _ptr(ds, C.c_int64),
                        _ptr(cl, C.c_int32), len(pre), _ptr(ps, C.c_int64), _ptr(pp, C.c_int32),
                        _ptr(pc, C.c_int32)), ds, cl, ps, pp, pc)   # the arrays keep the pointers alive
            object.__setattr__(self, "_c", c)
        return c[0]


class Context:
    """Owns a slw_ctx*.  Pointers passed in stay owned by the caller."""

    def __init__(self, n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, rms_eps,
                 rope_theta, max_pos, block_size=16):
        cfg = ModelCfg(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, rms_eps,
                       rope_theta, block_size, max_pos)
        h = C.c_void_p()
        _check(lib().slw_create(C.byref(cfg), C.byref(h)))
        self._h = h
        self.cfg = cfg

    @classmethod
    def from_shape(cls, shape) -> "Context":
        return cls(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                   shape.ffn_dim, shape.rms_eps, shape.rope_theta, shape.max_pos, shape.block_size)

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().slw_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # weights and pools
    def set_layer_weights(self, layer: int, wqkv: int, wo: int, wgu: int, wd: int, g1: int, g2: int):
        w = LayerWeightsC(wqkv, wo, wgu, wd, g1, g2)
        _check(lib().slw_set_layer_weights(self._h, layer, C.byref(w)))

    def kv_init(self, k_pool: int, v_pool: int, num_blocks: int):
        _check(lib().slw_kv_init(self._h, C.c_void_p(k_pool), C.c_void_p(v_pool), num_blocks))

    def free_blocks(self) -> int:
        n = C.c_int32()
        _check(lib().slw_kv_free_blocks(self._h, C.byref(n)))
        return n.value

    def seq_create(self, sid: int):
        _check(lib().slw_seq_create(self._h, sid))

    def seq_free(self, sid: int):
        _check(lib().slw_seq_free(self._h, sid))

    def seq_reserve(self, sid: int, new_len: int):
        _check(lib().slw_seq_reserve(self._h, sid, new_len))

    def block_table(self, sid: int) -> list:
        n = C.c_int32()
        _check(lib().slw_seq_block_table(self._h, sid, None, 0, C.byref(n)))
        out = np.zeros(max(n.value, 1), np.int32)
        _check(lib().slw_seq_block_table(self._h, sid, _ptr(out, C.c_int32), len(out), C.byref(n)))
        return out[: n.value].tolist()

    # iteration
    def workspace_size(self, max_c: int, max_b: int) -> int:
        b = C.c_size_t()
        _check(lib().slw_workspace_size(self._h, max_c, max_b, C.byref(b)))
        return b.value

    def workspace_view(self, which: int, c: int, b: int):
        off, nb = C.c_size_t(), C.c_size_t()
        _check(lib().slw_workspace_view(self._h, which, c, b, C.byref(off), C.byref(nb)))
        return off.value, nb.value

    def mixed_iteration(self, batch: Batch, x_in: int, x_out: int, ws: int, ws_bytes: int,
                        stream: int = 0):
        _check(lib().slw_mixed_iteration(self._h, C.byref(batch.c_struct()), x_in, x_out, ws, ws_bytes,
                                         stream or None))

    def mixed_iteration_static(self, batch: Batch, x_in: int, x_out: int, stream: int = 0):
        """The iteration on the library's static workspace (no allocation of any kind)."""
        _check(lib().slw_mixed_iteration_static(self._h, C.byref(batch.c_struct()), x_in, x_out, stream or None))

    def set_stage_timing(self, depth: int):
        """Record per-stage HIP events for the last `depth` iterations (0: off)."""
        _check(lib().slw_set_stage_timing(self._h, int(depth)))

    def stage_times(self, ago: int = 0) -> dict:
        """Per-stage ms of the iteration `ago` before the last (waits for it), summed over layers."""
        out = np.zeros(len(STAGES), np.float32)
        n = C.c_int32()
        _check(lib().slw_stage_times(self._h, int(ago), _ptr(out, C.c_float), len(out), C.byref(n)))
        return dict(zip(STAGES, out[: n.value].astype(float).tolist()))

    def last_slots(self) -> list:
        n = C.c_int32()
        _check(lib().slw_last_slots(self._h, None, 0, C.byref(n)))
        out = np.zeros(max(n.value, 1), np.int32)
        _check(lib().slw_last_slots(self._h, _ptr(out, C.c_int32), len(out), C.byref(n)))
        return out[: n.value].tolist()

    def build_cost_table(self, c_grid, b_grid, *, prefix_len: int, ctx_lo: int, ctx_hi: int,
                         seed: int, warmup: int, repeats: int, x_in: int, x_out: int, ws: int,
                         ws_bytes: int, flush_buf: int = 0, flush_bytes: int = 0,
                         stream: int = 0, p_grid=None) -> CostTable:
        """slw_build_cost_table; with p_grid (context points), slw_build_cost_table_ctx."""
        cg, bg = _i32(c_grid), _i32(b_grid)
        o = ProfileOpts(prefix_len, ctx_lo, ctx_hi, seed, warmup, repeats, flush_buf or None,
                        flush_bytes, x_in, x_out, ws, ws_bytes, stream or None)
        h = C.c_void_p()
        if p_grid is None:
            _check(lib().slw_build_cost_table(self._h, _ptr(cg, C.c_int32), len(cg), _ptr(bg, C.c_int32),
                                              len(bg), C.byref(o), C.byref(h)))
        else:
            pg = _i32(p_grid)
            _check(lib().slw_build_cost_table_ctx(self._h, _ptr(cg, C.c_int32), len(cg), _ptr(bg, C.c_int32),
                                                  len(bg), _ptr(pg, C.c_int32), len(pg), C.byref(o), C.byref(h)))
        return CostTable(h.value)

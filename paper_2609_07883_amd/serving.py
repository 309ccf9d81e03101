"""Request-level serving runs over slw_serve, and their metrics (Sec. 4.3).

``run`` drives one trace through the library's serving loop (the GPU
executor, or the analytic one that turns the same loop into the Sec. 4.1
simulator).  ``metrics`` turns the emitted token times into the quantities the
paper reports: P50/P99 TTFT, P99 of the within-request P99 TPOT, SLO
attainment and goodput.  Conventions: a one-token output meets any TPOT
objective; goodput divides requests meeting both objectives by the arrival
span, which is the same for every policy; throughput divides completed
requests by the makespan (first arrival to last token).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import api


def _nearest_rank(x: np.ndarray, q_num: int, q_den: int) -> int:
    """x_sorted[ceil(len(x) * q) - 1] for integer samples."""
    xs = np.sort(np.asarray(x, dtype=np.int64))
    k = len(xs)
    rank = (k * q_num + q_den - 1) // q_den
    return int(xs[max(rank, 1) - 1])


@dataclass
class RunResult:
    token_ns: list          # per request (input order): int64 array of token times
    iterations: np.ndarray  # api.ITERATION_DTYPE records


def run(trace, *, policy: str, tpot_ms: float, max_decode: int, fixed_chunk: int = 0, c_max: int = 4096,
        margin_ns: int = 0, table: api.CostTable | None = None, session=None, skip_idle: bool = True,
        residual_window: int = 0, exec_table: api.CostTable | None = None, slo_tpot_ms=None,
        slo_margin_ns=None, slo_ttft_ms=None, **variants) -> RunResult:
    """Serve `trace` (synth.RequestTrace; request ids are 0..n-1).

    session (runtime.Session) selects the GPU executor; without it the loop
    runs on exec_table's iteration times if given, else on the analytic cost
    model.  residual_window > 0 turns on the telemetry margin.  slo_* are
    optional per-request objectives; `variants` (queue, admit_ppm, aging_ns,
    aging_chunk, max_prefills) select the policy variants of api.serve.
    """
    pol = {"sloweave": api.POLICY_SLOWEAVE, "fixed": api.POLICY_FIXED}[policy]
    kw = {}
    if session is not None:
        kw = dict(executor=api.EXEC_GPU, ctx=session.ctx, skip_idle=skip_idle,
                  x_in=session.x_in.data_ptr(), x_out=session.x_out.data_ptr(),
                  max_rows=session.x_in.shape[0], ws=session.ws.data_ptr(), ws_bytes=session.ws_bytes,
                  stream=session.stream())
    elif exec_table is not None:
        kw = dict(executor=api.EXEC_TABLE, exec_table=exec_table)
    n = len(trace)
    tok, its = api.serve(np.arange(n), trace.arrival_ns, trace.prompt, trace.output, policy=pol,
                         tpot_ns=int(round(tpot_ms * 1e6)), max_decode=max_decode, fixed_chunk=fixed_chunk,
                         c_max=c_max, margin_ns=margin_ns, table=table, residual_window=residual_window,
                         slo_tpot_ns=None if slo_tpot_ms is None else np.rint(np.asarray(slo_tpot_ms) * 1e6),
                         slo_margin_ns=slo_margin_ns,
                         slo_ttft_ns=None if slo_ttft_ms is None else np.rint(np.asarray(slo_ttft_ms) * 1e6),
                         **variants, **kw)
    return RunResult(tok, its)


def metrics(trace, token_ns, ttft_slo_ms, tpot_slo_ms) -> dict:
    """Sec. 4.3 request-level results of one run (times in ms, rates per second).

    The objectives may be scalars or per-request arrays (Sec. 3.5).  Requests
    refused by admission control (token times -1) count as missed and stay
    out of the latency percentiles.
    """
    arrival_all = np.asarray(trace.arrival_ns, dtype=np.int64)
    served = np.array([len(t) > 0 and t[0] >= 0 for t in token_ns], dtype=bool)
    ttft_slo = np.rint(np.broadcast_to(np.asarray(ttft_slo_ms, dtype=np.float64), served.shape) * 1e6)[served]
    tpot_slo = np.rint(np.broadcast_to(np.asarray(tpot_slo_ms, dtype=np.float64), served.shape) * 1e6)[served]
    kept = [t for t, s in zip(token_ns, served) if s]
    arrival = arrival_all[served]
    first = np.array([t[0] for t in kept], dtype=np.int64)
    last = np.array([t[-1] for t in kept], dtype=np.int64)
    ttft = first - arrival
    tpot = np.array([_nearest_rank(np.diff(t), 99, 100) if len(t) > 1 else 0 for t in kept], dtype=np.int64)
    meets = (ttft <= ttft_slo) & (tpot <= tpot_slo)
    span = int(arrival_all.max() - arrival_all.min())
    makespan = int(last.max() - arrival_all.min()) if len(kept) else 0
    n = len(arrival_all)
    out_tokens = int(sum(len(t) for t in kept))
    ttft_missed, tpot_missed = int(np.sum(ttft > ttft_slo)), int(np.sum(tpot > tpot_slo))
    if not len(kept):  # percentiles of an empty run read 0
        ttft = tpot = np.zeros(1, np.int64)
    return {
        "requests": n,
        "rejected": int(n - served.sum()),
        "met": int(meets.sum()),
        "ttft_missed": ttft_missed,
        "tpot_missed": tpot_missed,
        "slo_attainment": float(meets.sum()) / n,
        "goodput_req_s": float(meets.sum()) / span * 1e9 if span > 0 else float("nan"),
        "throughput_req_s": len(kept) / makespan * 1e9 if makespan > 0 else 0.0,
        "output_tokens_s": out_tokens / makespan * 1e9 if makespan > 0 else 0.0,
        "p50_ttft_ms": _nearest_rank(ttft, 1, 2) / 1e6,
        "p99_ttft_ms": _nearest_rank(ttft, 99, 100) / 1e6,
        "p99_tpot_ms": _nearest_rank(tpot, 99, 100) / 1e6,
        "arrival_span_ns": span,
        "makespan_ns": makespan,
    }

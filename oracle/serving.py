"""Oracle for request-level serving: the iteration-level simulator and its metrics.

Test infrastructure only (see ``oracle/__init__``).

* ``simulate``: the event-driven iteration-level loop of Sec. 4.1 under the
  deadline model of Sec. 3.1.  Every iteration decodes one token for each
  active request and optionally runs one prefill chunk of the oldest pending
  request (oldest-first queueing shared by every policy, Sec. 4.3); requests
  that arrive while an iteration runs become eligible when it ends.  The
  chunk is Alg. 1 over a cost predictor (SLOWeave) or a fixed size.
* ``request_metrics`` / ``summarize``: TTFT, within-request P99 TPOT, SLO
  attainment and goodput of Sec. 4.3.

Times are integer nanoseconds throughout, so two implementations of the
same loop agree exactly.

Readings (the paper is silent or ambiguous here):
* the first output token is emitted at the end of the iteration that
  completes the prompt, and that end is l_i, the request's first token time
  (Sec. 3.1 sets l_i to the prefill completion time);
* a request's decode iterations start with the iteration after its prefill
  completes; a request whose output is one token finishes with its prefill;
* within-request TPOT is the nearest-rank P99 of the gaps between
  consecutive output tokens; a one-token output has no gap and meets any
  TPOT objective;
* the trace duration that divides goodput is the arrival span (first to last
  arrival), the same for every policy; throughput divides completed requests
  by the makespan (first arrival to last completion);
* with a cap on the decode batch, a pending request may run prefill only
  while fewer than that many requests decode (the prefill in flight is the
  only way the decode set grows, so the cap holds at all times);
* a decode set larger than the cost table's last decode-batch point cannot
  be priced: the iteration is decode-only;
* the telemetry margin (Sec. 3.3 proposes a margin taken from a high
  percentile of observed prediction errors; Sec. 5.1 feeds observed
  durations back to the controller) is relative:
  every iteration that ran a chunk leaves the residual
  floor((observed - predicted) * 1e6 / predicted) in parts per million, the
  last W of them form the window, and a decision adds
  ceil(q * T_hat(n, c) / 1e6) to every prediction it tests, q being the
  nearest-rank P99 of the window clamped to [0, 1e8] (0 while the window is
  empty).
"""
from __future__ import annotations

from dataclasses import dataclass, field

from .schedule import nearest_rank, select_chunk


@dataclass(frozen=True)
class Request:
    rid: int
    arrival_ns: int
    prompt: int      # prompt tokens (>= 1)
    output: int      # output tokens (>= 1), the first one emitted by the prefill


@dataclass
class Iteration:
    start_ns: int
    end_ns: int
    chunk: int
    n_decode: int
    prefill_rid: int     # -1 when the iteration runs no chunk
    budget_ns: int       # earliest deadline minus start (0 with no active decode)
    rel_margin_ppm: int = 0  # telemetry margin used by the decision


@dataclass
class Trace:
    token_ns: dict = field(default_factory=dict)    # rid -> [completion time of each output token]
    iterations: list = field(default_factory=list)


def simulate(requests, *, cost_ns, tpot_ns: int, policy: str = "sloweave", fixed_chunk: int = 0,
             predict=None, c_last: int | None = None, c_max: int = 4096, margin_ns: int = 0,
             max_decode: int | None = None, residual_window: int = 0, prefix_aware: bool = False,
             max_iterations: int = 10_000_000) -> Trace:
    """Run the trace through the iteration-level loop of Sec. 4.1.

    cost_ns(n, c) -> ns is how long an iteration with n decodes and a chunk
    of c tokens takes (the simulator's cost model); predict(n, c) -> ns is
    what the SLOWeave controller believes (defaults to cost_ns) and c_last
    the largest chunk it can price.  policy is "sloweave" (Alg. 1 with margin
    margin_ns and cap c_max) or "fixed" (chunks of fixed_chunk tokens).
    residual_window > 0 turns on the telemetry margin (module docstring).
    With prefix_aware, cost_ns and predict take a third argument, the cached
    prefix the iteration is priced at: that of the oldest eligible prompt
    (its tokens already processed), 0 with none.
    """
    if policy not in ("sloweave", "fixed"):
        raise ValueError(policy)
    if policy == "fixed" and fixed_chunk <= 0:
        raise ValueError("fixed_chunk must be positive")
    predict = predict or cost_ns

    def at(f, n, c, p):
        return f(n, c, p) if prefix_aware else f(n, c)
    reqs = sorted(requests, key=lambda r: (r.arrival_ns, r.rid))
    out = Trace(token_ns={r.rid: [] for r in reqs})
    pending = []            # eligible requests whose prompt is not finished, oldest first
    done_prompt = {}        # rid -> prompt tokens already processed
    active = {}             # rid -> (request, time of its latest token l_i)
    t = reqs[0].arrival_ns if reqs else 0
    nxt = 0
    finished = 0
    residuals = []          # relative residuals (ppm) of chunked iterations, oldest first
    for _ in range(max_iterations):
        if finished == len(reqs):
            return out
        while nxt < len(reqs) and reqs[nxt].arrival_ns <= t:
            pending.append(reqs[nxt])
            done_prompt[reqs[nxt].rid] = 0
            nxt += 1
        if not pending and not active:
            t = reqs[nxt].arrival_ns           # idle until the next arrival
            continue
        order = sorted(active)                 # decode rows in request-id order
        deadlines = [active[r][1] + tpot_ns for r in order]
        n = len(order)
        head = pending[0] if pending and (max_decode is None or n < max_decode) else None
        remaining = head.prompt - done_prompt[head.rid] if head else 0
        budget = min(deadlines) - t if deadlines else 0
        prefix = done_prompt[head.rid] if head else 0
        rel = 0
        if head is None:
            chunk = 0
        elif policy == "fixed":
            chunk = min(fixed_chunk, remaining)
        else:
            if residual_window > 0 and residuals:
                rel = min(max(nearest_rank(residuals[-residual_window:], 99, 100), 0), 10**8)

            def with_margin(nn, cc, q=rel, p=prefix):
                v = at(predict, nn, cc, p)
                return v + -(-q * v // 10**6)   # T_hat + ceil(q T_hat / 1e6)
            try:
                chunk = select_chunk(with_margin, deadlines, t, remaining, c_max, margin_ns, c_last=c_last)[0]
            except IndexError:                 # n above the priced decode batches
                chunk = 0
        end = t + at(cost_ns, n, chunk, prefix)
        out.iterations.append(Iteration(t, end, chunk, n, head.rid if chunk > 0 else -1, budget, rel))
        if residual_window > 0 and chunk > 0:
            pred = at(predict, n, chunk, prefix)
            if pred > 0:
                residuals.append((end - t - pred) * 10**6 // pred)
        for rid in order:
            req, _ = active[rid]
            out.token_ns[rid].append(end)
            if len(out.token_ns[rid]) == req.output:
                del active[rid]
                finished += 1
            else:
                active[rid] = (req, end)
        if chunk > 0:
            done_prompt[head.rid] += chunk
            if done_prompt[head.rid] == head.prompt:
                pending.pop(0)
                out.token_ns[head.rid].append(end)     # first output token
                if head.output == 1:
                    finished += 1
                else:
                    active[head.rid] = (head, end)
        t = end
    raise RuntimeError("iteration limit reached")


@dataclass(frozen=True)
class RequestMetrics:
    rid: int
    ttft_ns: int
    tpot_p99_ns: int
    finish_ns: int
    meets: bool


def request_metrics(req: Request, token_ns, ttft_slo_ns: int, tpot_slo_ns: int) -> RequestMetrics:
    """Sec. 4.3: TTFT and within-request P99 TPOT, and whether both meet their SLOs."""
    if len(token_ns) != req.output:
        raise ValueError(f"request {req.rid}: {len(token_ns)} tokens, expected {req.output}")
    ttft = token_ns[0] - req.arrival_ns
    gaps = [b - a for a, b in zip(token_ns, token_ns[1:])]
    tpot = nearest_rank(gaps, 99, 100) if gaps else 0
    return RequestMetrics(req.rid, ttft, tpot, token_ns[-1], ttft <= ttft_slo_ns and tpot <= tpot_slo_ns)


def summarize(requests, token_ns: dict, ttft_slo_ns: int, tpot_slo_ns: int) -> dict:
    """Request-level results of one run (Sec. 4.3), integer ns and exact ratios.

    goodput_num / goodput_den_ns is requests meeting both SLOs per
    nanosecond of arrival span.
    """
    reqs = sorted(requests, key=lambda r: (r.arrival_ns, r.rid))
    ms = [request_metrics(r, token_ns[r.rid], ttft_slo_ns, tpot_slo_ns) for r in reqs]
    span = reqs[-1].arrival_ns - reqs[0].arrival_ns
    if span <= 0:
        raise ValueError("the arrival span must be positive")
    makespan = max(m.finish_ns for m in ms) - reqs[0].arrival_ns
    met = sum(m.meets for m in ms)
    return {
        "requests": len(ms),
        "met": met,
        "goodput_num": met,
        "goodput_den_ns": span,
        "makespan_ns": makespan,
        "p50_ttft_ns": nearest_rank([m.ttft_ns for m in ms], 1, 2),
        "p99_ttft_ns": nearest_rank([m.ttft_ns for m in ms], 99, 100),
        "p99_tpot_ns": nearest_rank([m.tpot_p99_ns for m in ms], 99, 100),
        "output_tokens": sum(r.output for r in reqs),
        "prompt_tokens": sum(r.prompt for r in reqs),
    }

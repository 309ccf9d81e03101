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
* The policy variants of Sec. 3.3-3.5 (per-request objectives and class
  margins, queue disciplines, admission control, aging, first-fit prefill
  batching) are options of ``simulate``; its docstring states the reading
  of each.  Pinned by brute-force replay and closed-form cases in the tests
  of the policy variants.

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
  empty);
* the telemetry fallback (Sec. 5.1: the scheduler may fall back to
  decode-only execution when telemetry residuals exceed the configured
  margin; Table 1: telemetry records predicted and observed durations and
  fallback events) compares absolute residuals with the margin delta: every
  iteration the predictor prices leaves observed - predicted in ns, the last
  F of them form the fallback window, and while the window's nearest-rank
  P99 exceeds delta a SLOWeave decision that has a prompt to serve and
  active decodes to protect runs no chunk and is recorded as a fallback
  event (no fallback while the window is empty; with no active decode there
  is no deadline to protect and Alg. 1 runs as usual).  Decode-only
  iterations keep filling the window, so chunks return once the observed
  residuals are back within delta.
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
    tpot_ns: int = 0     # D_i (Sec. 3.5); 0: the run's D
    margin_ns: int = -1  # the request class's margin delta_i (Sec. 3.5); < 0: the run's delta
    ttft_ns: int = 0     # TTFT objective used by earliest-deadline queueing; 0: none


@dataclass
class Iteration:
    start_ns: int
    end_ns: int
    chunk: int           # prefill tokens run (over every prompt of the iteration)
    n_decode: int
    prefill_rid: int     # first prompt served, -1 when the iteration runs no chunk
    budget_ns: int       # earliest deadline minus start (0 with no active decode)
    rel_margin_ppm: int = 0  # telemetry margin used by the decision
    n_prefill: int = 0   # prompts served
    aged: bool = False   # the chunk was forced by the aging threshold
    fallback: bool = False   # decode-only because the residual P99 exceeded the margin
    resid_p99_ns: int = 0    # fallback window's P99 tested by the decision


@dataclass
class Trace:
    token_ns: dict = field(default_factory=dict)    # rid -> [completion time of each output token]
    iterations: list = field(default_factory=list)
    rejected: set = field(default_factory=set)      # rids refused by admission control


QUEUES = ("oldest", "srpt", "edf")


def _queue_key(queue, r: Request, remaining: int):
    """Sec. 3.4: the order in which pending prompts are served.  Ties go to
    the older request (arrival, then id)."""
    if queue == "srpt":             # shortest remaining prefill first
        return (remaining, r.arrival_ns, r.rid)
    if queue == "edf":              # earliest TTFT deadline first (none: last)
        return (r.arrival_ns + r.ttft_ns if r.ttft_ns > 0 else float("inf"), r.arrival_ns, r.rid)
    return (r.arrival_ns, r.rid)    # oldest first


def simulate(requests, *, cost_ns, tpot_ns: int, policy: str = "sloweave", fixed_chunk: int = 0,
             predict=None, c_last: int | None = None, c_max: int = 4096, margin_ns: int = 0,
             max_decode: int | None = None, residual_window: int = 0, prefix_aware: bool = False,
             queue: str = "oldest", admit_ppm: int = 0, aging_ns: int = 0, aging_chunk: int = 0,
             max_prefills: int = 1, fallback_window: int = 0, max_iterations: int = 10_000_000) -> Trace:
    """Run the trace through the iteration-level loop of Sec. 4.1.

    cost_ns(n, c) -> ns is how long an iteration with n decodes and c
    prefill tokens takes (the simulator's cost model); predict(n, c) -> ns is
    what the SLOWeave controller believes (defaults to cost_ns) and c_last
    the largest chunk it can price.  policy is "sloweave" (Alg. 1 with margin
    margin_ns and cap c_max) or "fixed" (chunks of fixed_chunk tokens).
    residual_window > 0 turns on the telemetry margin and fallback_window > 0
    the telemetry fallback (module docstring).
    With prefix_aware, cost_ns and predict take a third argument, the cached
    prefix the iteration is priced at: that of the first prompt it serves
    (its tokens already processed), 0 with none.

    Policy variants (Sec. 3.3-3.5; the paper gives no parameters, these are
    the readings this loop implements):
    * per-request objectives: request i's next-token deadline is
      l_i + D_i and its class margin delta_i; a chunk is admissible when
      T_hat + delta_i <= d_i - s_t for every active i, i.e. Alg. 1 runs on the
      deadlines d_i - (delta_i - margin_ns) with margin margin_ns;
    * queue: the pending prompt served first ("oldest", "srpt": fewest
      remaining prompt tokens, "edf": earliest arrival + TTFT objective);
    * admission control (admit_ppm > 0): a request that becomes eligible is
      refused when T_hat(n, 0) + delta_i > D_i * admit_ppm / 1e6, n counting
      the active decodes, the admitted pending prompts and itself (also
      refused when n is beyond the predictor); refused requests emit no
      token;
    * aging (aging_ns > 0, SLOWeave only): when Alg. 1 gives no chunk to a
      head that may run and that has waited aging_ns since it became eligible
      or last ran, min(aging_chunk, remaining, c_max) tokens run anyway;
    * prefill batching (max_prefills > 1, SLOWeave only): first fit.  When
      the head's chunk finishes its prompt, the next pending prompts in queue
      order join while the decode cap allows (counting the prompts that
      finish earlier in the iteration), each with the largest chunk c for
      which T_hat(n, S + c) still meets the budget, S being the tokens
      already placed (Alg. 1's search with the predictor shifted by S, caps
      c_max - S and c_last - S); a prompt that does not finish ends the list.
    """
    if policy not in ("sloweave", "fixed"):
        raise ValueError(policy)
    if policy == "fixed" and fixed_chunk <= 0:
        raise ValueError("fixed_chunk must be positive")
    if queue not in QUEUES:
        raise ValueError(queue)
    predict = predict or cost_ns

    def at(f, n, c, p):
        return f(n, c, p) if prefix_aware else f(n, c)
    reqs = sorted(requests, key=lambda r: (r.arrival_ns, r.rid))
    D = {r.rid: r.tpot_ns if r.tpot_ns > 0 else tpot_ns for r in reqs}
    delta = {r.rid: r.margin_ns if r.margin_ns >= 0 else margin_ns for r in reqs}
    out = Trace(token_ns={r.rid: [] for r in reqs})
    pending = []            # eligible requests whose prompt is not finished
    done_prompt = {}        # rid -> prompt tokens already processed
    waited = {}             # rid -> time it became eligible or last ran a chunk
    active = {}             # rid -> (request, time of its latest token l_i)
    t = reqs[0].arrival_ns if reqs else 0
    nxt = 0
    finished = 0
    residuals = []          # relative residuals (ppm) of chunked iterations, oldest first
    fb_resid = []           # absolute residuals (ns) of priced iterations, oldest first
    for _ in range(max_iterations):
        if finished == len(reqs):
            return out
        while nxt < len(reqs) and reqs[nxt].arrival_ns <= t:
            r = reqs[nxt]
            nxt += 1
            if admit_ppm > 0:
                n_future = len(active) + len(pending) + 1
                try:
                    cost = at(predict, n_future, 0, 0)
                except IndexError:                 # beyond the priced decode batches
                    cost = None
                if cost is None or (cost + delta[r.rid]) * 10**6 > D[r.rid] * admit_ppm:
                    out.rejected.add(r.rid)
                    finished += 1
                    continue
            pending.append(r)
            done_prompt[r.rid] = 0
            waited[r.rid] = t
        if finished == len(reqs):
            return out
        if not pending and not active:
            t = reqs[nxt].arrival_ns           # idle until the next arrival
            continue
        order = sorted(active)                 # decode rows in request-id order
        deadlines = [active[r][1] + D[r] for r in order]
        eff = [active[r][1] + D[r] - (delta[r] - margin_ns) for r in order]
        n = len(order)
        queue_order = sorted(pending, key=lambda r: _queue_key(queue, r, r.prompt - done_prompt[r.rid]))
        head = queue_order[0] if queue_order and (max_decode is None or n < max_decode) else None
        remaining = head.prompt - done_prompt[head.rid] if head else 0
        budget = min(deadlines) - t if deadlines else 0
        prefix = done_prompt[head.rid] if head else 0
        rel = 0
        aged = False
        fallback = False
        fb_p99 = 0
        plan = []                              # (request, tokens) served this iteration
        if head is None:
            chunk = 0
        elif policy == "fixed":
            chunk = min(fixed_chunk, remaining)
        else:
            if residual_window > 0 and residuals:
                rel = min(max(nearest_rank(residuals[-residual_window:], 99, 100), 0), 10**8)
            if fallback_window > 0 and fb_resid and n > 0:
                fb_p99 = nearest_rank(fb_resid[-fallback_window:], 99, 100)
                fallback = fb_p99 > margin_ns

            def with_margin(nn, cc, q=rel, p=prefix):
                v = at(predict, nn, cc, p)
                return v + -(-q * v // 10**6)   # T_hat + ceil(q T_hat / 1e6)
            if fallback:
                chunk = 0
            else:
                try:
                    chunk = select_chunk(with_margin, eff, t, remaining, c_max, margin_ns, c_last=c_last)[0]
                except IndexError:             # n above the priced decode batches
                    chunk = 0
            if chunk == 0 and aging_ns > 0 and t - waited[head.rid] >= aging_ns:
                chunk = min(aging_chunk, remaining, c_max)
                aged = True
        if chunk > 0:
            plan.append((head, chunk))
        if policy == "sloweave" and max_prefills > 1 and chunk == remaining and chunk > 0 and not aged:
            total = chunk
            for r in queue_order[1:]:
                if len(plan) >= max_prefills:
                    break
                if max_decode is not None and n + len(plan) >= max_decode:
                    break
                rem = r.prompt - done_prompt[r.rid]

                def shifted(nn, cc, base=total, q=rel, p=prefix):
                    v = at(predict, nn, base + cc, p)
                    return v + -(-q * v // 10**6)
                try:
                    c = select_chunk(shifted, eff, t, rem, c_max - total, margin_ns,
                                     c_last=None if c_last is None else c_last - total)[0]
                except IndexError:
                    c = 0
                if c <= 0:
                    break
                plan.append((r, c))
                total += c
                if c < rem:
                    break
            chunk = total
        end = t + at(cost_ns, n, chunk, prefix)
        out.iterations.append(Iteration(t, end, chunk, n, head.rid if chunk > 0 else -1, budget, rel,
                                        len(plan), aged, fallback, fb_p99))
        if residual_window > 0 and chunk > 0:
            try:
                pred = at(predict, n, chunk, prefix)
            except IndexError:                 # an aged chunk beside unpriced decodes
                pred = 0
            if pred > 0:
                residuals.append((end - t - pred) * 10**6 // pred)
        if fallback_window > 0:
            try:
                pred = at(predict, n, chunk, prefix)
            except IndexError:                 # not priced: no residual
                pred = 0
            if pred > 0:
                fb_resid.append(end - t - pred)
        for rid in order:
            req, _ = active[rid]
            out.token_ns[rid].append(end)
            if len(out.token_ns[rid]) == req.output:
                del active[rid]
                finished += 1
            else:
                active[rid] = (req, end)
        for r, c in plan:
            done_prompt[r.rid] += c
            waited[r.rid] = end
            if done_prompt[r.rid] == r.prompt:
                pending.remove(r)
                out.token_ns[r.rid].append(end)     # first output token
                if r.output == 1:
                    finished += 1
                else:
                    active[r.rid] = (r, end)
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


def summarize(requests, token_ns: dict, ttft_slo_ns: int, tpot_slo_ns: int, rejected=()) -> dict:
    """Request-level results of one run (Sec. 4.3), integer ns and exact ratios.

    goodput_num / goodput_den_ns is requests meeting both SLOs per
    nanosecond of arrival span.  Requests refused by admission control
    count as missed and are left out of the latency percentiles.
    """
    reqs = sorted(requests, key=lambda r: (r.arrival_ns, r.rid))
    rejected = set(rejected)
    ms = [request_metrics(r, token_ns[r.rid], ttft_slo_ns, tpot_slo_ns) for r in reqs if r.rid not in rejected]
    span = reqs[-1].arrival_ns - reqs[0].arrival_ns
    if span <= 0:
        raise ValueError("the arrival span must be positive")
    makespan = max(m.finish_ns for m in ms) - reqs[0].arrival_ns if ms else 0
    met = sum(m.meets for m in ms)
    return {
        "requests": len(reqs),
        "rejected": len(rejected),
        "met": met,
        "goodput_num": met,
        "goodput_den_ns": span,
        "makespan_ns": makespan,
        "p50_ttft_ns": nearest_rank([m.ttft_ns for m in ms], 1, 2) if ms else 0,
        "p99_ttft_ns": nearest_rank([m.ttft_ns for m in ms], 99, 100) if ms else 0,
        "p99_tpot_ns": nearest_rank([m.tpot_p99_ns for m in ms], 99, 100) if ms else 0,
        "output_tokens": sum(r.output for r in reqs if r.rid not in rejected),
        "prompt_tokens": sum(r.prompt for r in reqs if r.rid not in rejected),
    }

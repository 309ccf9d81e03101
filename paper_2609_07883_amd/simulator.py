"""The Sec. 4 simulator study on the library's serving loop.

The loop in the library (slw_serve) runs on the analytic cost model of
Sec. 4.1 (the simulator's executor), so the simulator is the same scheduler
as the GPU runtime, not a second program.  This module sweeps the four
workloads of Sec. 4.2 (``synth.SIM_WORKLOADS``: 1,000 requests per run, five
seeds) over the TPOT objectives and the policies of Sec. 4.3 (full-prompt
prefill, fixed chunks of 64, 256 and 1,024, SLOWeave with C_max 4,096) and
reports the mean over seeds of P99 TTFT, P99 request-level TPOT, SLO
attainment and goodput, the layout of the paper's Table 3 and Table 4.

SLOWeave prices iterations with a table of the same analytic model on a
dense grid (every decode batch up to 2,048, chunks every 16 tokens up to
C_max, interpolated exactly since the model is linear in c), so its
predictions equal the executor's costs, as in the paper's simulator.

Run as ``python -m paper_2609_07883_amd.simulator [--requests N] [--seeds K]``;
``--classes`` runs the two-class study of Sec. 3.5 (``classes_study``) instead.
"""
from __future__ import annotations

import argparse
import json
import time

import numpy as np

from . import api, serving, synth

C_MAX = 4096
MAX_DECODE = 2048
TPOTS_MS = (10.0, 25.0, 50.0)
POLICIES = (("Full", "fixed", 1 << 30), ("Fixed-64", "fixed", 64), ("Fixed-256", "fixed", 256),
            ("Fixed-1024", "fixed", 1024), ("SLOWeave", "sloweave", 0))
# Sec. 3.3 prefill batching by first fit (up to four prompts per iteration)
BATCHING_POLICY = ("SLOWeave + first-fit batching", "sloweave", 0, {"max_prefills": 4})


def analytic_table() -> api.CostTable:
    """The analytic model on a dense grid (exact under the table's lookups)."""
    return api.CostTable.analytic(list(range(0, C_MAX + 1, 16)), list(range(0, MAX_DECODE + 1)))


def run_one(trace, table, policy: str, chunk: int, tpot_ms: float, ttft_slo_ms: float, **variants) -> dict:
    res = serving.run(trace, policy=policy, fixed_chunk=chunk, tpot_ms=tpot_ms, max_decode=MAX_DECODE,
                      c_max=C_MAX, table=table if policy == "sloweave" else None, **variants)
    return serving.metrics(trace, res.token_ns, ttft_slo_ms=ttft_slo_ms, tpot_slo_ms=tpot_ms)


def study(workloads=tuple(synth.SIM_WORKLOADS), tpots=TPOTS_MS, policies=POLICIES, n: int = 1000,
          seeds=(0, 1, 2, 3, 4), table: api.CostTable | None = None) -> list[dict]:
    """Mean over seeds of each (workload, TPOT objective, policy)."""
    table = table or analytic_table()
    rows = []
    for wname in workloads:
        w = synth.SIM_WORKLOADS[wname]
        traces = [synth.sim_trace(wname, n, s) for s in seeds]
        for tpot in tpots:
            for pname, pol, chunk, *opt in policies:
                kw = opt[0] if opt else {}
                ms = [run_one(tr, table, pol, chunk, tpot, w.ttft_slo_ms, **kw) for tr in traces]
                rows.append({"workload": wname, "tpot_slo_ms": tpot, "ttft_slo_ms": w.ttft_slo_ms,
                             "policy": pname,
                             "p99_ttft_ms": float(np.mean([m["p99_ttft_ms"] for m in ms])),
                             "p99_tpot_ms": float(np.mean([m["p99_tpot_ms"] for m in ms])),
                             "slo_attainment": float(np.mean([m["slo_attainment"] for m in ms])),
                             "goodput_req_s": float(np.mean([m["goodput_req_s"] for m in ms])),
                             "throughput_req_s": float(np.mean([m["throughput_req_s"] for m in ms]))})
    return rows


def gains(rows: list[dict]) -> dict:
    """SLOWeave goodput over the best non-SLOWeave policy, per (workload, TPOT)."""
    out = {}
    for r in rows:
        if r["policy"] != "SLOWeave":
            continue
        others = [o for o in rows if o["workload"] == r["workload"] and o["tpot_slo_ms"] == r["tpot_slo_ms"]
                  and not o["policy"].startswith("SLOWeave")]
        best = max(others, key=lambda o: o["goodput_req_s"])
        out[f'{r["workload"]} {r["tpot_slo_ms"]:g}ms'] = {
            "vs": best["policy"],
            "ratio": round(r["goodput_req_s"] / best["goodput_req_s"], 3) if best["goodput_req_s"] > 0 else None}
    return out


CLASS_POLICIES = (("SLOWeave per-request D", "sloweave", 0, "classes"),
                  ("SLOWeave D = 10 ms for all", "sloweave", 0, 10.0),
                  ("SLOWeave D = 50 ms for all", "sloweave", 0, 50.0),
                  ("Fixed-256", "fixed", 256, "classes"), ("Fixed-1024", "fixed", 1024, "classes"))


def _subset(trace, idx):
    return synth.RequestTrace(trace.arrival_ns[idx], trace.prompt[idx], trace.output[idx])


def classes_study(workload: str = "mixed", n: int = 1000, seeds=(0, 1, 2, 3, 4), interactive: float = 0.5,
                  d_ms=(10.0, 50.0), rate_scale: float = 1.0, table: api.CostTable | None = None,
                  policies=CLASS_POLICIES) -> list[dict]:
    """Sec. 3.5 on the simulator: a fraction `interactive` of the requests
    (a seeded coin per request) carries the tight objective d_ms[0], the
    others d_ms[1].  The controller either sees each request's own D (its
    budget is the earliest of the active requests' deadlines) or one D for
    all; each class is scored against its own objective."""
    table = table or analytic_table()
    w = synth.SIM_WORKLOADS[workload]
    rows = []
    for pname, pol, chunk, ctl in policies:
        acc = {"interactive": [], "batch": [], "all": []}
        for seed in seeds:
            tr = synth.sim_trace(workload, n, seed, rate_scale)
            inter = np.random.default_rng(10_000 + seed).random(len(tr)) < interactive
            d = np.where(inter, d_ms[0], d_ms[1])
            kw = dict(slo_tpot_ms=d, tpot_ms=d_ms[1]) if ctl == "classes" else dict(tpot_ms=float(ctl))
            res = serving.run(tr, policy=pol, fixed_chunk=chunk, max_decode=MAX_DECODE, c_max=C_MAX,
                              table=table if pol == "sloweave" else None, **kw)
            acc["all"].append(serving.metrics(tr, res.token_ns, w.ttft_slo_ms, d))
            for cname, mask in (("interactive", inter), ("batch", ~inter)):
                idx = np.nonzero(mask)[0]
                acc[cname].append(serving.metrics(_subset(tr, idx), [res.token_ns[i] for i in idx],
                                                  w.ttft_slo_ms, d[idx]))
        row = {"workload": workload, "policy": pname}
        for cname, ms in acc.items():
            row[f"{cname}_slo_attainment"] = float(np.mean([m["slo_attainment"] for m in ms]))
            row[f"{cname}_p99_ttft_ms"] = float(np.mean([m["p99_ttft_ms"] for m in ms]))
        row["goodput_req_s"] = float(np.mean([m["goodput_req_s"] for m in acc["all"]]))
        rows.append(row)
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--requests", type=int, default=1000)
    ap.add_argument("--seeds", type=int, default=5)
    ap.add_argument("--classes", action="store_true", help="the two-class study of Sec. 3.5 instead")
    ap.add_argument("--interactive", type=float, default=0.03, help="share of 10 ms requests (--classes)")
    ap.add_argument("--batching", action="store_true",
                    help="add SLOWeave with first-fit prefill batching (Sec. 3.3) to the study")
    args = ap.parse_args(argv)
    t0 = time.time()
    if args.classes:
        rows = classes_study(n=args.requests, seeds=tuple(range(args.seeds)), interactive=args.interactive)
        for r in rows:
            print(f'{r["policy"]:28s} SLO interactive {100 * r["interactive_slo_attainment"]:5.1f}%  '
                  f'batch {100 * r["batch_slo_attainment"]:5.1f}%  all {100 * r["all_slo_attainment"]:5.1f}%  '
                  f'P99 TTFT {r["all_p99_ttft_ms"]:8.1f} ms  goodput {r["goodput_req_s"]:6.1f} req/s')
        print(json.dumps({"rows": rows, "requests": args.requests, "seeds": args.seeds,
                          "interactive": args.interactive, "wall_s": round(time.time() - t0, 1)}))
        return
    rows = study(n=args.requests, seeds=tuple(range(args.seeds)),
                 policies=POLICIES + ((BATCHING_POLICY,) if args.batching else ()))
    for r in rows:
        print(f'{r["workload"]:7s} TPOT {r["tpot_slo_ms"]:4.0f} ms  {r["policy"]:10s}  '
              f'P99 TTFT {r["p99_ttft_ms"]:8.1f} ms  P99 TPOT {r["p99_tpot_ms"]:6.1f} ms  '
              f'SLO {100 * r["slo_attainment"]:5.1f}%  goodput {r["goodput_req_s"]:6.1f} req/s')
    print(json.dumps({"rows": rows, "sloweave_vs_best_other": gains(rows), "requests": args.requests,
                      "seeds": args.seeds, "wall_s": round(time.time() - t0, 1)}))


if __name__ == "__main__":
    main()

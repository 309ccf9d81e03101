"""Reference oracle for the SLOWeave mixed iteration (arXiv 2609.07883).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code,
headers, tables or constants with the HIP library; the two meet only through
the seeded input generators, which hold none of the method's arithmetic.

Contents
--------
``layer``    The decoder layer a mixed iteration runs (pre-norm RMSNorm, GQA
             attention with rotate-half RoPE over each sequence's cached keys,
             SwiGLU MLP), written as its textbook definition in float64 over
             dense per-sequence K/V.  The paper leaves the model untouched
             (Sec. 1; Sec. 5.1), so chunking and paging change the schedule,
             never the arithmetic: the oracle therefore computes the plain
             unchunked, unpaged result.
``paging``   The paged-KV block manager of Table 1 ("KV manager"): lowest
             free block first, block tables and slot mapping.
``schedule`` Eq. 1 and Alg. 1 (chunk selection), the profiler's P50/P99
             table with a cumulative maximum along the chunk axis
             (Sec. 5.1) and its lookup between grid points (Sec. 6.4), and
             the simulator's analytic cost model (Sec. 4.1).
``serving``  The iteration-level serving loop of Sec. 4.1 under the deadline
             model of Sec. 3.1 (SLOWeave or fixed chunks, oldest-first), and
             the request-level metrics of Sec. 4.3 (TTFT, within-request P99
             TPOT, SLO attainment, goodput).

Every function states the passage it follows, and each reading taken where
the paper is silent or ambiguous is stated at the function that relies on it.
"""

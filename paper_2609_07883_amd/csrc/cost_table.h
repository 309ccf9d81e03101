// Cost table of measured iteration times (Sec. 5.1 profiler, Sec. 6.4 calibration).
#pragma once

#include <cstdint>
#include <vector>

// Planes of (decode batch) x (chunk) tables, one per cached-context point.
// A table built without a context axis has one plane that serves every
// prefix (p_grid = {0}, has_ctx false).
struct slw_cost_table {
    std::vector<int32_t> c_grid;   // strictly increasing, c_grid[0] == 0
    std::vector<int32_t> b_grid;   // strictly increasing, >= 0
    std::vector<int32_t> p_grid;   // strictly increasing, >= 0: prefix length of the chunk's sequence
    bool has_ctx = false;
    int32_t repeats = 0;
    std::vector<int64_t> samples;  // [np][nb][nc][repeats] ns
    std::vector<int64_t> p50;      // [np][nb][nc]
    std::vector<int64_t> p99;      // [np][nb][nc]
    std::vector<int64_t> t_hat;    // [np][nb][nc] running max of p99 along c

    int32_t nc() const { return static_cast<int32_t>(c_grid.size()); }
    int32_t nb() const { return static_cast<int32_t>(b_grid.size()); }
    int32_t np() const { return static_cast<int32_t>(p_grid.size()); }
};

namespace slw {

// Validates grids, fills the percentiles and the running maximum.  SLW_* code.
int finish_table(slw_cost_table* t);

// Nearest-rank percentile num/den of xs (sorted in place): sorted[ceil(k num/den) - 1].
int64_t nearest_rank(std::vector<int64_t>& xs, int64_t num, int64_t den);

// Alg. 1 with the margin of Sec. 3.3 split into an absolute part (ns) and a
// part relative to the prediction: a chunk c is admissible when
// T_hat(prefix, n, c) + ceil(rel_margin_ppm * T_hat / 1e6) + margin_ns <= budget.
// slw_select_chunk is this with prefix 0 and rel_margin_ppm 0.
int select_chunk_core(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active, int64_t now_ns,
                      int32_t prefix, int32_t remaining, int32_t c_max, int64_t margin_ns, int64_t rel_margin_ppm,
                      int32_t* chunk, uint32_t* flags, int32_t* n_lookups);

// The same search with base tokens already placed in the iteration: the
// largest c <= min(remaining, c_max - base, last grid chunk - base) with
// T_hat(prefix, n, base + c) + ceil(rel * T_hat / 1e6) + margin_ns <= budget
// (first-fit prefill batching, Sec. 3.3).  select_chunk_core is base 0.
int select_chunk_after(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active, int64_t now_ns,
                       int32_t prefix, int32_t base, int32_t remaining, int32_t c_max, int64_t margin_ns,
                       int64_t rel_margin_ppm, int32_t* chunk, uint32_t* flags, int32_t* n_lookups);

// T_hat at (prefix, n, c) with the lookup rules of the ABI; SLW_ERANGE outside the grids.
int lookup_ctx(const slw_cost_table* t, int32_t prefix, int32_t n, int32_t c, int64_t* t_ns);

// The simulator's default cost model (Sec. 4.1), in ns:
// T(n, c) = 0.35 + 1[n>0](0.90 + 0.055 n) + 1[c>0](0.40 + 0.006 c) ms.
int64_t analytic_iteration_ns(int32_t n, int32_t c);

}  // namespace slw

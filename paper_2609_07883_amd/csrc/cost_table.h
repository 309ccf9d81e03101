// Cost table of measured iteration times (Sec. 5.1 profiler, Sec. 6.4 calibration).
#pragma once

#include <cstdint>
#include <vector>

struct slw_cost_table {
    std::vector<int32_t> c_grid;   // strictly increasing, c_grid[0] == 0
    std::vector<int32_t> b_grid;   // strictly increasing, >= 0
    int32_t repeats = 0;
    std::vector<int64_t> samples;  // [nb][nc][repeats] ns
    std::vector<int64_t> p50;      // [nb][nc]
    std::vector<int64_t> p99;      // [nb][nc]
    std::vector<int64_t> t_hat;    // [nb][nc] running max of p99 along c

    int32_t nc() const { return static_cast<int32_t>(c_grid.size()); }
    int32_t nb() const { return static_cast<int32_t>(b_grid.size()); }
};

namespace slw {

// Validates grids, fills the percentiles and the running maximum.  SLW_* code.
int finish_table(slw_cost_table* t);

// The simulator's default cost model (Sec. 4.1), in ns:
// T(n, c) = 0.35 + 1[n>0](0.90 + 0.055 n) + 1[c>0](0.40 + 0.006 c) ms.
int64_t analytic_iteration_ns(int32_t n, int32_t c);

}  // namespace slw

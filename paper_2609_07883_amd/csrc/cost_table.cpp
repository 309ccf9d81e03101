// Cost table and chunk controller.
//
// Sec. 5.1: the profiler keeps P50 and P99 per (decode batch, chunk) grid
// point and applies a running maximum along the chunk axis, and the
// runtime's table is indexed by decode batch, cached context and chunk;
// Sec. 6.4: interpolate between profiled points.  Eq. 1 (the largest chunk
// whose predicted iteration, plus the margin of Sec. 3.3, meets the earliest
// deadline) is found by bisection, which Sec. 3.2 allows because the
// prediction is monotone in the chunk.
#include "cost_table.h"

#include <algorithm>
#include <cinttypes>
#include <cstdio>
#include <cstring>
#include <memory>

#include "common.h"

namespace slw {

// Nearest-rank percentile num/den: sorted[ceil(k*num/den) - 1].
int64_t nearest_rank(std::vector<int64_t>& xs, int64_t num, int64_t den) {
    std::sort(xs.begin(), xs.end());
    int64_t k = static_cast<int64_t>(xs.size());
    int64_t rank = (k * num + den - 1) / den;
    if (rank < 1) rank = 1;
    return xs[rank - 1];
}

namespace {

int check_grids(const int32_t* c_grid, int32_t nc, const int32_t* b_grid, int32_t nb) {
    if (!c_grid || !b_grid || nc < 1 || nb < 1) return fail(SLW_EINVAL, "empty grid");
    if (c_grid[0] != 0) return fail(SLW_EINVAL, "c_grid[0] must be 0 (the decode-only column)");
    for (int32_t j = 1; j < nc; ++j)
        if (c_grid[j] <= c_grid[j - 1]) return fail(SLW_EINVAL, "c_grid must increase strictly");
    if (b_grid[0] < 0) return fail(SLW_EINVAL, "b_grid values must be >= 0");
    for (int32_t i = 1; i < nb; ++i)
        if (b_grid[i] <= b_grid[i - 1]) return fail(SLW_EINVAL, "b_grid must increase strictly");
    return SLW_OK;
}

int check_p_grid(const int32_t* p_grid, int32_t np) {
    if (!p_grid || np < 1) return fail(SLW_EINVAL, "empty context grid");
    if (p_grid[0] < 0) return fail(SLW_EINVAL, "p_grid values must be >= 0");
    for (int32_t k = 1; k < np; ++k)
        if (p_grid[k] <= p_grid[k - 1]) return fail(SLW_EINVAL, "p_grid must increase strictly");
    return SLW_OK;
}

// Index of the first grid point >= v, or -1.
int32_t first_at_least(const std::vector<int32_t>& g, int32_t v) {
    auto it = std::lower_bound(g.begin(), g.end(), v);
    if (it == g.end()) return -1;
    return static_cast<int32_t>(it - g.begin());
}

// Table row (plane * nb + decode row) for (prefix, n), or -1 outside the grids.
int32_t row_for(const slw_cost_table* t, int32_t prefix, int32_t n) {
    const int32_t b = first_at_least(t->b_grid, n);
    if (b < 0) return -1;
    const int32_t p = t->has_ctx ? first_at_least(t->p_grid, prefix) : 0;
    if (p < 0) return -1;
    return p * t->nb() + b;
}

// T_hat on row `row` at chunk c (0 <= c <= last grid C).
int64_t lookup_row(const slw_cost_table* t, int32_t row, int32_t c) {
    const int64_t* r = t->t_hat.data() + static_cast<size_t>(row) * t->nc();
    if (c == 0) return r[0];
    auto it = std::lower_bound(t->c_grid.begin() + 1, t->c_grid.end(), c);
    int32_t j = static_cast<int32_t>(it - t->c_grid.begin());  // c_grid[j-1] < c <= c_grid[j]
    if (j == 1) return r[1];
    int64_t lo_c = t->c_grid[j - 1], hi_c = t->c_grid[j];
    int64_t num = (r[j] - r[j - 1]) * (c - lo_c);
    int64_t den = hi_c - lo_c;
    return r[j - 1] + (num + den - 1) / den;  // num >= 0: r is a running maximum
}

int range_error(const slw_cost_table* t, int32_t prefix, int32_t n) {
    if (first_at_least(t->b_grid, n) < 0)
        return fail(SLW_ERANGE, "n=%d above the decode grid (last %d)", n, t->b_grid.back());
    return fail(SLW_ERANGE, "prefix %d above the context grid (last %d)", prefix, t->p_grid.back());
}

std::unique_ptr<slw_cost_table> make_table(const int32_t* c_grid, int32_t nc, const int32_t* b_grid, int32_t nb,
                                           const int32_t* p_grid, int32_t np, const int64_t* samples,
                                           int32_t repeats) {
    auto t = std::make_unique<slw_cost_table>();
    t->c_grid.assign(c_grid, c_grid + nc);
    t->b_grid.assign(b_grid, b_grid + nb);
    if (p_grid) {
        t->p_grid.assign(p_grid, p_grid + np);
        t->has_ctx = true;
    } else {
        t->p_grid.assign(1, 0);
    }
    t->repeats = repeats;
    t->samples.assign(samples, samples + static_cast<size_t>(t->np()) * nb * nc * repeats);
    return t;
}

}  // namespace

int finish_table(slw_cost_table* t) {
    int rc = check_grids(t->c_grid.data(), t->nc(), t->b_grid.data(), t->nb());
    if (rc) return rc;
    rc = check_p_grid(t->p_grid.data(), t->np());
    if (rc) return rc;
    if (!t->has_ctx && t->np() != 1) return fail(SLW_EINVAL, "a table without a context axis has one plane");
    if (t->repeats < 1) return fail(SLW_EINVAL, "repeats must be >= 1");
    const size_t rows = static_cast<size_t>(t->np()) * t->nb();
    const size_t cells = rows * t->nc();
    if (t->samples.size() != cells * t->repeats) return fail(SLW_EINVAL, "sample count mismatch");
    t->p50.assign(cells, 0);
    t->p99.assign(cells, 0);
    t->t_hat.assign(cells, 0);
    std::vector<int64_t> tmp(t->repeats);
    for (size_t cell = 0; cell < cells; ++cell) {
        std::copy_n(t->samples.data() + cell * t->repeats, t->repeats, tmp.begin());
        t->p50[cell] = nearest_rank(tmp, 1, 2);
        t->p99[cell] = nearest_rank(tmp, 99, 100);
    }
    for (size_t i = 0; i < rows; ++i) {
        int64_t best = INT64_MIN;
        for (int32_t j = 0; j < t->nc(); ++j) {
            size_t cell = i * t->nc() + j;
            best = std::max(best, t->p99[cell]);
            t->t_hat[cell] = best;
        }
    }
    return SLW_OK;
}

int lookup_ctx(const slw_cost_table* t, int32_t prefix, int32_t n, int32_t c, int64_t* t_ns) {
    if (!t || !t_ns) return fail(SLW_EINVAL, "null argument");
    if (n < 0 || prefix < 0) return fail(SLW_EINVAL, "negative decode count or prefix");
    const int32_t row = row_for(t, prefix, n);
    if (row < 0) return range_error(t, prefix, n);
    if (c < 0 || c > t->c_grid.back()) return fail(SLW_ERANGE, "c=%d outside [0, %d]", c, t->c_grid.back());
    *t_ns = lookup_row(t, row, c);
    return SLW_OK;
}

int64_t analytic_iteration_ns(int32_t n, int32_t c) {
    int64_t t = 350000;
    if (n > 0) t += 900000 + 55000 * static_cast<int64_t>(n);
    if (c > 0) t += 400000 + 6000 * static_cast<int64_t>(c);
    return t;
}

// First x in [lo, hi) with pred(x) false, for a predicate true on a prefix
// of the range and false after it; hi if it holds everywhere.  Each probe
// halves the interval, so ceil(log2(hi - lo + 1)) probes at most.
template <class Pred>
int32_t first_false(int32_t lo, int32_t hi, Pred pred) {
    int32_t n = hi - lo;
    while (n > 0) {
        const int32_t half = n / 2;
        if (pred(lo + half)) {
            lo += half + 1;
            n -= half + 1;
        } else {
            n = half;
        }
    }
    return lo;
}

int select_chunk_core(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active, int64_t now_ns,
                      int32_t prefix, int32_t remaining, int32_t c_max, int64_t margin_ns, int64_t rel_margin_ppm,
                      int32_t* chunk, uint32_t* flags, int32_t* n_lookups) {
    return select_chunk_after(t, deadlines_ns, n_active, now_ns, prefix, 0, remaining, c_max, margin_ns,
                              rel_margin_ppm, chunk, flags, n_lookups);
}

int select_chunk_after(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active, int64_t now_ns,
                       int32_t prefix, int32_t base, int32_t remaining, int32_t c_max, int64_t margin_ns,
                       int64_t rel_margin_ppm, int32_t* chunk, uint32_t* flags, int32_t* n_lookups) {
    if (!t || !chunk || !flags) return fail(SLW_EINVAL, "null argument");
    *chunk = 0;
    *flags = 0;
    if (n_lookups) *n_lookups = 0;
    if (n_active < 0 || (n_active > 0 && !deadlines_ns)) return fail(SLW_EINVAL, "bad active set");
    if (prefix < 0) return fail(SLW_EINVAL, "negative prefix");
    if (rel_margin_ppm < 0 || rel_margin_ppm > 100000000) return fail(SLW_ERANGE, "relative margin out of range");
    if (base < 0) return fail(SLW_EINVAL, "negative base chunk");
    if (remaining <= 0) {  // no pending prefill
        *flags = SLW_FLAG_NO_PENDING;
        return SLW_OK;
    }
    int32_t cap = std::min(c_max - base, remaining);
    uint32_t fl = 0;
    if (t->c_grid.back() - base < cap) {
        cap = t->c_grid.back() - base;
        fl |= SLW_FLAG_CAPPED_BY_GRID;
    }
    if (cap < 0) cap = 0;
    if (n_active == 0) {  // nothing constrains the chunk
        *chunk = cap;
        *flags = fl | SLW_FLAG_NO_ACTIVE;
        return SLW_OK;
    }
    const int32_t row = row_for(t, prefix, n_active);
    if (row < 0) return range_error(t, prefix, n_active);
    int64_t earliest = deadlines_ns[0];
    for (int32_t i = 1; i < n_active; ++i) earliest = std::min(earliest, deadlines_ns[i]);
    const int64_t budget = earliest - now_ns;
    // predicted time plus the relative margin ceil(rel * T_hat / 1e6) (monotone in c like T_hat)
    auto predict = [&](int32_t c) {
        const int64_t v = lookup_row(t, row, base + c);
        return v + (rel_margin_ppm * v + 999999) / 1000000;
    };
    // Eq. 1 over c in [0, cap]: feasible(c) = predict(c) + margin <= budget
    // holds on a prefix of the range (predict is monotone in c), so the
    // chunk is one less than the first c in [1, cap] that is infeasible.
    int32_t lookups = 0;
    auto feasible = [&](int32_t c) {
        ++lookups;
        return predict(c) + margin_ns <= budget;
    };
    const int32_t lo = first_false(1, cap + 1, feasible) - 1;
    if (lo == 0 && !feasible(0)) fl |= SLW_FLAG_DECODE_INFEASIBLE;
    *chunk = lo;
    *flags = fl;
    if (n_lookups) *n_lookups = lookups;
    return SLW_OK;
}

}  // namespace slw

using namespace slw;

extern "C" int slw_cost_table_analytic(const int32_t* c_grid, int32_t nc, const int32_t* b_grid, int32_t nb,
                                       slw_cost_table** out) {
    return guarded([&] {
        if (!c_grid || !b_grid || !out || nc < 1 || nb < 1) return fail(SLW_EINVAL, "bad grids");
        std::vector<int64_t> v(static_cast<size_t>(nc) * nb);
        for (int32_t i = 0; i < nb; ++i)
            for (int32_t j = 0; j < nc; ++j) v[static_cast<size_t>(i) * nc + j] = analytic_iteration_ns(b_grid[i], c_grid[j]);
        return slw_cost_table_from_samples(c_grid, nc, b_grid, nb, v.data(), 1, out);
    });
}

extern "C" int slw_cost_table_from_samples(const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                                           int32_t nb, const int64_t* samples, int32_t repeats,
                                           slw_cost_table** out) {
    return guarded([&] {
        if (!out || !samples) return fail(SLW_EINVAL, "null argument");
        *out = nullptr;
        int rc = check_grids(c_grid, nc, b_grid, nb);
        if (rc) return rc;
        if (repeats < 1) return fail(SLW_EINVAL, "repeats must be >= 1");
        auto t = make_table(c_grid, nc, b_grid, nb, nullptr, 1, samples, repeats);
        rc = finish_table(t.get());
        if (rc) return rc;
        *out = t.release();
        return SLW_OK;
    });
}

extern "C" int slw_cost_table_from_samples_ctx(const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                                               int32_t nb, const int32_t* p_grid, int32_t np,
                                               const int64_t* samples, int32_t repeats, slw_cost_table** out) {
    return guarded([&] {
        if (!out || !samples) return fail(SLW_EINVAL, "null argument");
        *out = nullptr;
        int rc = check_grids(c_grid, nc, b_grid, nb);
        if (rc) return rc;
        rc = check_p_grid(p_grid, np);
        if (rc) return rc;
        if (repeats < 1) return fail(SLW_EINVAL, "repeats must be >= 1");
        auto t = make_table(c_grid, nc, b_grid, nb, p_grid, np, samples, repeats);
        rc = finish_table(t.get());
        if (rc) return rc;
        *out = t.release();
        return SLW_OK;
    });
}

extern "C" void slw_cost_table_free(slw_cost_table* t) { delete t; }

extern "C" int slw_cost_table_dims(const slw_cost_table* t, int32_t* nc, int32_t* nb, int32_t* repeats) {
    if (!t) return fail(SLW_EINVAL, "null table");
    if (nc) *nc = t->nc();
    if (nb) *nb = t->nb();
    if (repeats) *repeats = t->repeats;
    return SLW_OK;
}

extern "C" int slw_cost_table_grids(const slw_cost_table* t, int32_t* c_grid, int32_t* b_grid) {
    if (!t) return fail(SLW_EINVAL, "null table");
    if (c_grid) std::copy(t->c_grid.begin(), t->c_grid.end(), c_grid);
    if (b_grid) std::copy(t->b_grid.begin(), t->b_grid.end(), b_grid);
    return SLW_OK;
}

extern "C" int slw_cost_table_prefixes(const slw_cost_table* t, int32_t* p_grid, int32_t cap, int32_t* np) {
    if (!t || !np) return fail(SLW_EINVAL, "null argument");
    *np = t->has_ctx ? t->np() : 0;
    if (p_grid && t->has_ctx) {
        if (cap < t->np()) return fail(SLW_ERANGE, "%d context points, cap %d", t->np(), cap);
        std::copy(t->p_grid.begin(), t->p_grid.end(), p_grid);
    }
    return SLW_OK;
}

extern "C" int slw_cost_table_values(const slw_cost_table* t, int32_t which, int64_t* out, size_t cap) {
    if (!t || !out) return fail(SLW_EINVAL, "null argument");
    const std::vector<int64_t>* v = nullptr;
    switch (which) {
        case SLW_TABLE_SAMPLES: v = &t->samples; break;
        case SLW_TABLE_P50: v = &t->p50; break;
        case SLW_TABLE_P99: v = &t->p99; break;
        case SLW_TABLE_THAT: v = &t->t_hat; break;
        default: return fail(SLW_EINVAL, "unknown table view %d", which);
    }
    if (cap < v->size()) return fail(SLW_ERANGE, "output holds %zu values, need %zu", cap, v->size());
    std::copy(v->begin(), v->end(), out);
    return SLW_OK;
}

extern "C" int slw_cost_table_lookup(const slw_cost_table* t, int32_t n, int32_t c, int64_t* t_ns) {
    return lookup_ctx(t, 0, n, c, t_ns);
}

extern "C" int slw_cost_table_lookup_ctx(const slw_cost_table* t, int32_t prefix, int32_t n, int32_t c,
                                         int64_t* t_ns) {
    return lookup_ctx(t, prefix, n, c, t_ns);
}

extern "C" int slw_cost_table_monotone(const slw_cost_table* t, int32_t* violations, int64_t* worst_ns) {
    if (!t) return fail(SLW_EINVAL, "null table");
    int32_t count = 0;
    int64_t worst = 0;
    const size_t rows = static_cast<size_t>(t->np()) * t->nb();
    for (size_t i = 0; i < rows; ++i)
        for (int32_t j = 1; j < t->nc(); ++j) {
            int64_t a = t->p99[i * t->nc() + j - 1];
            int64_t b = t->p99[i * t->nc() + j];
            if (b < a) {
                ++count;
                worst = std::max(worst, a - b);
            }
        }
    if (violations) *violations = count;
    if (worst_ns) *worst_ns = worst;
    return SLW_OK;
}

// Text format: version 1 (no context axis) or 2 (a line of context points after the b grid).
extern "C" int slw_cost_table_save(const slw_cost_table* t, const char* path) {
    if (!t || !path) return fail(SLW_EINVAL, "null argument");
    FILE* f = fopen(path, "w");
    if (!f) return fail(SLW_EINVAL, "cannot open %s for writing", path);
    if (t->has_ctx) fprintf(f, "sloweave-cost-table 2\n%d %d %d %d\n", t->nc(), t->nb(), t->np(), t->repeats);
    else fprintf(f, "sloweave-cost-table 1\n%d %d %d\n", t->nc(), t->nb(), t->repeats);
    for (int32_t c : t->c_grid) fprintf(f, "%d ", c);
    fprintf(f, "\n");
    for (int32_t b : t->b_grid) fprintf(f, "%d ", b);
    fprintf(f, "\n");
    if (t->has_ctx) {
        for (int32_t p : t->p_grid) fprintf(f, "%d ", p);
        fprintf(f, "\n");
    }
    for (size_t i = 0; i < t->samples.size(); ++i)
        fprintf(f, "%" PRId64 "%c", t->samples[i], (i + 1) % t->repeats ? ' ' : '\n');
    int bad = ferror(f);
    if (fclose(f) != 0 || bad) return fail(SLW_EINVAL, "write to %s failed", path);
    return SLW_OK;
}

extern "C" int slw_cost_table_load(const char* path, slw_cost_table** out) {
    return guarded([&] {
        if (!path || !out) return fail(SLW_EINVAL, "null argument");
        *out = nullptr;
        FILE* f = fopen(path, "r");
        if (!f) return fail(SLW_EINVAL, "cannot open %s", path);
        std::unique_ptr<FILE, int (*)(FILE*)> guard(f, fclose);
        int version = 0, nc = 0, nb = 0, np = 1, reps = 0;
        if (fscanf(f, "sloweave-cost-table %d", &version) != 1 || (version != 1 && version != 2))
            return fail(SLW_EINVAL, "%s: bad header", path);
        const int got = version == 1 ? fscanf(f, "%d %d %d", &nc, &nb, &reps) : fscanf(f, "%d %d %d %d", &nc, &nb, &np, &reps);
        if (got != (version == 1 ? 3 : 4) || nc < 1 || nb < 1 || np < 1 || reps < 1 || nc > (1 << 20) ||
            nb > (1 << 20) || np > (1 << 20) || reps > (1 << 20))
            return fail(SLW_EINVAL, "%s: bad header", path);
        auto t = std::make_unique<slw_cost_table>();
        t->c_grid.resize(nc);
        t->b_grid.resize(nb);
        t->p_grid.assign(np, 0);
        t->has_ctx = version == 2;
        t->repeats = reps;
        for (auto& c : t->c_grid)
            if (fscanf(f, "%d", &c) != 1) return fail(SLW_EINVAL, "%s: truncated c grid", path);
        for (auto& b : t->b_grid)
            if (fscanf(f, "%d", &b) != 1) return fail(SLW_EINVAL, "%s: truncated b grid", path);
        if (t->has_ctx)
            for (auto& p : t->p_grid)
                if (fscanf(f, "%d", &p) != 1) return fail(SLW_EINVAL, "%s: truncated context grid", path);
        t->samples.resize(static_cast<size_t>(np) * nc * nb * reps);
        for (auto& s : t->samples)
            if (fscanf(f, "%" SCNd64, &s) != 1) return fail(SLW_EINVAL, "%s: truncated samples", path);
        int rc = finish_table(t.get());
        if (rc) return rc;
        *out = t.release();
        return SLW_OK;
    });
}

extern "C" int slw_select_chunk(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active,
                                int64_t now_ns, int32_t remaining, int32_t c_max, int64_t margin_ns,
                                int32_t* chunk, uint32_t* flags, int32_t* n_lookups) {
    return select_chunk_core(t, deadlines_ns, n_active, now_ns, 0, remaining, c_max, margin_ns, 0, chunk, flags,
                             n_lookups);
}

extern "C" int slw_select_chunk_ctx(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active,
                                    int64_t now_ns, int32_t prefix, int32_t remaining, int32_t c_max,
                                    int64_t margin_ns, int32_t* chunk, uint32_t* flags, int32_t* n_lookups) {
    return select_chunk_core(t, deadlines_ns, n_active, now_ns, prefix, remaining, c_max, margin_ns, 0, chunk,
                             flags, n_lookups);
}

// Serving loop: the iteration-level scheduler that drives the mixed iteration
// (Sec. 3.1 deadline model, Sec. 3.2 / Alg. 1 chunk choice, Sec. 4.1 iteration
// semantics, Sec. 4.3 oldest-first queueing), with the policy variants of
// Sec. 3.3-3.5 as options (per-request objectives and class margins, queue
// disciplines, admission control, aging, first-fit prefill batching).  It
// uses the KV manager, the chunk search of Alg. 1 and slw_mixed_iteration.
//
// Two executors share every scheduling decision: the GPU one runs each
// iteration on the device and reads the host clock once the stream drains;
// the analytic one advances a virtual clock by the Sec. 4.1 cost model, which
// makes the same loop an iteration-level simulator.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstdint>
#include <limits>
#include <map>
#include <thread>
#include <vector>

#include "common.h"
#include "cost_table.h"
#include "sloweave.h"

namespace slw {
namespace {

int64_t host_ns() {
    return std::chrono::duration_cast<std::chrono::nanoseconds>(
               std::chrono::steady_clock::now().time_since_epoch())
        .count();
}

struct Live {
    int32_t req;          // index into the caller's array
    int32_t prompt_done;  // prompt tokens processed
    int32_t emitted;      // output tokens emitted
    int64_t last_ns;      // l_i: time of the latest token
    int64_t waited_ns;    // pending: when it became eligible or last ran a chunk
    bool started;         // prompt begun (KV sequence exists)
};

int64_t kv_blocks_for(const slw_request& r) {
    // positions 0 .. prompt + output - 2 are cached (the last token is never fed back)
    return ceil_div(static_cast<int64_t>(r.prompt_len) + r.output_len - 1, 16);
}

int check_opts(slw_ctx* ctx, const slw_request* reqs, int32_t n, const slw_serve_opts* o) {
    if (!o || (n > 0 && !reqs)) return fail(SLW_EINVAL, "null argument");
    if (n < 0) return fail(SLW_EINVAL, "negative request count");
    if (o->policy != SLW_POLICY_SLOWEAVE && o->policy != SLW_POLICY_FIXED)
        return fail(SLW_EINVAL, "unknown policy %d", o->policy);
    if (o->policy == SLW_POLICY_FIXED && o->fixed_chunk < 1) return fail(SLW_EINVAL, "fixed_chunk must be >= 1");
    if (o->policy == SLW_POLICY_SLOWEAVE && (!o->table || o->c_max < 1))
        return fail(SLW_EINVAL, "SLOWeave needs a cost table and c_max >= 1");
    if (o->max_decode < 1) return fail(SLW_EINVAL, "max_decode must be >= 1");
    if (o->tpot_ns <= 0 || o->margin_ns < 0) return fail(SLW_EINVAL, "bad TPOT objective or margin");
    if (o->executor != SLW_EXEC_GPU && o->executor != SLW_EXEC_ANALYTIC && o->executor != SLW_EXEC_TABLE)
        return fail(SLW_EINVAL, "unknown executor %d", o->executor);
    if (o->executor == SLW_EXEC_TABLE && !o->exec_table) return fail(SLW_EINVAL, "table executor needs exec_table");
    if (o->residual_window < 0 || o->residual_window > 65536)
        return fail(SLW_ERANGE, "residual_window must be in [0, 65536]");
    if (o->queue < SLW_QUEUE_OLDEST || o->queue > SLW_QUEUE_EDF) return fail(SLW_EINVAL, "unknown queue %d", o->queue);
    if (o->admit_ppm < 0 || o->admit_ppm > 10000000) return fail(SLW_ERANGE, "admit_ppm must be in [0, 1e7]");
    if (o->admit_ppm > 0 && !o->table) return fail(SLW_EINVAL, "admission control needs a cost table");
    if (o->aging_ns < 0 || (o->aging_ns > 0 && o->aging_chunk < 1))
        return fail(SLW_EINVAL, "aging needs aging_ns >= 0 and aging_chunk >= 1");
    if (o->max_prefills < 0) return fail(SLW_EINVAL, "max_prefills must be >= 0");
    if (o->log_every < 0) return fail(SLW_EINVAL, "log_every must be >= 0");
    if (o->fallback_window < 0 || o->fallback_window > 65536)
        return fail(SLW_ERANGE, "fallback_window must be in [0, 65536]");
    if (o->fallback_window > 0 && !o->table) return fail(SLW_EINVAL, "the telemetry fallback needs a cost table");
    if (o->max_prefills > SLW_MAX_PREFILLS && o->executor == SLW_EXEC_GPU)
        return fail(SLW_ERANGE, "max_prefills %d above SLW_MAX_PREFILLS on the GPU executor", o->max_prefills);
    if (o->executor == SLW_EXEC_GPU) {
        if (!ctx || !o->x_in || !o->x_out || !o->ws) return fail(SLW_EINVAL, "GPU executor needs ctx and buffers");
        const int64_t cap = o->policy == SLW_POLICY_FIXED ? o->fixed_chunk : o->c_max;
        if (cap + o->max_decode > o->max_rows)
            return fail(SLW_ERANGE, "chunk cap %lld + max_decode %d exceeds max_rows %d",
                        static_cast<long long>(cap), o->max_decode, o->max_rows);
    }
    std::map<int64_t, int> seen;
    for (int32_t i = 0; i < n; ++i) {
        const slw_request& r = reqs[i];
        if (r.prompt_len < 1 || r.output_len < 1 || r.arrival_ns < 0)
            return fail(SLW_EINVAL, "request %lld: bad lengths or arrival", static_cast<long long>(r.id));
        if (seen[r.id]++) return fail(SLW_EINVAL, "duplicate request id %lld", static_cast<long long>(r.id));
        if (o->slo && (o->slo[i].tpot_ns < 0 || o->slo[i].ttft_ns < 0))
            return fail(SLW_EINVAL, "request %lld: negative objective", static_cast<long long>(r.id));
    }
    return SLW_OK;
}

int serve_impl(slw_ctx* ctx, const slw_request* reqs, int32_t n, const slw_serve_opts* o, int64_t* token_ns,
               int64_t token_cap, slw_iteration_record* iters, int64_t iter_cap, int64_t* n_iters) {
    int rc = check_opts(ctx, reqs, n, o);
    if (rc) return rc;
    if (!n_iters || (n > 0 && (!token_ns || !iters))) return fail(SLW_EINVAL, "null output");
    *n_iters = 0;
    std::vector<int64_t> tok_off(n + 1, 0);
    for (int32_t i = 0; i < n; ++i) tok_off[i + 1] = tok_off[i] + reqs[i].output_len;
    if (tok_off[n] > token_cap) return fail(SLW_ERANGE, "token_ns holds %lld, need %lld",
                                           static_cast<long long>(token_cap), static_cast<long long>(tok_off[n]));
    if (n == 0) return SLW_OK;

    const bool gpu = o->executor == SLW_EXEC_GPU;
    int64_t pool_blocks = 0;
    if (gpu) {
        int32_t free_blocks = 0;
        rc = slw_kv_free_blocks(ctx, &free_blocks);
        if (rc) return rc;
        pool_blocks = free_blocks;
        for (int32_t i = 0; i < n; ++i)
            if (kv_blocks_for(reqs[i]) > pool_blocks)
                return fail(SLW_ENOMEM, "request %lld needs %lld KV blocks, the pool has %lld free",
                            static_cast<long long>(reqs[i].id), static_cast<long long>(kv_blocks_for(reqs[i])),
                            static_cast<long long>(pool_blocks));
    }

    std::vector<int32_t> order(n);  // arrival order (arrival, id)
    for (int32_t i = 0; i < n; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
        return reqs[a].arrival_ns != reqs[b].arrival_ns ? reqs[a].arrival_ns < reqs[b].arrival_ns
                                                        : reqs[a].id < reqs[b].id;
    });

    // per-request objectives (Sec. 3.5)
    auto D_of = [&](int32_t i) { return o->slo && o->slo[i].tpot_ns > 0 ? o->slo[i].tpot_ns : o->tpot_ns; };
    auto delta_of = [&](int32_t i) { return o->slo && o->slo[i].margin_ns >= 0 ? o->slo[i].margin_ns : o->margin_ns; };
    auto edf_key = [&](int32_t i) {
        return o->slo && o->slo[i].ttft_ns > 0 ? reqs[i].arrival_ns + o->slo[i].ttft_ns
                                               : std::numeric_limits<int64_t>::max();
    };
    // queue order (Sec. 3.4), ties to the older request
    auto before = [&](const Live& x, const Live& y) {
        const slw_request& a = reqs[x.req];
        const slw_request& b = reqs[y.req];
        if (o->queue == SLW_QUEUE_SRPT) {
            const int32_t ra = a.prompt_len - x.prompt_done, rb = b.prompt_len - y.prompt_done;
            if (ra != rb) return ra < rb;
        } else if (o->queue == SLW_QUEUE_EDF) {
            const int64_t ea = edf_key(x.req), eb = edf_key(y.req);
            if (ea != eb) return ea < eb;
        }
        return a.arrival_ns != b.arrival_ns ? a.arrival_ns < b.arrival_ns : a.id < b.id;
    };
    const int32_t max_prefills = std::max(o->max_prefills, 1);

    std::vector<Live> pending;           // eligible, prompt not finished (queue order once sorted)
    std::map<int64_t, Live> active;      // decoding, keyed (and batched) by id
    int64_t committed_blocks = 0;        // KV blocks every started request may reach
    int32_t next = 0, finished = 0;

    // Trace clock.  Analytic: purely virtual.  GPU: host time since the start
    // minus the idle gaps jumped over.
    int64_t virt = reqs[order[0]].arrival_ns;
    const int64_t t0_host = host_ns();
    int64_t host_shift = virt;  // trace time = host_ns() - t0_host + host_shift
    auto now = [&]() { return gpu ? host_ns() - t0_host + host_shift : virt; };

    std::vector<int64_t> dec_ids, deadlines, eff;
    std::vector<int32_t> ctx_lens;
    std::vector<std::pair<int32_t, int32_t>> plan;  // (index into pending, tokens) served this iteration
    std::vector<int64_t> pf_seq;                     // GPU batch: the plan's sequences, prefixes, chunks
    std::vector<int32_t> pf_prefix, pf_chunk;
    // telemetry: relative residuals (ppm) of the last residual_window chunked iterations
    const int32_t W = o->residual_window;
    std::vector<int64_t> resid(std::max(W, 1)), scratch;
    int64_t n_resid = 0;
    // telemetry fallback: absolute residuals (ns) of the last fallback_window priced iterations
    const int32_t FW = o->fallback_window;
    std::vector<int64_t> fb_resid(std::max(FW, 1));
    int64_t n_fb = 0;
    const hipStream_t stream = static_cast<hipStream_t>(o->stream);

    auto finish = [&](const slw_request& r) {
        if (gpu) {
            const int e = slw_seq_free(ctx, r.id);
            if (e) return e;
            committed_blocks -= kv_blocks_for(r);
        }
        ++finished;
        return SLW_OK;
    };

    while (finished < n) {
        int64_t t = now();
        while (next < n && reqs[order[next]].arrival_ns <= t) {
            const int32_t i = order[next++];
            if (o->admit_ppm > 0) {  // admission control (Sec. 3.4)
                const int32_t nf = static_cast<int32_t>(active.size() + pending.size() + 1);
                int64_t cost = 0;
                const bool priced = lookup_ctx(o->table, 0, nf, 0, &cost) == SLW_OK;
                if (!priced) clear_error();
                if (!priced || (cost + delta_of(i)) * 1000000 > D_of(i) * o->admit_ppm) {
                    std::fill(token_ns + tok_off[i], token_ns + tok_off[i + 1], int64_t{-1});
                    ++finished;
                    continue;
                }
            }
            pending.push_back(Live{i, 0, 0, 0, t, false});
        }
        if (finished == n) break;
        if (pending.empty() && active.empty()) {
            const int64_t arr = reqs[order[next]].arrival_ns;  // next < n: someone is still to come
            if (!gpu) {
                virt = arr;
            } else if (o->skip_idle) {
                host_shift += arr - t;
            } else {
                std::this_thread::sleep_for(std::chrono::nanoseconds(std::max<int64_t>(0, arr - t)));
            }
            continue;
        }
        if (*n_iters >= iter_cap) return fail(SLW_ERANGE, "more than %lld iterations", static_cast<long long>(iter_cap));
        slw_iteration_record rec{};
        rec.start_ns = t;
        rec.prefill_id = -1;
        rec.predicted_ns = -1;

        const int64_t t_dec0 = host_ns();
        dec_ids.clear();
        deadlines.clear();
        eff.clear();
        ctx_lens.clear();
        for (const auto& kv : active) {
            const Live& a = kv.second;
            const slw_request& r = reqs[a.req];
            dec_ids.push_back(r.id);
            deadlines.push_back(a.last_ns + D_of(a.req));
            eff.push_back(a.last_ns + D_of(a.req) - (delta_of(a.req) - o->margin_ns));
            ctx_lens.push_back(r.prompt_len + a.emitted - 1);
        }
        const int32_t nd = static_cast<int32_t>(dec_ids.size());
        if (nd > 0) rec.budget_ns = *std::min_element(deadlines.begin(), deadlines.end()) - t;
        if (o->queue != SLW_QUEUE_OLDEST) std::sort(pending.begin(), pending.end(), before);

        Live* head = nullptr;
        if (!pending.empty()) {
            Live& h = pending.front();
            if (nd >= o->max_decode) {
                rec.flags |= SLW_SERVE_DECODE_CAP;
            } else if (gpu && !h.started && committed_blocks + kv_blocks_for(reqs[h.req]) > pool_blocks) {
                rec.flags |= SLW_SERVE_KV_WAIT;
            } else {
                head = &h;
            }
        }
        int32_t chunk = 0;
        int64_t rel = 0;
        plan.clear();
        const int32_t prefix = head ? head->prompt_done : 0;  // context the iteration is priced at
        if (head) {
            const int32_t remaining = reqs[head->req].prompt_len - head->prompt_done;
            rec.remaining = remaining;
            if (o->policy == SLW_POLICY_FIXED) {
                chunk = std::min(o->fixed_chunk, remaining);
            } else {
                if (W > 0 && n_resid > 0) {
                    scratch.assign(resid.begin(), resid.begin() + std::min<int64_t>(n_resid, W));
                    rel = std::min<int64_t>(std::max<int64_t>(nearest_rank(scratch, 99, 100), 0), 100000000);
                }
                rec.rel_margin_ppm = rel;
                bool fallback = false;
                if (FW > 0 && n_fb > 0 && nd > 0) {  // with no decode there is no deadline to protect
                    scratch.assign(fb_resid.begin(), fb_resid.begin() + std::min<int64_t>(n_fb, FW));
                    rec.resid_p99_ns = nearest_rank(scratch, 99, 100);
                    fallback = rec.resid_p99_ns > o->margin_ns;
                }
                if (fallback) {
                    chunk = 0;
                    rec.flags |= SLW_SERVE_FALLBACK;
                } else {
                    uint32_t fl = 0;
                    rc = select_chunk_core(o->table, eff.data(), nd, t, prefix, remaining, o->c_max, o->margin_ns,
                                           rel, &chunk, &fl, nullptr);
                    if (rc == SLW_ERANGE) {  // more decodes than the table prices
                        clear_error();
                        chunk = 0;
                        fl = SLW_SERVE_UNPRICED;
                    } else if (rc) {
                        return rc;
                    }
                    rec.flags |= fl;
                }
                if (chunk == 0 && o->aging_ns > 0 && t - head->waited_ns >= o->aging_ns) {
                    chunk = std::min({o->aging_chunk, remaining, o->c_max});
                    rec.flags |= SLW_SERVE_AGED;
                }
            }
            if (chunk > 0) plan.emplace_back(0, chunk);
            // first-fit prefill batching (Sec. 3.3)
            if (o->policy == SLW_POLICY_SLOWEAVE && max_prefills > 1 && chunk > 0 && chunk == remaining &&
                !(rec.flags & SLW_SERVE_AGED)) {
                // GPU: blocks committed by the prompts this iteration starts
                int64_t starting = gpu && !head->started ? kv_blocks_for(reqs[head->req]) : 0;
                for (size_t k = 1; k < pending.size(); ++k) {
                    if (static_cast<int32_t>(plan.size()) >= max_prefills) break;
                    if (nd + static_cast<int32_t>(plan.size()) >= o->max_decode) break;
                    if (gpu && !pending[k].started) {  // the pool must hold it to its last token
                        const int64_t need = kv_blocks_for(reqs[pending[k].req]);
                        if (committed_blocks + starting + need > pool_blocks) break;
                        starting += need;
                    }
                    const int32_t rem = reqs[pending[k].req].prompt_len - pending[k].prompt_done;
                    int32_t c = 0;
                    uint32_t fl = 0;
                    rc = select_chunk_after(o->table, eff.data(), nd, t, prefix, chunk, rem, o->c_max, o->margin_ns,
                                            rel, &c, &fl, nullptr);
                    if (rc == SLW_ERANGE) {
                        clear_error();
                        c = 0;
                    } else if (rc) {
                        return rc;
                    }
                    if (c <= 0) break;
                    plan.emplace_back(static_cast<int32_t>(k), c);
                    chunk += c;
                    if (c < rem) break;
                }
            }
        }
        rec.decide_ns = host_ns() - t_dec0;
        rec.chunk = chunk;
        rec.n_decode = nd;
        rec.n_prefill = static_cast<int32_t>(plan.size());
        if (o->table) {
            int64_t p = 0;
            if (lookup_ctx(o->table, prefix, nd, chunk, &p) == SLW_OK) rec.predicted_ns = p;
            else clear_error();
        }

        if (gpu) {
            pf_seq.clear();
            pf_prefix.clear();
            pf_chunk.clear();
            for (const auto& pc : plan) {
                Live& h = pending[pc.first];
                if (!h.started) {
                    rc = slw_seq_create(ctx, reqs[h.req].id);
                    if (rc) return rc;
                    h.started = true;
                    committed_blocks += kv_blocks_for(reqs[h.req]);
                }
                pf_seq.push_back(reqs[h.req].id);
                pf_prefix.push_back(h.prompt_done);
                pf_chunk.push_back(pc.second);
            }
            slw_batch b{};
            b.C = chunk;
            b.prefill_seq = chunk > 0 ? pf_seq[0] : 0;
            b.prefix_len = chunk > 0 ? pf_prefix[0] : 0;
            b.B = nd;
            b.decode_seqs = dec_ids.data();
            b.context_lens = ctx_lens.data();
            if (plan.size() > 1) {
                b.n_prefill = static_cast<int32_t>(plan.size());
                b.prefill_seqs = pf_seq.data();
                b.prefix_lens = pf_prefix.data();
                b.chunk_lens = pf_chunk.data();
            }
            rc = slw_mixed_iteration(ctx, &b, o->x_in, o->x_out, o->ws, o->ws_bytes, o->stream);
            if (rc) return rc;
            if (hipStreamSynchronize(stream) != hipSuccess)
                return fail(SLW_EHIP, "stream synchronisation failed after iteration %lld",
                            static_cast<long long>(*n_iters));
        } else if (o->executor == SLW_EXEC_ANALYTIC) {
            virt = t + analytic_iteration_ns(nd, chunk);
        } else {
            int64_t dt = 0;
            rc = lookup_ctx(o->exec_table, prefix, nd, chunk, &dt);
            if (rc) return rc;
            virt = t + dt;
        }
        const int64_t end = now();
        rec.end_ns = end;
        if (chunk > 0) rec.prefill_id = reqs[head->req].id;
        iters[(*n_iters)++] = rec;
        if (o->log_every > 0 && *n_iters % o->log_every == 0)
            std::fprintf(stderr, "slw_serve: %lld iterations, trace clock %.1f s, %d of %d requests done\n",
                         static_cast<long long>(*n_iters), static_cast<double>(end) * 1e-9, finished, n);
        if (W > 0 && chunk > 0 && rec.predicted_ns > 0) {
            const int64_t num = (end - t - rec.predicted_ns) * 1000000;
            int64_t q = num / rec.predicted_ns;
            if (num % rec.predicted_ns != 0 && num < 0) --q;  // floor
            resid[n_resid % W] = q;
            ++n_resid;
        }
        if (FW > 0 && rec.predicted_ns > 0) {
            fb_resid[n_fb % FW] = end - t - rec.predicted_ns;
            ++n_fb;
        }

        // decodes: one token each
        for (auto it = active.begin(); it != active.end();) {
            Live& a = it->second;
            const slw_request& r = reqs[a.req];
            token_ns[tok_off[a.req] + a.emitted] = end;
            ++a.emitted;
            a.last_ns = end;
            if (a.emitted == r.output_len) {
                rc = finish(r);
                if (rc) return rc;
                it = active.erase(it);
            } else {
                ++it;
            }
        }
        // the chunks: a prompt's last chunk emits its first token
        bool any_done = false;
        for (const auto& pc : plan) {
            Live& h = pending[pc.first];
            h.prompt_done += pc.second;
            h.waited_ns = end;
            const slw_request& r = reqs[h.req];
            if (h.prompt_done == r.prompt_len) {
                any_done = true;
                token_ns[tok_off[h.req]] = end;
                h.emitted = 1;
                h.last_ns = end;
                if (r.output_len == 1) {
                    rc = finish(r);
                    if (rc) return rc;
                } else {
                    active.emplace(r.id, h);
                }
            }
        }
        if (any_done)
            pending.erase(std::remove_if(pending.begin(), pending.end(),
                                         [&](const Live& x) { return x.prompt_done == reqs[x.req].prompt_len; }),
                          pending.end());
    }
    return SLW_OK;
}

}  // namespace
}  // namespace slw

extern "C" int slw_serve(slw_ctx* ctx, const slw_request* reqs, int32_t n, const slw_serve_opts* opts,
                         int64_t* token_ns, int64_t token_cap, slw_iteration_record* iters, int64_t iter_cap,
                         int64_t* n_iters) {
    return slw::guarded([&] { return slw::serve_impl(ctx, reqs, n, opts, token_ns, token_cap, iters, iter_cap, n_iters); });
}

// Context, paged-KV bookkeeping, the mixed iteration and the cost profiler.
//
// A mixed iteration (Sec. 3: one prefill chunk plus one token for every
// active decode; Sec. 5.1: the chunk arrives through ordinary sequence
// metadata) is: host-side reservation and slot mapping, one upload of the
// per-iteration metadata through a pinned staging ring, a RoPE table for the
// iteration's positions, then per layer: RMSNorm, QKV GEMM (RoPE and KV
// append in its epilogue), chunk and decode attention, output GEMM into an
// fp32 residual, RMSNorm, gate/up GEMM (SiLU*mul epilogue), down GEMM.
#include <algorithm>
#include <chrono>
#include <cstring>
#include <limits>
#include <memory>
#include <mutex>
#include <random>
#include <unordered_set>
#include <vector>

#include "common.h"
#include "cost_table.h"
#include "kernels.h"
#include "kv_manager.h"

using namespace slw;

namespace {

constexpr int kRing = 4;                 // pinned staging buffers in flight
// Decode attention runs one wave per work-group, two per SIMD (its register
// use allows no more): kDecodeWaves of them fill a 256-CU part once.  Their
// keys are cut into equal runs (at least kDecodeMinKeys each), so that every
// wave of the launch finishes at about the same time.
constexpr int kDecodeWaves = 2048;
constexpr int kDecodeMinKeys = 128;
// Chunk attention runs one work-group per CU (its register use allows no
// more), so a launch of kChunkSlots work-groups with equal work finishes in
// one round on a 256-CU part.  A work-group takes at least kChunkMinTiles
// 64-key tiles, which keeps its fixed costs (Q load, partial write) small.
constexpr int kChunkSlots = 256;
constexpr int kChunkMinTiles = 4;
// Whole query tiles per work-group when the largest group's load is within
// 11/10 of an equal share.
constexpr int64_t kChunkWholeSlackNum = 11, kChunkWholeSlackDen = 10;
// Chunk and decode attention share one launch (decode waves run as chunk
// work-groups leave CUs free) unless the chunk holds at least this many
// (query, key) pairs: then decode attention runs on a second stream beside
// the chunk kernel for its whole length, which a long chunk kernel even
// finishes sooner (8B layer, 4096-token chunk at a 28 K prefix with eight
// 16-32 K decodes: 2256 us with the decodes beside it, 2432 us alone).  One
// launch saves the fork and join, 9-20 us an iteration on the layer sweep's
// and the chat mix's chunks; the two ways measured even at 8-9 M pairs.
constexpr int64_t kTwoStreamMinPairs = int64_t{8} << 20;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

#define HIP_TRY(expr)                                                                      \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess) return fail(SLW_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

// One prefill of an iteration: `c` chunk rows from row `row0` on, at positions
// prefix .. prefix + c - 1 of sequence `seq`.
struct Prefill {
    int64_t seq;
    int32_t prefix;
    int32_t c;
    int32_t row0;
};

}  // namespace

// Work lists of the two attentions of one iteration (host build areas).
struct DecodePlan {
    std::vector<int32_t> b, kb, ke;  // items: decode, first key (a multiple of 64), key past the last
    std::vector<int32_t> off;        // [B + 1] first item of each decode
    std::vector<int32_t> slot_off;   // [slots + 1] first item of each wave slot
};
struct ChunkPlan {
    std::vector<int32_t> items;       // [3 n]: query tile, first key, key past the last
    std::vector<int32_t> slot_off;    // [slots + 1] first entry of each work-group in slot_items
    std::vector<int32_t> slot_items;  // [n] the items of each work-group in turn
    std::vector<int32_t> qt_off;      // [n_qt + 1] first item of each query tile
    bool whole = false;               // whole query tiles per work-group
};

struct slw_ctx {
    slw_model_cfg cfg{};
    std::vector<slw_layer_weights> w;
    std::vector<char> have_w;
    void* k_pool = nullptr;
    void* v_pool = nullptr;
    KvManager kv;
    bool kv_ready = false;
    std::vector<int32_t> last_slots;
    std::vector<int32_t> slots_build;  // slots of the iteration being built
    std::vector<Prefill> prefills;     // the iteration's prefills in row order
    std::vector<int32_t> meta;  // host build area
    DecodePlan dplan;           // the iteration's attention work (host build areas)
    ChunkPlan cplan;

    // HIP resources, created on first device use
    bool hip_ready = false;
    int32_t* staging[kRing] = {};      // coherent pinned host memory
    int32_t* staging_dev[kRing] = {};  // the same memory's device address
    size_t staging_cap[kRing] = {};
    hipEvent_t staged[kRing] = {};
    int ring = 0;
    // second stream for decode attention next to a long chunk's attention,
    // with a fork and a join event per layer
    hipStream_t side = nullptr;
    std::vector<hipEvent_t> fork_ev, join_ev;

    // stage telemetry: a ring of `stage_depth` event sets, each [layer][stage boundary]
    int stage_depth = 0;
    std::vector<hipEvent_t> stage_ev;
    std::vector<uint32_t> stage_mask;  // per set: stages that iteration ran (0: none recorded)
    int64_t stage_iter = 0;            // iterations recorded so far

    ~slw_ctx() {
        if (!hip_ready) return;
        for (int i = 0; i < kRing; ++i) {
            if (staged[i]) {
                (void)hipEventSynchronize(staged[i]);
                (void)hipEventDestroy(staged[i]);
            }
            if (staging[i]) (void)hipHostFree(staging[i]);
        }
        for (hipEvent_t e : stage_ev) (void)hipEventDestroy(e);
        if (side) {
            (void)hipStreamSynchronize(side);
            (void)hipStreamDestroy(side);
        }
        for (hipEvent_t e : fork_ev) (void)hipEventDestroy(e);
        for (hipEvent_t e : join_ev) (void)hipEventDestroy(e);
    }
};

namespace {

int qkv_width(const slw_model_cfg& c) { return (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim; }
int max_blocks(const slw_model_cfg& c) { return static_cast<int>(ceil_div(c.max_pos, 16)); }
int decode_slot_cap(const slw_model_cfg& c) { return std::max(1, kDecodeWaves / c.n_kv_heads); }
// A run crosses at most one decode boundary more than it has runs: items <= slots + B - 1.
int decode_work_cap(const slw_model_cfg& c, int B) { return decode_slot_cap(c) + B + 1; }

// Query tiles of the chunk rows: each prefill's rows are tiled on their own,
// so up to SLW_MAX_PREFILLS - 1 tiles more than one prefill of C rows needs.
int chunk_tiles(const slw_model_cfg& c, int C) {
    if (C <= 0) return 0;
    return static_cast<int>(ceil_div(C, chunk_tile_positions(c.n_q_heads / c.n_kv_heads))) +
           std::min(C, static_cast<int>(SLW_MAX_PREFILLS)) - 1;
}
int chunk_slot_cap(const slw_model_cfg& c) { return std::max(1, kChunkSlots / c.n_kv_heads); }
int chunk_item_cap(const slw_model_cfg& c, int C) {
    return C > 0 ? chunk_tiles(c, C) + chunk_slot_cap(c) : 0;
}

size_t meta_ints(const slw_model_cfg& c, int C, int B) {
    const int M = C + B;
    const size_t mb = static_cast<size_t>(max_blocks(c));
    const size_t np = C > 0 ? static_cast<size_t>(std::min(C, static_cast<int>(SLW_MAX_PREFILLS))) : 0;
    return 2 * static_cast<size_t>(M) + B + (B + 1) + static_cast<size_t>(B) * mb + np * mb +
           3 * static_cast<size_t>(decode_work_cap(c, B)) + (B + 1) + decode_slot_cap(c) + 1 +
           4 * static_cast<size_t>(chunk_item_cap(c, C)) +
           5 * static_cast<size_t>(chunk_tiles(c, C)) + 1 + chunk_slot_cap(c) + 1;
}

struct Layout {
    size_t xn, qkv, attn, h, act, rope, meta, part_o, part_ml, cpart_o, cpart_ml, gemm_part, end_fixed;
};

Layout layout(const slw_model_cfg& c, int C, int B) {
    const size_t M = static_cast<size_t>(C) + B;
    const int W = decode_work_cap(c, B);
    Layout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t at = off;
        off += align_up(bytes);
        return at;
    };
    L.xn = take(M * c.d_model * 2);
    L.qkv = take(M * qkv_width(c) * 2);
    L.attn = take(M * c.n_q_heads * c.head_dim * 2);
    L.h = take(M * c.d_model * 4);  // fp32 residual stream inside the layer
    L.act = take(M * c.ffn_dim * 2);
    L.rope = take(M * (c.head_dim / 2) * 8);
    L.meta = take(meta_ints(c, C, B) * 4);
    L.part_o = take(B > 0 ? static_cast<size_t>(W) * c.n_q_heads * c.head_dim * 4 : 0);
    L.part_ml = take(B > 0 ? static_cast<size_t>(W) * c.n_q_heads * 2 * 4 : 0);
    const size_t crows = static_cast<size_t>(chunk_item_cap(c, C)) * c.n_kv_heads * 256;
    L.cpart_o = take(crows * c.head_dim * 4);
    L.cpart_ml = take(crows * 2 * 4);
    L.gemm_part = off;  // split-K partials take the rest of the workspace
    L.end_fixed = off;
    return L;
}

size_t gemm_partial_bytes(const slw_model_cfg& c, int M) {
    size_t b = 0;
    b = std::max(b, plan_gemm(M, qkv_width(c), c.d_model).partial_bytes);
    b = std::max(b, plan_gemm(M, c.d_model, c.n_q_heads * c.head_dim).partial_bytes);
    b = std::max(b, plan_gemm(M, 2 * c.ffn_dim, c.d_model).partial_bytes);
    b = std::max(b, plan_gemm(M, c.d_model, c.ffn_dim).partial_bytes);
    return b;
}

int check_cfg(const slw_model_cfg& c) {
    if (c.n_layers < 1) return fail(SLW_EINVAL, "n_layers must be >= 1");
    if (c.head_dim != 64 && c.head_dim != 128) return fail(SLW_EUNSUPPORTED, "head_dim must be 64 or 128");
    if (c.n_q_heads < 1 || c.n_kv_heads < 1 || c.n_q_heads % c.n_kv_heads)
        return fail(SLW_EINVAL, "n_q_heads must be a positive multiple of n_kv_heads");
    const int group = c.n_q_heads / c.n_kv_heads;
    if (group > 16 || (group & (group - 1))) return fail(SLW_EUNSUPPORTED, "GQA group must be 1, 2, 4, 8 or 16");
    if (c.d_model < 128 || c.d_model % 128 || c.d_model > 8192)
        return fail(SLW_EUNSUPPORTED, "d_model must be a multiple of 128 in [128, 8192]");
    if (c.ffn_dim < 64 || c.ffn_dim % 64) return fail(SLW_EUNSUPPORTED, "ffn_dim must be a multiple of 64");
    if (qkv_width(c) % 128) return fail(SLW_EUNSUPPORTED, "(Hq + 2 Hkv) * hd must be a multiple of 128");
    if ((c.n_q_heads * c.head_dim) % 64) return fail(SLW_EUNSUPPORTED, "Hq * hd must be a multiple of 64");
    if (c.block_size != 16) return fail(SLW_EUNSUPPORTED, "block_size must be 16");
    if (c.max_pos < 1 || c.max_pos > (1 << 20)) return fail(SLW_EINVAL, "max_pos out of range");
    if (!(c.rms_eps > 0.f) || !(c.rope_theta > 0.f)) return fail(SLW_EINVAL, "rms_eps and rope_theta must be > 0");
    return SLW_OK;
}

// The iteration's events order work on this device only: a staging event
// tells the host that the set-up kernel has finished reading a pinned buffer
// (nothing the GPU wrote has to reach the host), and the fork and join
// events order the two streams' kernels.  Without the system-scope fence an
// event record does no cache write-back and invalidation (the CUs sat idle
// for 6-11 us at each record): 8B-layer sweep +1.4%, chat mix +1.6%.
constexpr unsigned kSyncEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;

int ensure_hip(slw_ctx* ctx) {
    if (ctx->hip_ready) return SLW_OK;
    for (int i = 0; i < kRing; ++i) HIP_TRY(hipEventCreateWithFlags(&ctx->staged[i], kSyncEventFlags));
    HIP_TRY(hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking));
    ctx->fork_ev.assign(ctx->cfg.n_layers, nullptr);
    ctx->join_ev.assign(ctx->cfg.n_layers, nullptr);
    for (int l = 0; l < ctx->cfg.n_layers; ++l) {
        HIP_TRY(hipEventCreateWithFlags(&ctx->fork_ev[l], kSyncEventFlags));
        HIP_TRY(hipEventCreateWithFlags(&ctx->join_ev[l], kSyncEventFlags));
    }
    ctx->hip_ready = true;
    return SLW_OK;
}

// Pinned buffer of the next ring slot with room for n ints (waits for its
// last copy).  The buffers are coherent and mapped: the iteration's first
// kernel reads them over the bus, so the upload needs no copy engine.
int next_staging(slw_ctx* ctx, size_t n, int32_t** buf, int* slot_out) {
    const int slot = ctx->ring;
    ctx->ring = (ctx->ring + 1) % kRing;
    HIP_TRY(hipEventSynchronize(ctx->staged[slot]));
    if (ctx->staging_cap[slot] < n) {
        if (ctx->staging[slot]) HIP_TRY(hipHostFree(ctx->staging[slot]));
        ctx->staging[slot] = nullptr;
        ctx->staging_dev[slot] = nullptr;
        ctx->staging_cap[slot] = 0;
        size_t cap = std::max<size_t>(n, 1 << 16);
        void* p = nullptr;
        HIP_TRY(hipHostMalloc(&p, cap * 4, hipHostMallocMapped | hipHostMallocCoherent));
        ctx->staging[slot] = static_cast<int32_t*>(p);
        void* dp = nullptr;
        HIP_TRY(hipHostGetDevicePointer(&dp, p, 0));
        ctx->staging_dev[slot] = static_cast<int32_t*>(dp);
        ctx->staging_cap[slot] = cap;
    }
    *buf = ctx->staging[slot];
    *slot_out = slot;
    return SLW_OK;
}

constexpr int kStages = SLW_N_STAGES;

int ensure_stage_events(slw_ctx* ctx) {
    const size_t need = static_cast<size_t>(ctx->stage_depth) * ctx->cfg.n_layers * (kStages + 1);
    while (ctx->stage_ev.size() < need) {
        hipEvent_t e;
        HIP_TRY(hipEventCreate(&e));
        ctx->stage_ev.push_back(e);
    }
    return SLW_OK;
}

int enqueue_iteration(slw_ctx* ctx, const slw_batch* bt, const void* x_in, void* x_out, void* ws,
                      const Layout& L, hipStream_t stream, bool no_alloc);

// One iteration: validation, KV reservation (all or nothing), then the
// metadata, its upload and the kernels.  A failure after the reservation
// returns the reserved blocks, so a failed call leaves the block manager as
// it found it.  no_alloc: the workspace is the static array, the metadata is
// copied with hipMemcpyAsync from host memory the context holds, both
// attentions run on `stream` and no stage events are recorded, so the call
// creates no HIP object and allocates no memory of any kind on the device or
// pinned on the host.
int mixed_iteration_impl(slw_ctx* ctx, const slw_batch* bt, const void* x_in, void* x_out, void* ws,
                         size_t ws_bytes, hipStream_t stream, bool no_alloc = false) {
    const slw_model_cfg& c = ctx->cfg;
    if (!bt) return fail(SLW_EINVAL, "null batch");
    const int C = bt->C, B = bt->B;
    if (C < 0 || B < 0) return fail(SLW_EINVAL, "negative C or B");
    if (C == 0 && B == 0) {
        ctx->last_slots.clear();
        return SLW_OK;
    }
    if (!ctx->kv_ready) return fail(SLW_EINVAL, "KV pools not attached (slw_kv_init)");
    for (int l = 0; l < c.n_layers; ++l)
        if (!ctx->have_w[l]) return fail(SLW_EINVAL, "weights of layer %d not set", l);
    if (!x_in || !x_out || !ws) return fail(SLW_EINVAL, "null device buffer");
    if (B > 0 && (!bt->decode_seqs || !bt->context_lens)) return fail(SLW_EINVAL, "null decode arrays");

    // validation; the chunk rows' prefills in row order
    std::vector<Prefill>& pre = ctx->prefills;
    pre.clear();
    if (bt->n_prefill > 1) {
        if (bt->n_prefill > SLW_MAX_PREFILLS) return fail(SLW_ERANGE, "n_prefill %d above %d", bt->n_prefill, SLW_MAX_PREFILLS);
        if (!bt->prefill_seqs || !bt->prefix_lens || !bt->chunk_lens) return fail(SLW_EINVAL, "null prefill arrays");
        int64_t rows = 0;
        for (int i = 0; i < bt->n_prefill; ++i) {
            if (bt->chunk_lens[i] < 1) return fail(SLW_EINVAL, "prefill %d has chunk_len %d", i, bt->chunk_lens[i]);
            pre.push_back({bt->prefill_seqs[i], bt->prefix_lens[i], bt->chunk_lens[i], static_cast<int32_t>(rows)});
            rows += bt->chunk_lens[i];
        }
        if (rows != C) return fail(SLW_EINVAL, "chunk_lens add up to %lld, C is %d", (long long)rows, C);
    } else if (C > 0) {
        pre.push_back({bt->prefill_seq, bt->prefix_len, C, 0});
    }
    std::vector<std::pair<int64_t, int32_t>> req;
    req.reserve(B + pre.size());
    std::unordered_set<int64_t> seen;
    seen.reserve(2 * (B + pre.size()) + 2);
    for (const Prefill& f : pre) {
        if (f.prefix < 0) return fail(SLW_EINVAL, "negative prefix_len");
        if (static_cast<int64_t>(f.prefix) + f.c > c.max_pos) return fail(SLW_ERANGE, "prefix_len + chunk exceeds max_pos");
        if (!ctx->kv.exists(f.seq)) return fail(SLW_EINVAL, "prefill sequence %lld unknown", (long long)f.seq);
        if (!seen.insert(f.seq).second)
            return fail(SLW_EINVAL, "sequence %lld appears twice in the batch", (long long)f.seq);
        if (ctx->kv.reserved(f.seq) < f.prefix)
            return fail(SLW_EINVAL, "prefill sequence %lld holds %d positions, prefix_len is %d", (long long)f.seq,
                        ctx->kv.reserved(f.seq), f.prefix);
        req.emplace_back(f.seq, f.prefix + f.c);
    }
    {
        for (int b = 0; b < B; ++b) {
            const int64_t id = bt->decode_seqs[b];
            const int32_t L = bt->context_lens[b];
            if (!ctx->kv.exists(id)) return fail(SLW_EINVAL, "decode sequence %lld unknown", (long long)id);
            if (!seen.insert(id).second)
                return fail(SLW_EINVAL, "sequence %lld appears twice in the batch", (long long)id);
            if (L < 0 || L + 1 > c.max_pos) return fail(SLW_ERANGE, "context_len %d out of range", L);
            if (ctx->kv.reserved(id) < L)
                return fail(SLW_EINVAL, "decode sequence %lld holds %d positions, context_len is %d",
                            (long long)id, ctx->kv.reserved(id), L);
            req.emplace_back(id, L + 1);
        }
    }
    const Layout L = layout(c, C, B);
    const size_t gpart = gemm_partial_bytes(c, C + B);
    if (ws_bytes < L.end_fixed + gpart)
        return fail(SLW_ENOMEM, "%s holds %zu bytes, this iteration needs %zu",
                    no_alloc ? "the static workspace (SLW_STATIC_WS_BYTES)" : "the workspace", ws_bytes,
                    L.end_fixed + gpart);
    int rc = SLW_OK;
    if (!no_alloc) {
        rc = ensure_hip(ctx);
        if (rc) return rc;
        if (ctx->stage_depth > 0) {
            rc = ensure_stage_events(ctx);
            if (rc) return rc;
        }
    }
    KvManager::Undo undo;
    rc = ctx->kv.reserve_all(req, &undo);
    if (rc) return rc;
    rc = enqueue_iteration(ctx, bt, x_in, x_out, ws, L, stream, no_alloc);
    if (rc) ctx->kv.rollback(undo);
    return rc;
}

// Metadata, upload and kernels of an iteration whose blocks are reserved.
// Query tiles of the chunk rows: each prefill's rows cut into tiles of
// chunk_tile_positions(group) positions (a tile never mixes sequences).
// Tile q: first chunk row, rows, first position and, when wanted, the offset
// of its sequence's block table (bt_of_prefill[i] for prefill i).
void query_tiles(const slw_model_cfg& c, const std::vector<Prefill>& pre, std::vector<int32_t>& row0,
                 std::vector<int32_t>& rows, std::vector<int32_t>& pos0, std::vector<int32_t>* bt,
                 const std::vector<int32_t>& bt_of_prefill) {
    const int pwg = chunk_tile_positions(c.n_q_heads / c.n_kv_heads);
    row0.clear();
    rows.clear();
    pos0.clear();
    if (bt) bt->clear();
    for (size_t i = 0; i < pre.size(); ++i)
        for (int j = 0; j < pre[i].c; j += pwg) {
            row0.push_back(pre[i].row0 + j);
            rows.push_back(std::min(pwg, pre[i].c - j));
            pos0.push_back(pre[i].prefix + j);
            if (bt) bt->push_back(bt_of_prefill[i]);
        }
}

// Decode attention work.  The keys of all decodes (decode b attends to
// context_lens[b] + 1 of them), laid end to end with each decode's range
// padded to a multiple of 64, are cut into equal runs (multiples of 64 keys,
// so that every item starts on a page pair; at least kDecodeMinKeys each, at
// most decode_slot_cap(c) runs), one per wave of each kv head; a run that
// crosses decodes becomes one item per decode it touches, and padding alone
// makes no item.  Items come out in decode order, so each decode's items are
// contiguous for the merge.
int plan_decode(const slw_model_cfg& c, int B, const int32_t* context_lens, DecodePlan& p) {
    p.b.clear();
    p.kb.clear();
    p.ke.clear();
    p.off.assign(B + 1, 0);
    p.slot_off.assign(1, 0);
    if (B <= 0) return SLW_OK;
    int64_t padded = 0;
    for (int b = 0; b < B; ++b) padded += ceil_div(context_lens[b] + 1, 64) * 64;
    const int64_t want = std::min<int64_t>(decode_slot_cap(c), std::max<int64_t>(1, padded / kDecodeMinKeys));
    const int64_t per = ceil_div(ceil_div(padded, want), 64) * 64;
    const int n_slots = static_cast<int>(ceil_div(padded, per));
    p.slot_off.clear();
    int b = 0;
    int64_t start_b = 0;  // first key of decode b in the padded layout
    for (int sl = 0; sl < n_slots; ++sl) {
        p.slot_off.push_back(static_cast<int32_t>(p.b.size()));
        int64_t r0 = sl * per;
        const int64_t r1 = std::min(padded, r0 + per);
        while (r0 < r1) {
            const int32_t len = context_lens[b] + 1;
            const int64_t span = ceil_div(len, 64) * 64;
            if (r0 >= start_b + span) {  // past decode b
                start_b += span;
                p.off[++b] = static_cast<int32_t>(p.b.size());
                continue;
            }
            const int64_t k0 = r0 - start_b, k1 = std::min<int64_t>(r1 - start_b, span);
            if (k0 < len) {
                p.b.push_back(b);
                p.kb.push_back(static_cast<int32_t>(k0));
                p.ke.push_back(static_cast<int32_t>(std::min<int64_t>(k1, len)));
            }
            r0 = start_b + k1;
        }
    }
    p.slot_off.push_back(static_cast<int32_t>(p.b.size()));
    while (b < B) p.off[++b] = static_cast<int32_t>(p.b.size());
    if (static_cast<int>(p.b.size()) > decode_work_cap(c, B) || n_slots > decode_slot_cap(c))
        return fail(SLW_EINVAL, "internal: decode work %zu / slots %d above cap", p.b.size(), n_slots);
    for (int d = 0; d < B; ++d) {  // the items of each decode tile its keys
        int64_t at = 0;
        for (int i = p.off[d]; i < p.off[d + 1]; ++i) {
            if (p.b[i] != d || p.kb[i] != at || p.ke[i] <= at) return fail(SLW_EINVAL, "internal: decode plan");
            at = p.ke[i];
        }
        if (at != context_lens[d] + 1) return fail(SLW_EINVAL, "internal: decode plan");
    }
    return SLW_OK;
}

// Chunk attention work over query tiles q (first position qt_pos0[q],
// qt_rows[q] rows, keys 0 .. qt_pos0[q] + qt_rows[q] - 1).  Whole query tiles
// where they balance: the tiles, longest first, each go to the least loaded
// of `want` work-groups (LPT); when the largest load stays within
// kChunkWholeSlack of an equal share, no tile is split and nothing is merged
// (long prompts: many tiles of similar length).  Otherwise (fewer tiles than
// work-groups, or tiles of very different lengths, as at the start of a
// prompt) the 64-key tiles of every query tile, laid end to end, are cut into
// equal runs, one per work-group of each kv head; a run that crosses query
// tiles becomes one item per query tile it touches.  Items stay in query-tile
// order; slot_items lists each work-group's items.
int plan_chunk(const slw_model_cfg& c, int C, const std::vector<int32_t>& qt_pos0, const std::vector<int32_t>& qt_rows,
               ChunkPlan& p) {
    const int n_qt = static_cast<int>(qt_pos0.size());
    p.items.clear();
    p.slot_off.clear();
    p.slot_items.clear();
    p.whole = false;
    auto key_end = [&](int q) { return static_cast<int64_t>(qt_pos0[q]) + qt_rows[q]; };
    std::vector<int64_t> tile_end(n_qt + 1, 0);
    for (int q = 0; q < n_qt; ++q) tile_end[q + 1] = tile_end[q] + ceil_div(key_end(q), 64);
    const int64_t total_tiles = tile_end[n_qt];
    std::vector<int32_t>& it = p.items;
    int n_slots = 0;
    if (n_qt > 0) {
        const int64_t want = std::min<int64_t>(chunk_slot_cap(c), std::max<int64_t>(1, total_tiles / kChunkMinTiles));
        const int64_t per = ceil_div(total_tiles, want);
        if (n_qt >= want) {
            std::vector<int32_t> order(n_qt);
            for (int q = 0; q < n_qt; ++q) order[q] = q;
            auto len = [&](int q) { return tile_end[q + 1] - tile_end[q]; };
            std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return len(x) > len(y); });
            std::vector<int64_t> load(want, 0);
            std::vector<int32_t> owner(n_qt);
            for (int q : order) {
                const int g = static_cast<int>(std::min_element(load.begin(), load.end()) - load.begin());
                load[g] += len(q);
                owner[q] = g;
            }
            const int64_t mx = *std::max_element(load.begin(), load.end());
            if (mx * kChunkWholeSlackDen <= per * kChunkWholeSlackNum) {
                p.whole = true;
                n_slots = static_cast<int>(want);
                for (int q = 0; q < n_qt; ++q) {
                    it.push_back(q);
                    it.push_back(0);
                    it.push_back(static_cast<int32_t>(key_end(q)));
                }
                p.slot_off.assign(n_slots + 1, 0);
                for (int q = 0; q < n_qt; ++q) ++p.slot_off[owner[q] + 1];
                for (int g = 0; g < n_slots; ++g) p.slot_off[g + 1] += p.slot_off[g];
                p.slot_items.resize(n_qt);
                std::vector<int32_t> fill(p.slot_off.begin(), p.slot_off.end() - 1);
                for (int q = 0; q < n_qt; ++q) p.slot_items[fill[owner[q]]++] = q;
            }
        }
        if (!p.whole) {
            n_slots = static_cast<int>(ceil_div(total_tiles, per));
            p.slot_off.resize(n_slots + 1);
            int q = 0;
            for (int sl = 0; sl < n_slots; ++sl) {
                p.slot_off[sl] = static_cast<int32_t>(it.size() / 3);
                int64_t t0 = sl * per;
                const int64_t t1 = std::min(total_tiles, t0 + per);
                while (t0 < t1) {
                    while (tile_end[q + 1] <= t0) ++q;
                    const int64_t seg_end = std::min(t1, tile_end[q + 1]);
                    it.push_back(q);
                    it.push_back(static_cast<int32_t>((t0 - tile_end[q]) * 64));
                    it.push_back(static_cast<int32_t>(std::min(key_end(q), (seg_end - tile_end[q]) * 64)));
                    t0 = seg_end;
                }
            }
            p.slot_off[n_slots] = static_cast<int32_t>(it.size() / 3);
            p.slot_items.resize(it.size() / 3);
            for (size_t i = 0; i < p.slot_items.size(); ++i) p.slot_items[i] = static_cast<int32_t>(i);
        }
    } else {
        p.slot_off.assign(1, 0);
    }
    const int n_items = static_cast<int>(it.size() / 3);
    p.qt_off.assign(n_qt + 1, 0);
    for (int q = 0, i = 0; q <= n_qt; ++q) {
        while (i < n_items && it[3 * i] < q) ++i;
        p.qt_off[q] = i;
    }
    if (n_items > chunk_item_cap(c, C) || n_slots > chunk_slot_cap(c))
        return fail(SLW_EINVAL, "internal: chunk items %d / slots %d above cap", n_items, n_slots);
    for (int q = 0; q < n_qt; ++q) {  // the items of each query tile tile its key range
        int64_t at = 0;
        for (int i = p.qt_off[q]; i < p.qt_off[q + 1]; ++i) {
            if (it[3 * i + 1] != at || it[3 * i + 2] <= at) return fail(SLW_EINVAL, "internal: chunk plan");
            at = it[3 * i + 2];
        }
        if (at != key_end(q)) return fail(SLW_EINVAL, "internal: chunk plan");
    }
    return SLW_OK;
}

int enqueue_iteration(slw_ctx* ctx, const slw_batch* bt, const void* x_in, void* x_out, void* ws,
                      const Layout& L, hipStream_t stream, bool no_alloc) {
    const slw_model_cfg& c = ctx->cfg;
    const int C = bt->C, B = bt->B;
    const std::vector<Prefill>& pre = ctx->prefills;
    int rc = SLW_OK;

    // ---- metadata (host) ----
    const int M = C + B;

    std::vector<int32_t>& m = ctx->meta;
    m.clear();
    m.reserve(meta_ints(c, C, B));
    // slot[M], pos[M]
    std::vector<int32_t>& slots = ctx->slots_build;
    slots.resize(M);
    for (const Prefill& f : pre)
        for (int j = 0; j < f.c; ++j) slots[f.row0 + j] = ctx->kv.slot(f.seq, f.prefix + j);
    for (int b = 0; b < B; ++b) slots[C + b] = ctx->kv.slot(bt->decode_seqs[b], bt->context_lens[b]);
    m.insert(m.end(), slots.begin(), slots.end());
    for (const Prefill& f : pre)
        for (int j = 0; j < f.c; ++j) m.push_back(f.prefix + j);
    for (int b = 0; b < B; ++b) m.push_back(bt->context_lens[b]);
    const size_t o_kvlen = m.size();
    for (int b = 0; b < B; ++b) m.push_back(bt->context_lens[b] + 1);
    const size_t o_btoff = m.size();
    m.resize(m.size() + B + 1);
    const size_t o_bt = m.size();
    for (int b = 0; b < B; ++b) {
        m[o_btoff + b] = static_cast<int32_t>(m.size() - o_bt);
        const auto& t = ctx->kv.table(bt->decode_seqs[b]);
        const int nb = static_cast<int>(ceil_div(bt->context_lens[b] + 1, 16));
        m.insert(m.end(), t.begin(), t.begin() + nb);
    }
    m[o_btoff + B] = static_cast<int32_t>(m.size() - o_bt);
    // block tables of the prefills, one after the other
    const size_t o_pre = m.size();
    std::vector<int32_t> pre_bt(pre.size());
    for (size_t i = 0; i < pre.size(); ++i) {
        pre_bt[i] = static_cast<int32_t>(m.size() - o_pre);
        const auto& t = ctx->kv.table(pre[i].seq);
        const int nb = static_cast<int>(ceil_div(pre[i].prefix + pre[i].c, 16));
        m.insert(m.end(), t.begin(), t.begin() + nb);
    }
    // Decode attention work (plan_decode).
    const size_t o_workb = m.size();
    DecodePlan& dp = ctx->dplan;
    if ((rc = plan_decode(c, B, bt->context_lens, dp))) return rc;
    const int n_work = static_cast<int>(dp.b.size()), n_dslots = static_cast<int>(dp.slot_off.size()) - 1;
    int64_t chunk_pairs = 0;  // (query, key) pairs of the chunk rows: c p + c (c + 1) / 2 per prefill
    for (const auto& q : pre) chunk_pairs += int64_t{q.c} * q.prefix + int64_t{q.c} * (q.c + 1) / 2;
    m.insert(m.end(), dp.b.begin(), dp.b.end());
    m.insert(m.end(), dp.kb.begin(), dp.kb.end());
    m.insert(m.end(), dp.ke.begin(), dp.ke.end());
    m.insert(m.end(), dp.off.begin(), dp.off.end());
    m.insert(m.end(), dp.slot_off.begin(), dp.slot_off.end());
    // Chunk attention work.  Each prefill's rows are cut into query tiles of
    // pwg positions (a tile never mixes sequences); query tile q covers chunk
    // rows qt_row0 .. + qt_rows at positions from qt_pos0 on and reads the
    // block table at qt_bt, over keys 0 .. qt_pos0 + qt_rows - 1; plan_chunk
    // hands the tiles out to the work-groups.  A query tile covered by one
    // item is written directly, one covered by several is combined by the
    // merge kernel.
    std::vector<int32_t> qt_row0, qt_rows, qt_pos0, qt_bt;
    query_tiles(c, pre, qt_row0, qt_rows, qt_pos0, &qt_bt, pre_bt);
    const int n_qt = static_cast<int>(qt_row0.size());
    if (n_qt > chunk_tiles(c, C)) return fail(SLW_EINVAL, "internal: %d query tiles above cap", n_qt);
    ChunkPlan& cp = ctx->cplan;
    if ((rc = plan_chunk(c, C, qt_pos0, qt_rows, cp))) return rc;
    const std::vector<int32_t>& it = cp.items;
    const std::vector<int32_t>& slot_off = cp.slot_off;
    const std::vector<int32_t>& slot_items = cp.slot_items;
    const std::vector<int32_t>& qt_off = cp.qt_off;
    const int n_items = static_cast<int>(it.size() / 3), n_slots = static_cast<int>(slot_off.size()) - 1;
    const size_t o_item = m.size();
    m.resize(m.size() + 3 * static_cast<size_t>(n_items));
    for (int i = 0; i < n_items; ++i) {
        m[o_item + i] = it[3 * i];
        m[o_item + n_items + i] = it[3 * i + 1];
        m[o_item + 2 * n_items + i] = it[3 * i + 2];
    }
    const size_t o_slot = m.size();
    m.insert(m.end(), slot_off.begin(), slot_off.end());
    const size_t o_slot_items = m.size();
    m.insert(m.end(), slot_items.begin(), slot_items.end());
    const size_t o_qtoff = m.size();
    m.insert(m.end(), qt_off.begin(), qt_off.end());
    const size_t o_qt = m.size();  // [4][n_qt]: first row, rows, first position, block-table offset
    m.insert(m.end(), qt_row0.begin(), qt_row0.end());
    m.insert(m.end(), qt_rows.begin(), qt_rows.end());
    m.insert(m.end(), qt_pos0.begin(), qt_pos0.end());
    m.insert(m.end(), qt_bt.begin(), qt_bt.end());

    if (m.size() > meta_ints(c, C, B)) return fail(SLW_EINVAL, "internal: metadata %zu ints above its region", m.size());

    // ---- upload ----
    char* wsb = static_cast<char*>(ws);
    int32_t* dmeta = reinterpret_cast<int32_t*>(wsb + L.meta);
    float2* rope = reinterpret_cast<float2*>(wsb + L.rope);
    if (no_alloc) {
        // From the context's host vector, which the next call refills: a copy
        // from pageable memory may still be reading it when hipMemcpyAsync
        // returns, so the stream is synchronised right after it.
        HIP_TRY(hipMemcpyAsync(dmeta, m.data(), m.size() * 4, hipMemcpyHostToDevice, stream));
        HIP_TRY(hipStreamSynchronize(stream));
        launch_iteration_setup(dmeta, nullptr, 0, dmeta + M, rope, M, c.head_dim, static_cast<double>(c.rope_theta),
                               stream);
        HIP_TRY(hipGetLastError());
    } else {
        int32_t* stage = nullptr;
        int slot = 0;
        rc = next_staging(ctx, m.size(), &stage, &slot);
        if (rc) return rc;
        std::memcpy(stage, m.data(), m.size() * 4);
        // metadata copy and RoPE table (positions follow the M slots) in one kernel
        launch_iteration_setup(dmeta, ctx->staging_dev[slot], m.size(), ctx->staging_dev[slot] + M, rope, M,
                               c.head_dim, static_cast<double>(c.rope_theta), stream);
        HIP_TRY(hipGetLastError());
        HIP_TRY(hipEventRecord(ctx->staged[slot], stream));
    }

    const int32_t* d_slot = dmeta;
    void* xn = wsb + L.xn;
    void* qkv = wsb + L.qkv;
    void* attn = wsb + L.attn;
    void* hbuf = wsb + L.h;
    void* act = wsb + L.act;
    void* gpartp = wsb + L.gemm_part;

    const int d = c.d_model, hq = c.n_q_heads, hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
    const int qw = qkv_width(c);
    const GemmPlan p_qkv = plan_gemm(M, qw, d);
    const GemmPlan p_o = plan_gemm(M, d, hq * hd);
    const GemmPlan p_gu = plan_gemm(M, 2 * F, d);
    const GemmPlan p_d = plan_gemm(M, d, F);
    const size_t layer_pool = static_cast<size_t>(ctx->kv.num_blocks()) * hkv * hd * 16 * 2;

    const bool timing = !no_alloc && ctx->stage_depth > 0;
    size_t set_base = 0;
    int set = 0;
    if (timing) {
        set = static_cast<int>(ctx->stage_iter % ctx->stage_depth);
        set_base = static_cast<size_t>(set) * c.n_layers * (kStages + 1);
        ctx->stage_mask[set] = 0;
    }
    auto mark = [&](int l, int stage) -> int {
        if (timing)
            HIP_TRY(hipEventRecord(ctx->stage_ev[set_base + static_cast<size_t>(l) * (kStages + 1) + stage], stream));
        return SLW_OK;
    };

    for (int l = 0; l < c.n_layers; ++l) {
        const slw_layer_weights& wl = ctx->w[l];
        const void* cur = l == 0 ? x_in : x_out;
        void* kp = static_cast<char*>(ctx->k_pool) + l * layer_pool;
        void* vp = static_cast<char*>(ctx->v_pool) + l * layer_pool;

        if ((rc = mark(l, 0))) return rc;
        launch_rmsnorm(cur, false, wl.g1, xn, M, d, c.rms_eps, stream);
        if ((rc = mark(l, 1))) return rc;  // the RoPE table stage is empty: the setup kernel fills the table
        if ((rc = mark(l, 2))) return rc;
        {
            GemmArgs ga{xn, wl.wqkv, qkv, nullptr, M, qw, d, d, qw, EPI_QKV};
            ga.rope_cs = rope;
            ga.slot = d_slot;
            ga.k_pool = kp;
            ga.v_pool = vp;
            ga.hq = hq;
            ga.hkv = hkv;
            ga.hd = hd;
            launch_gemm(ga, p_qkv, gpartp, stream);
        }
        if ((rc = mark(l, 3))) return rc;
        // Both attentions in one launch, or on two streams for a long
        // chunk (see kTwoStreamMinPairs); per-stage events separate them.
        ChunkAttnArgs ca{};
        if (C > 0) {
            ca.qkv = qkv;
            ca.out = attn;
            ca.k_pool = kp;
            ca.v_pool = vp;
            ca.bt = dmeta + o_pre;
            ca.item_qt = dmeta + o_item;
            ca.item_kb = dmeta + o_item + n_items;
            ca.item_ke = dmeta + o_item + 2 * n_items;
            ca.qt_off = dmeta + o_qtoff;
            ca.part_o = reinterpret_cast<float*>(wsb + L.cpart_o);
            ca.part_ml = reinterpret_cast<float*>(wsb + L.cpart_ml);
            ca.c = C;
            ca.n_qt = n_qt;
            ca.qt_row0 = dmeta + o_qt;
            ca.qt_rows = dmeta + o_qt + n_qt;
            ca.qt_pos0 = dmeta + o_qt + 2 * n_qt;
            ca.qt_bt = dmeta + o_qt + 3 * n_qt;
            ca.hq = hq;
            ca.hkv = hkv;
            ca.hd = hd;
            ca.ld_qkv = qw;
            ca.slot_off = dmeta + o_slot;
            ca.slot_items = dmeta + o_slot_items;
            ca.n_items = n_items;
            ca.n_slots = n_slots;
            ca.split = n_items > n_qt ? 1 : 0;
        }
        DecodeAttnArgs da{};
        if (B > 0) {
            da.q = static_cast<const char*>(qkv) + static_cast<size_t>(C) * qw * 2;
            da.out = static_cast<char*>(attn) + static_cast<size_t>(C) * hq * hd * 2;
            da.k_pool = kp;
            da.v_pool = vp;
            da.kv_len = dmeta + o_kvlen;
            da.bt_off = dmeta + o_btoff;
            da.bt = dmeta + o_bt;
            da.work_b = dmeta + o_workb;
            da.work_kb = dmeta + o_workb + n_work;
            da.work_ke = dmeta + o_workb + 2 * n_work;
            da.work_off = dmeta + o_workb + 3 * n_work;
            da.slot_off = dmeta + o_workb + 3 * n_work + B + 1;
            da.n_slots = n_dslots;
            da.part_o = reinterpret_cast<float*>(wsb + L.part_o);
            da.part_ml = reinterpret_cast<float*>(wsb + L.part_ml);
            da.b = B;
            da.n_work = n_work;
            da.hq = hq;
            da.hkv = hkv;
            da.hd = hd;
            da.ld_q = qw;
        }
        if (timing) {
            if (C > 0) launch_chunk_attention(ca, stream);
            if ((rc = mark(l, 4))) return rc;
            if (B > 0) launch_decode_attention_split(da, stream);
        } else if (C > 0 && B > 0 && !no_alloc && chunk_pairs >= kTwoStreamMinPairs) {
            HIP_TRY(hipEventRecord(ctx->fork_ev[l], stream));
            HIP_TRY(hipStreamWaitEvent(ctx->side, ctx->fork_ev[l], 0));
            launch_chunk_attention(ca, stream);
            launch_decode_attention_split(da, ctx->side);
            HIP_TRY(hipEventRecord(ctx->join_ev[l], ctx->side));
            HIP_TRY(hipStreamWaitEvent(stream, ctx->join_ev[l], 0));
        } else {
            launch_attention(ca, da, stream);
        }
        if ((rc = mark(l, 5))) return rc;
        launch_attention_merge(&ca, &da, stream);
        if ((rc = mark(l, 6))) return rc;
        launch_gemm(GemmArgs{attn, wl.wo, hbuf, cur, M, d, hq * hd, hq * hd, d, EPI_RESID_F32OUT}, p_o, gpartp,
                    stream);
        if ((rc = mark(l, 7))) return rc;
        launch_rmsnorm(hbuf, true, wl.g2, xn, M, d, c.rms_eps, stream);
        if ((rc = mark(l, 8))) return rc;
        launch_gemm(GemmArgs{xn, wl.wgu, act, nullptr, M, 2 * F, d, d, F, EPI_SWIGLU}, p_gu, gpartp, stream);
        if ((rc = mark(l, 9))) return rc;
        launch_gemm(GemmArgs{act, wl.wd, x_out, hbuf, M, d, F, F, d, EPI_RESID_F32IN}, p_d, gpartp, stream);
        if ((rc = mark(l, 10))) return rc;
    }
    HIP_TRY(hipGetLastError());
    if (timing) {
        // the merge stage (5) runs when decodes or split chunk query tiles need it
        const bool merge = B > 0 || (C > 0 && n_items > n_qt);
        ctx->stage_mask[set] = 0x3FFu & ~(C > 0 ? 0u : (1u << 3)) & ~(B > 0 ? 0u : (1u << 4)) &
                               ~(merge ? 0u : (1u << 5));
        ++ctx->stage_iter;
    }
    ctx->last_slots.swap(slots);
    return SLW_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" int slw_create(const slw_model_cfg* cfg, slw_ctx** out) {
    return guarded([&] {
        if (!cfg || !out) return fail(SLW_EINVAL, "null argument");
        *out = nullptr;
        int rc = check_cfg(*cfg);
        if (rc) return rc;
        auto ctx = std::make_unique<slw_ctx>();
        ctx->cfg = *cfg;
        ctx->w.assign(cfg->n_layers, slw_layer_weights{});
        ctx->have_w.assign(cfg->n_layers, 0);
        *out = ctx.release();
        return SLW_OK;
    });
}

extern "C" int slw_destroy(slw_ctx* ctx) {
    delete ctx;
    return SLW_OK;
}

extern "C" int slw_attention_plan(const slw_model_cfg* cfg, int32_t B, const int32_t* context_lens,
                                  int32_t n_prefill, const int32_t* prefix_lens, const int32_t* chunk_lens,
                                  int64_t out[12]) {
    return guarded([&] {
        if (!cfg || !out || (B > 0 && !context_lens) || (n_prefill > 0 && (!prefix_lens || !chunk_lens)))
            return fail(SLW_EINVAL, "null argument");
        int rc = check_cfg(*cfg);
        if (rc) return rc;
        if (B < 0 || n_prefill < 0 || n_prefill > SLW_MAX_PREFILLS)
            return fail(SLW_EINVAL, "B >= 0 and 0 <= n_prefill <= %d", SLW_MAX_PREFILLS);
        std::vector<Prefill> pre;
        int C = 0;
        for (int i = 0; i < n_prefill; ++i) {
            if (chunk_lens[i] < 1 || prefix_lens[i] < 0 ||
                static_cast<int64_t>(prefix_lens[i]) + chunk_lens[i] > cfg->max_pos)
                return fail(SLW_EINVAL, "prefill %d: chunk >= 1, prefix >= 0, prefix + chunk <= max_pos", i);
            pre.push_back(Prefill{i, prefix_lens[i], chunk_lens[i], C});
            C += chunk_lens[i];
        }
        for (int b = 0; b < B; ++b)
            if (context_lens[b] < 0 || context_lens[b] >= cfg->max_pos)
                return fail(SLW_EINVAL, "decode %d: context in [0, max_pos)", b);
        DecodePlan dp;
        ChunkPlan cp;
        std::vector<int32_t> row0, rows, pos0;
        query_tiles(*cfg, pre, row0, rows, pos0, nullptr, {});
        if ((rc = plan_decode(*cfg, B, context_lens, dp))) return rc;
        if ((rc = plan_chunk(*cfg, C, pos0, rows, cp))) return rc;
        const int dslots = static_cast<int>(dp.slot_off.size()) - 1;
        int64_t dmax = 0, dmin = dslots > 0 ? std::numeric_limits<int64_t>::max() : 0;
        for (int sl = 0; sl < dslots; ++sl) {
            int64_t keys = 0;
            for (int i = dp.slot_off[sl]; i < dp.slot_off[sl + 1]; ++i) keys += dp.ke[i] - dp.kb[i];
            dmax = std::max(dmax, keys);
            dmin = std::min(dmin, keys);
        }
        const int cslots = static_cast<int>(cp.slot_off.size()) - 1;
        int64_t cmax = 0, cmin = cslots > 0 ? std::numeric_limits<int64_t>::max() : 0, ctot = 0;
        for (int g = 0; g < cslots; ++g) {
            int64_t tiles = 0;
            for (int k = cp.slot_off[g]; k < cp.slot_off[g + 1]; ++k) {
                const int i = cp.slot_items[k];
                tiles += ceil_div(cp.items[3 * i + 2], 64) - cp.items[3 * i + 1] / 64;
            }
            cmax = std::max(cmax, tiles);
            cmin = std::min(cmin, tiles);
            ctot += tiles;
        }
        const int64_t v[12] = {static_cast<int64_t>(dp.b.size()), dslots, dmax, dmin,
                               static_cast<int64_t>(rows.size()), static_cast<int64_t>(cp.items.size() / 3), cslots,
                               cp.whole ? 1 : 0, cmax, cmin, ctot, 0};
        for (int i = 0; i < 12; ++i) out[i] = v[i];
        return SLW_OK;
    });
}

extern "C" int slw_gemm_plan(int32_t m, int32_t n, int32_t k, int32_t out[6]) {
    if (!out) return fail(SLW_EINVAL, "null argument");
    if (m < 1 || n < 128 || n % 128 || k < 64 || k % 64)
        return fail(SLW_EINVAL, "m >= 1, n a multiple of 128 and k of 64 (got %d, %d, %d)", m, n, k);
    const GemmPlan p = plan_gemm(m, n, k);
    const int32_t v[6] = {p.cfg, p.bm, p.bn, p.splits, p.sk_workers, p.dp_tiles};
    for (int i = 0; i < 6; ++i) out[i] = v[i];
    return SLW_OK;
}

extern "C" int slw_set_layer_weights(slw_ctx* ctx, int32_t layer, const slw_layer_weights* w) {
    if (!ctx || !w) return fail(SLW_EINVAL, "null argument");
    if (layer < 0 || layer >= ctx->cfg.n_layers) return fail(SLW_ERANGE, "layer %d out of range", layer);
    if (!w->wqkv || !w->wo || !w->wgu || !w->wd || !w->g1 || !w->g2)
        return fail(SLW_EINVAL, "null weight pointer");
    const void* ptrs[6] = {w->wqkv, w->wo, w->wgu, w->wd, w->g1, w->g2};
    for (const void* p : ptrs)
        if (reinterpret_cast<uintptr_t>(p) % 16) return fail(SLW_EINVAL, "weights must be 16-byte aligned");
    ctx->w[layer] = *w;
    ctx->have_w[layer] = 1;
    return SLW_OK;
}

extern "C" int slw_kv_init(slw_ctx* ctx, void* k_pool, void* v_pool, int32_t num_blocks) {
    return guarded([&] {
        if (!ctx || !k_pool || !v_pool) return fail(SLW_EINVAL, "null argument");
        if (num_blocks < 1) return fail(SLW_EINVAL, "num_blocks must be >= 1");
        if (reinterpret_cast<uintptr_t>(k_pool) % 16 || reinterpret_cast<uintptr_t>(v_pool) % 16)
            return fail(SLW_EINVAL, "pools must be 16-byte aligned");
        ctx->k_pool = k_pool;
        ctx->v_pool = v_pool;
        ctx->kv.reset(num_blocks, 16);
        ctx->kv_ready = true;
        return SLW_OK;
    });
}

extern "C" int slw_kv_free_blocks(slw_ctx* ctx, int32_t* n_free) {
    if (!ctx || !n_free) return fail(SLW_EINVAL, "null argument");
    if (!ctx->kv_ready) return fail(SLW_EINVAL, "KV pools not attached");
    *n_free = ctx->kv.free_count();
    return SLW_OK;
}

extern "C" int slw_seq_create(slw_ctx* ctx, int64_t id) {
    return guarded([&] {
        if (!ctx) return fail(SLW_EINVAL, "null context");
        if (!ctx->kv_ready) return fail(SLW_EINVAL, "KV pools not attached");
        return ctx->kv.create(id);
    });
}

extern "C" int slw_seq_free(slw_ctx* ctx, int64_t id) {
    return guarded([&] {
        if (!ctx) return fail(SLW_EINVAL, "null context");
        if (!ctx->kv_ready) return fail(SLW_EINVAL, "KV pools not attached");
        return ctx->kv.release(id);
    });
}

extern "C" int slw_seq_reserve(slw_ctx* ctx, int64_t id, int32_t new_len) {
    return guarded([&] {
        if (!ctx) return fail(SLW_EINVAL, "null context");
        if (!ctx->kv_ready) return fail(SLW_EINVAL, "KV pools not attached");
        if (new_len > ctx->cfg.max_pos) return fail(SLW_ERANGE, "length %d above max_pos", new_len);
        return ctx->kv.reserve_all({{id, new_len}});
    });
}

extern "C" int slw_seq_block_table(slw_ctx* ctx, int64_t id, int32_t* out, int32_t cap, int32_t* n) {
    return guarded([&] {
        if (!ctx || !n) return fail(SLW_EINVAL, "null argument");
        if (!ctx->kv_ready || !ctx->kv.exists(id)) return fail(SLW_EINVAL, "sequence %lld unknown", (long long)id);
        const auto& t = ctx->kv.table(id);
        *n = static_cast<int32_t>(t.size());
        if (out) {
            if (cap < *n) return fail(SLW_ERANGE, "table has %d entries, cap %d", *n, cap);
            std::copy(t.begin(), t.end(), out);
        }
        return SLW_OK;
    });
}

extern "C" int slw_workspace_size(slw_ctx* ctx, int32_t max_C, int32_t max_B, size_t* bytes) {
    return guarded([&] {
        if (!ctx || !bytes) return fail(SLW_EINVAL, "null argument");
        if (max_C < 0 || max_B < 0) return fail(SLW_EINVAL, "negative size");
        size_t gp = 0;
        for (int m = 1; m <= max_C + max_B; ++m) gp = std::max(gp, gemm_partial_bytes(ctx->cfg, m));
        *bytes = layout(ctx->cfg, max_C, max_B).end_fixed + gp;
        return SLW_OK;
    });
}

extern "C" int slw_workspace_view(slw_ctx* ctx, int32_t which, int32_t C, int32_t B, size_t* offset,
                                  size_t* bytes) {
    if (!ctx || !offset || !bytes) return fail(SLW_EINVAL, "null argument");
    if (C < 0 || B < 0) return fail(SLW_EINVAL, "negative size");
    const slw_model_cfg& c = ctx->cfg;
    const Layout L = layout(c, C, B);
    const size_t M = static_cast<size_t>(C) + B;
    switch (which) {
        case SLW_VIEW_QKV: *offset = L.qkv; *bytes = M * qkv_width(c) * 2; break;
        case SLW_VIEW_ATTN: *offset = L.attn; *bytes = M * c.n_q_heads * c.head_dim * 2; break;
        case SLW_VIEW_H: *offset = L.h; *bytes = M * c.d_model * 4; break;
        case SLW_VIEW_ACT: *offset = L.act; *bytes = M * c.ffn_dim * 2; break;
        default: return fail(SLW_EINVAL, "unknown view %d", which);
    }
    return SLW_OK;
}

extern "C" int slw_mixed_iteration(slw_ctx* ctx, const slw_batch* batch, const void* x_in, void* x_out,
                                   void* ws, size_t ws_bytes, void* stream) {
    return guarded([&] {
        if (!ctx) return fail(SLW_EINVAL, "null context");
        return mixed_iteration_impl(ctx, batch, x_in, x_out, ws, ws_bytes, static_cast<hipStream_t>(stream));
    });
}

// ---------------------------------------------------------------------------
// The allocation-free variant: the workspace is a file-scope device array of
// SLW_STATIC_WS_BYTES, one copy per GPU, held until the process ends.  Its
// address on each device is taken once, with that device current, through
// hipGetSymbolAddress; host code uses only that address (the array's name
// is a host-side stand-in).  No value in it needs to start at zero: every
// word a kernel reads was written earlier in the same call.  Calls that
// overlap on one GPU share the array and race.
// ---------------------------------------------------------------------------

namespace {

constexpr size_t kStaticWsBytes = SLW_STATIC_WS_BYTES;
static __device__ __attribute__((aligned(256))) unsigned char scratch[kStaticWsBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int static_workspace(void** out) {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(SLW_ERANGE, "device %d above %d", dev, kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(SLW_EHIP, "hipGetSymbolAddress gave a null address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return SLW_OK;
}

}  // namespace

extern "C" int slw_mixed_iteration_static(slw_ctx* ctx, const slw_batch* batch, const void* x_in, void* x_out,
                                          void* stream) {
    return guarded([&] {
        if (!ctx) return fail(SLW_EINVAL, "null context");
        void* ws = nullptr;
        int rc = static_workspace(&ws);
        if (rc) return rc;
        return mixed_iteration_impl(ctx, batch, x_in, x_out, ws, kStaticWsBytes, static_cast<hipStream_t>(stream),
                                    true);
    });
}

extern "C" int slw_fill_normal(void* dst, size_t n, uint64_t seed, float mean, float std, void* stream) {
    return guarded([&] {
        if (!dst && n) return fail(SLW_EINVAL, "null buffer");
        if (reinterpret_cast<uintptr_t>(dst) % 2) return fail(SLW_EINVAL, "buffer must be 2-byte aligned");
        if (n / 4 >= (static_cast<size_t>(1) << 62)) return fail(SLW_ERANGE, "too many elements");
        launch_fill_normal(dst, n, seed, mean, std, static_cast<hipStream_t>(stream));
        HIP_TRY(hipGetLastError());
        return SLW_OK;
    });
}

extern "C" int slw_flush_cache(void* buf, size_t bytes, void* stream) {
    return guarded([&] {
        if (!buf && bytes) return fail(SLW_EINVAL, "null buffer");
        if (reinterpret_cast<uintptr_t>(buf) % 16) return fail(SLW_EINVAL, "buffer must be 16-byte aligned");
        launch_cache_sweep(buf, bytes, 0x9e3779b9u, static_cast<hipStream_t>(stream));
        HIP_TRY(hipGetLastError());
        return SLW_OK;
    });
}

extern "C" int slw_set_stage_timing(slw_ctx* ctx, int32_t depth) {
    return guarded([&] {
        if (!ctx) return fail(SLW_EINVAL, "null context");
        if (depth < 0 || depth > 4096) return fail(SLW_ERANGE, "depth must be in [0, 4096]");
        ctx->stage_depth = depth;
        ctx->stage_mask.assign(depth, 0u);
        ctx->stage_iter = 0;
        return SLW_OK;
    });
}

extern "C" int slw_stage_times(slw_ctx* ctx, int32_t ago, float* ms, int32_t cap, int32_t* n) {
    if (!ctx || !ms || !n) return fail(SLW_EINVAL, "null argument");
    if (ctx->stage_depth <= 0) return fail(SLW_EINVAL, "stage timing is off");
    if (ago < 0 || ago >= ctx->stage_depth || ago >= ctx->stage_iter)
        return fail(SLW_ERANGE, "iteration %d ago is not recorded", ago);
    if (cap < kStages) return fail(SLW_ERANGE, "need room for %d stages", kStages);
    const int set = static_cast<int>((ctx->stage_iter - 1 - ago) % ctx->stage_depth);
    const uint32_t mask = ctx->stage_mask[set];
    const size_t base0 = static_cast<size_t>(set) * ctx->cfg.n_layers * (kStages + 1);
    if (mask) HIP_TRY(hipEventSynchronize(ctx->stage_ev[base0 + static_cast<size_t>(ctx->cfg.n_layers) * (kStages + 1) - 1]));
    for (int s = 0; s < kStages; ++s) {
        float tot = 0.f;
        if (mask & (1u << s)) {
            for (int l = 0; l < ctx->cfg.n_layers; ++l) {
                float t = 0.f;
                const size_t base = base0 + static_cast<size_t>(l) * (kStages + 1);
                HIP_TRY(hipEventElapsedTime(&t, ctx->stage_ev[base + s], ctx->stage_ev[base + s + 1]));
                tot += t;
            }
        }
        ms[s] = tot;
    }
    *n = kStages;
    return SLW_OK;
}

extern "C" int slw_last_slots(slw_ctx* ctx, int32_t* out, int32_t cap, int32_t* n) {
    if (!ctx || !n) return fail(SLW_EINVAL, "null argument");
    *n = static_cast<int32_t>(ctx->last_slots.size());
    if (out) {
        if (cap < *n) return fail(SLW_ERANGE, "%d slots, cap %d", *n, cap);
        std::copy(ctx->last_slots.begin(), ctx->last_slots.end(), out);
    }
    return SLW_OK;
}

// ---------------------------------------------------------------------------
// Profiler (Sec. 5.1): time the mixed iteration over a (decode batch, chunk)
// grid, keep every sample, then P50/P99 and a running maximum along chunks.
// ---------------------------------------------------------------------------

namespace {

// Profile planes of the table: for each prefix in p_grid (or the single
// prefix opts->prefix_len when p_grid is null) time the iteration over every
// (b, c) of b_grid x c_grid.
int build_table_core(slw_ctx* ctx, const int32_t* c_grid, int32_t nc, const int32_t* b_grid, int32_t nb,
                     const int32_t* p_grid, int32_t np, const slw_profile_opts* o, slw_cost_table** out) {
    if (!ctx || !o || !out || !c_grid || !b_grid) return fail(SLW_EINVAL, "null argument");
    *out = nullptr;
    if (!ctx->kv_ready) return fail(SLW_EINVAL, "KV pools not attached");
    if (nc < 1 || nb < 1 || (p_grid && np < 1)) return fail(SLW_EINVAL, "empty grid");
    if (o->repeats < 1 || o->warmup < 0) return fail(SLW_EINVAL, "repeats must be >= 1, warmup >= 0");
    if (o->prefix_len < 0 || o->ctx_lo < 0 || o->ctx_hi < o->ctx_lo)
        return fail(SLW_EINVAL, "bad prefix or context range");
    auto t = std::make_unique<slw_cost_table>();
    t->c_grid.assign(c_grid, c_grid + nc);
    t->b_grid.assign(b_grid, b_grid + nb);
    if (p_grid) {
        t->p_grid.assign(p_grid, p_grid + np);
        t->has_ctx = true;
    } else {
        t->p_grid.assign(1, o->prefix_len);
    }
    t->repeats = o->repeats;
    // validate grids before reserving anything (finish_table repeats the check)
    t->samples.assign(static_cast<size_t>(t->np()) * nb * nc * o->repeats, 0);
    int rc = finish_table(t.get());
    if (rc) return rc;
    const int c_last = c_grid[nc - 1], b_last = b_grid[nb - 1];
    const int p_last = t->p_grid.back();

    const int64_t base = INT64_MIN + 1;  // profiler-reserved ids
    const int64_t pre_id = base;
    std::vector<int64_t> dec(b_last);
    std::vector<int32_t> ctxl(b_last);
    std::mt19937_64 rng(o->seed);
    std::uniform_int_distribution<int32_t> dist(o->ctx_lo, o->ctx_hi);
    for (int i = 0; i < b_last; ++i) {
        dec[i] = base + 1 + i;
        ctxl[i] = dist(rng);
    }
    std::vector<int64_t> made;
    auto cleanup = [&] {
        for (int64_t id : made) (void)ctx->kv.release(id);
    };
    rc = ctx->kv.create(pre_id);
    if (rc) return rc;
    made.push_back(pre_id);
    for (int i = 0; i < b_last; ++i) {
        rc = ctx->kv.create(dec[i]);
        if (rc) { cleanup(); return rc; }
        made.push_back(dec[i]);
    }
    std::vector<std::pair<int64_t, int32_t>> req;
    req.emplace_back(pre_id, p_last + c_last);
    for (int i = 0; i < b_last; ++i) req.emplace_back(dec[i], ctxl[i] + 1);
    rc = ctx->kv.reserve_all(req);
    if (rc) { cleanup(); return rc; }

    hipStream_t s = static_cast<hipStream_t>(o->stream);
    auto run = [&](int prefix, int b, int cc) {
        slw_batch batch{cc, pre_id, prefix, b, dec.data(), ctxl.data()};
        return mixed_iteration_impl(ctx, &batch, o->x_in, o->x_out, o->ws, o->ws_bytes, s);
    };
    auto sync = [&]() -> int {
        hipError_t e = hipStreamSynchronize(s);
        if (e != hipSuccess) return fail(SLW_EHIP, "hipStreamSynchronize: %s", hipGetErrorString(e));
        return SLW_OK;
    };
    for (int k = 0; k < t->np() && !rc; ++k)
        for (int i = 0; i < nb && !rc; ++i)
            for (int j = 0; j < nc && !rc; ++j) {
                const int prefix = t->p_grid[k];
                for (int r = 0; r < o->warmup && !rc; ++r) rc = run(prefix, b_grid[i], c_grid[j]);
                if (!rc) rc = sync();
                for (int r = 0; r < o->repeats && !rc; ++r) {
                    if (o->flush_buf && o->flush_bytes) {
                        launch_cache_sweep(o->flush_buf, o->flush_bytes, 0x9e3779b9u + static_cast<uint32_t>(r), s);
                        rc = sync();
                        if (rc) break;
                    }
                    auto t0 = std::chrono::steady_clock::now();
                    rc = run(prefix, b_grid[i], c_grid[j]);
                    if (!rc) rc = sync();
                    auto t1 = std::chrono::steady_clock::now();
                    t->samples[((static_cast<size_t>(k) * nb + i) * nc + j) * o->repeats + r] =
                        std::chrono::duration_cast<std::chrono::nanoseconds>(t1 - t0).count();
                }
            }
    cleanup();
    if (rc) return rc;
    if (!p_grid) t->p_grid.assign(1, 0);  // one plane serves every prefix
    rc = finish_table(t.get());
    if (rc) return rc;
    *out = t.release();
    return SLW_OK;
}

}  // namespace

extern "C" int slw_build_cost_table(slw_ctx* ctx, const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                                    int32_t nb, const slw_profile_opts* o, slw_cost_table** out) {
    return guarded([&]() -> int { return build_table_core(ctx, c_grid, nc, b_grid, nb, nullptr, 0, o, out); });
}

extern "C" int slw_build_cost_table_ctx(slw_ctx* ctx, const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                                        int32_t nb, const int32_t* p_grid, int32_t np, const slw_profile_opts* o,
                                        slw_cost_table** out) {
    return guarded([&]() -> int {
        if (!p_grid) return fail(SLW_EINVAL, "null context grid");
        return build_table_core(ctx, c_grid, nc, b_grid, nb, p_grid, np, o, out);
    });
}

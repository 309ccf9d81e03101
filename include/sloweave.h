/*
 * sloweave.h -- C ABI of libsloweave.so, an MI355X (gfx950) implementation of
 * the mixed prefill+decode iteration that SLOWeave schedules (arXiv
 * 2609.07883), the profiler that prices it, and the controller that sizes
 * each iteration's prefill chunk.
 *
 * Conventions
 *   - Every call returns SLW_OK (0) or a negative SLW_E* code; the message of
 *     the last failure on the calling thread is returned by slw_last_error().
 *     No C++ exception crosses this boundary.
 *   - "device" pointers are HIP device memory on the current device; "host"
 *     pointers are ordinary CPU memory.  The library never allocates device
 *     memory: weights, KV pools, activations and the workspace all belong to
 *     the caller.  It owns only host state (sequence tables, cost tables) plus
 *     a small pinned host staging ring, HIP events and one non-blocking
 *     stream (decode attention beside a long chunk's), created on first use,
 *     and the static workspace array of slw_mixed_iteration_static, which is
 *     part of its device code (loaded with it, never allocated by a call).
 *   - Streams are passed as void* holding a hipStream_t (NULL = the null
 *     stream).  Device work is enqueued asynchronously; kernel faults surface
 *     at the caller's next synchronisation.
 *   - bf16 is the 16-bit brain-float format stored as uint16 bit patterns.
 *   - A context is not thread-safe; slw_select_chunk and the cost-table
 *     queries are pure and may be called from any thread.
 */
#ifndef SLOWEAVE_H
#define SLOWEAVE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SLW_OK 0
#define SLW_EINVAL (-1)       /* bad argument or inconsistent state            */
#define SLW_ERANGE (-2)       /* argument outside a grid or a capacity          */
#define SLW_ENOMEM (-3)       /* KV block pool or workspace too small           */
#define SLW_EHIP (-4)         /* a HIP runtime call failed                      */
#define SLW_EUNSUPPORTED (-5) /* shape outside what the kernels implement      */

/* flags reported by slw_select_chunk */
#define SLW_FLAG_NO_PENDING 1u         /* no pending prefill: chunk 0          */
#define SLW_FLAG_NO_ACTIVE 2u          /* empty active set: chunk = cap        */
#define SLW_FLAG_DECODE_INFEASIBLE 4u  /* even a decode-only iteration misses  */
#define SLW_FLAG_CAPPED_BY_GRID 8u     /* cap lowered to the last profiled C   */

typedef struct slw_ctx slw_ctx;
typedef struct slw_cost_table slw_cost_table;

/* Thread-local message describing the last failure ("" if none). */
const char* slw_last_error(void);

/* ------------------------------------------------------------------------ */
/* Model                                                                     */
/* ------------------------------------------------------------------------ */

/*
 * Shape of the decoder stack the iteration runs.  The paper schedules an
 * unmodified dense decoder (Sec. 5.1, Sec. 5.2); the block is the standard
 * pre-norm one: RMSNorm, QKV projection, rotate-half RoPE, grouped-query
 * causal attention over the paged cache, output projection + residual,
 * RMSNorm, SwiGLU MLP + residual.
 * Supported: head_dim in {64, 128}; n_q_heads % n_kv_heads == 0 with group
 * n_q_heads / n_kv_heads in {1, 2, 4, 8, 16}; d_model a multiple of 128 in
 * [128, 8192]; ffn_dim a multiple of 64; (n_q_heads + 2 n_kv_heads) *
 * head_dim a multiple of 128; block_size == 16; 1 <= max_pos <= 1048576.
 */
typedef struct slw_model_cfg {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t ffn_dim;
    float rms_eps;      /* RMSNorm epsilon                                      */
    float rope_theta;   /* RoPE base: angle(p, i) = p * theta^(-2i/head_dim)    */
    int32_t block_size; /* KV positions per block; must be 16                  */
    int32_t max_pos;    /* largest sequence length any call may reach          */
} slw_model_cfg;

/*
 * Device pointers to one layer's bf16 weights, row-major [out][in]:
 *   wqkv [(Hq + 2 Hkv) * hd][d]   q rows, then k rows, then v rows
 *   wo   [d][Hq * hd]
 *   wgu  [2 F][d]                 gate rows, then up rows
 *   wd   [d][F]
 *   g1, g2 [d]                    RMSNorm gains (before attention / MLP)
 * The caller keeps the memory alive while the context uses it.
 */
typedef struct slw_layer_weights {
    const void* wqkv;
    const void* wo;
    const void* wgu;
    const void* wd;
    const void* g1;
    const void* g2;
} slw_layer_weights;

/* Create a context for cfg (host state only; touches no GPU).  *out owns it. */
int slw_create(const slw_model_cfg* cfg, slw_ctx** out);
/* Destroy a context (waits for nothing: synchronise your streams first). */
int slw_destroy(slw_ctx* ctx);
/* Register layer `layer`'s weights (0 <= layer < n_layers). */
int slw_set_layer_weights(slw_ctx* ctx, int32_t layer, const slw_layer_weights* w);

/* ------------------------------------------------------------------------ */
/* Paged KV cache (Table 1, "KV manager": layout unchanged, blocks allocated */
/* as chunks are processed)                                                  */
/* ------------------------------------------------------------------------ */

/*
 * Attach caller-owned KV pools of num_blocks blocks each (device, bf16):
 *   k_pool  [n_layers][num_blocks][Hkv][hd/32][16][32]
 *           element (token t of the block, dim d) at (d/32)*512 + t*32 + d%32
 *           within the (layer, block, head) page of 16*hd values;
 *   v_pool  [n_layers][num_blocks][Hkv][hd][16]
 *           element (t, d) at d*16 + t within the page.
 * Resets the block manager (all sequences are forgotten).
 */
int slw_kv_init(slw_ctx* ctx, void* k_pool, void* v_pool, int32_t num_blocks);
/* Number of free blocks. */
int slw_kv_free_blocks(slw_ctx* ctx, int32_t* n_free);

/*
 * Sequences.  A sequence grows by whole blocks, always taking the
 * lowest-numbered free block first; slw_seq_reserve(id, n) makes room for
 * positions 0..n-1 (a no-op if already there).  A reservation the pool cannot
 * cover returns SLW_ENOMEM and changes nothing.  slw_seq_free returns all the
 * sequence's blocks.  Ids below -2^62 are reserved for the profiler.
 */
int slw_seq_create(slw_ctx* ctx, int64_t id);
int slw_seq_free(slw_ctx* ctx, int64_t id);
int slw_seq_reserve(slw_ctx* ctx, int64_t id, int32_t new_len);
/* Copy the sequence's block table (host int32, at most cap entries) and its length to *n. */
int slw_seq_block_table(slw_ctx* ctx, int64_t id, int32_t* out, int32_t cap, int32_t* n);

/* ------------------------------------------------------------------------ */
/* The mixed iteration (Sec. 3: one prefill chunk plus one decode token per */
/* active request; Sec. 5.1: the chunk rides in ordinary sequence metadata)  */
/* ------------------------------------------------------------------------ */

/*
 * One iteration's batch (host memory):
 *   C             prefill-chunk tokens (0: decode-only iteration)
 *   prefill_seq   sequence the chunk belongs to (ignored when C == 0)
 *   prefix_len    tokens of prefill_seq already cached; the chunk occupies
 *                 positions prefix_len .. prefix_len + C - 1
 *   B             decode requests (0: prefill-only iteration)
 *   decode_seqs   [B] sequence ids, distinct and different from prefill_seq
 *   context_lens  [B] tokens cached for each decode BEFORE this iteration; the
 *                 decode token sits at position context_lens[b] and attends to
 *                 context_lens[b] + 1 keys
 * Prefill batching (Sec. 3.3: several pending prompts in one iteration):
 *   n_prefill     > 1: the C chunk rows come from n_prefill prompts (at most
 *                 SLW_MAX_PREFILLS), prompt i's chunk_lens[i] >= 1 rows after
 *                 those of prompts 0 .. i-1, at positions prefix_lens[i] ..
 *                 prefix_lens[i] + chunk_lens[i] - 1 of prefill_seqs[i]; the
 *                 chunk_lens add up to C and prefill_seq / prefix_len are
 *                 ignored.  0 or 1: one prefill as above (the arrays are ignored).
 */
#define SLW_MAX_PREFILLS 16
typedef struct slw_batch {
    int32_t C;
    int64_t prefill_seq;
    int32_t prefix_len;
    int32_t B;
    const int64_t* decode_seqs;
    const int32_t* context_lens;
    int32_t n_prefill;
    const int64_t* prefill_seqs;
    const int32_t* prefix_lens;
    const int32_t* chunk_lens;
} slw_batch;

/*
 * Device workspace bytes needed by any iteration with C <= max_C and
 * B <= max_B (activations, split partials, per-iteration metadata).
 */
int slw_workspace_size(slw_ctx* ctx, int32_t max_C, int32_t max_B, size_t* bytes);

/*
 * Run all n_layers layers over the batch (asynchronous on `stream`).
 *   x_in   device bf16 [C + B][d]: chunk rows first, then decode rows
 *   x_out  device bf16 [C + B][d]; may equal x_in
 *   ws     device workspace of ws_bytes >= slw_workspace_size(ctx, C, B)
 * Reserves KV room (each prefill sequence up to its prefix + chunk, in row
 * order, then each decode up to context_lens[b] + 1; all or nothing, SLW_ENOMEM if the pool cannot cover
 * it; a call that fails after reserving returns the blocks), builds the slot mapping and block tables on the host, writes them to
 * a coherent pinned staging ring that a first kernel copies into the
 * workspace, then enqueues per layer: RMSNorm, QKV GEMM
 * whose epilogue applies RoPE and appends K/V to the pages, chunk attention
 * and split decode attention (one launch; for a chunk of at least 8 M
 * query-key pairs, decode attention on the context's own stream beside it,
 * joined back to `stream` by an event before the merge), output GEMM +
 * residual (kept in fp32 within the layer), RMSNorm, gate/up GEMM with
 * SiLU*mul, down GEMM + residual.
 * Each row's K/V is written at slot(seq, pos) = bt[pos/16]*16 + pos%16 of its
 * sequence in every layer.  C == 0 and B == 0 together is a no-op.
 */
int slw_mixed_iteration(slw_ctx* ctx, const slw_batch* batch, const void* x_in, void* x_out,
                        void* ws, size_t ws_bytes, void* stream);

/*
 * The mixed iteration for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Same batch, inputs, outputs and results as
 * slw_mixed_iteration, but it takes no workspace: it uses a device array of
 * SLW_STATIC_WS_BYTES inside the library, one per GPU, which each GPU the
 * library runs on holds until the process ends.  The call allocates nothing
 * (no hipMalloc, no pinned host memory, no stream or event): the metadata is
 * copied from host memory the context already holds, `stream` is
 * synchronised once after that copy (the iteration's kernels then run
 * asynchronously), both attentions run on `stream`, and no stage timing is
 * recorded.  An iteration whose workspace would exceed the array
 * (slw_workspace_size(ctx, C, B) gives an upper bound) is refused with
 * SLW_ENOMEM before anything is reserved or enqueued.  Every call on a GPU
 * shares that GPU's array, which keeps the last call's contents: calls that
 * overlap on one GPU (several streams or threads) race.
 */
#define SLW_STATIC_WS_BYTES ((size_t)128 << 20)
int slw_mixed_iteration_static(slw_ctx* ctx, const slw_batch* batch, const void* x_in, void* x_out, void* stream);

/* Slot of every row of the last slw_mixed_iteration (host int32, chunk rows first). */
int slw_last_slots(slw_ctx* ctx, int32_t* out, int32_t cap, int32_t* n);

/*
 * Where an intermediate of the LAST layer of an iteration with (C, B) lives
 * in the workspace, for inspection after the stream is synchronised:
 *   SLW_VIEW_QKV   bf16 [C+B][(Hq+2Hkv)*hd] (q and k after RoPE)
 *   SLW_VIEW_ATTN  bf16 [C+B][Hq*hd] attention output
 *   SLW_VIEW_H     fp32 [C+B][d] residual stream after attention
 *   SLW_VIEW_ACT   bf16 [C+B][F] silu(gate) * up
 */
#define SLW_VIEW_QKV 0
#define SLW_VIEW_ATTN 1
#define SLW_VIEW_H 2
#define SLW_VIEW_ACT 3
int slw_workspace_view(slw_ctx* ctx, int32_t which, int32_t C, int32_t B, size_t* offset,
                       size_t* bytes);

/*
 * Stage telemetry (Fig. 1 and Table 1 record observed iteration durations).
 * slw_set_stage_timing(ctx, depth) with depth > 0 makes every following
 * slw_mixed_iteration record HIP events on its stream before each stage of
 * each layer and after the last one, keeping the events of the last `depth`
 * iterations (depth 0 turns recording off; at most 4096).
 * slw_stage_times(ctx, ago, ms, cap, n) waits for the iteration `ago` steps
 * before the most recent one (0 = most recent) and writes, per stage, its
 * elapsed milliseconds summed over layers:
 *   0 RMSNorm (attention)  1 RoPE table    2 QKV GEMM with RoPE and KV append
 *   3 chunk attention      4 decode attention  5 attention merges (split
 *   chunk query tiles and decode key splits, one launch)  6 output GEMM
 *   7 RMSNorm (MLP)        8 gate/up GEMM  9 down GEMM
 * Stages absent from that iteration (C == 0 or B == 0) read 0.  Stage 1 is
 * kept for the layout of the array and reads (close to) 0: the RoPE table is
 * filled by the iteration's first kernel, together with the metadata copy,
 * before stage 0 of layer 0.
 */
#define SLW_N_STAGES 10
int slw_set_stage_timing(slw_ctx* ctx, int32_t depth);
int slw_stage_times(slw_ctx* ctx, int32_t ago, float* ms, int32_t cap, int32_t* n);

/* ------------------------------------------------------------------------ */
/* Cost table (Sec. 5.1 profiler: P50/P99 per grid point, cumulative max    */
/* along the chunk axis; Sec. 6.4: profile at start-up, interpolate)         */
/* ------------------------------------------------------------------------ */

typedef struct slw_profile_opts {
    int32_t prefix_len;   /* cached tokens of the profiled prefill sequence           */
    int32_t ctx_lo;       /* decode contexts uniform in [ctx_lo, ctx_hi]               */
    int32_t ctx_hi;
    uint64_t seed;        /* seed of the context draw                                 */
    int32_t warmup;       /* untimed iterations per grid point (>= 0)                 */
    int32_t repeats;      /* timed iterations per grid point (>= 1)                   */
    void* flush_buf;      /* device buffer read in full before every timed iteration  */
    size_t flush_bytes;   /* (evicts the last-level cache without dirtying it; its    */
                          /* contents are left as they are); 0 = no flush            */
    const void* x_in;     /* device bf16 [max C + max B][d] input rows                */
    void* x_out;          /* device bf16 [max C + max B][d]                           */
    void* ws;             /* device workspace for (max C, max B)                      */
    size_t ws_bytes;
    void* stream;
} slw_profile_opts;

/*
 * Time slw_mixed_iteration over every (b, c) of b_grid x c_grid and build the
 * table (synchronous).  Grids strictly increase; c_grid[0] must be 0 (the
 * decode-only column); b_grid values are >= 0.  Each repeat is timed on the
 * host clock from the call to the end of a stream synchronisation, so launch
 * overhead is part of T.  Temporary sequences (one prefill sequence, max(b)
 * decodes) are reserved from the pool and freed before returning; KV contents
 * are whatever the pool holds.  *out receives a new table (slw_cost_table_free).
 */
int slw_build_cost_table(slw_ctx* ctx, const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                         int32_t nb, const slw_profile_opts* opts, slw_cost_table** out);
/*
 * The same with a cached-context axis (Sec. 5.1 indexes the runtime's table
 * by decode batch, cached context and chunk): one (b, c) plane per entry of
 * p_grid (strictly increasing, >= 0), each profiled with the chunk's sequence
 * holding that many cached tokens (opts->prefix_len is ignored; the decode
 * contexts are drawn as above).  Lookups take the prefix of the chunk's
 * sequence and use the plane of the first p_grid point >= it.
 */
int slw_build_cost_table_ctx(slw_ctx* ctx, const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                             int32_t nb, const int32_t* p_grid, int32_t np, const slw_profile_opts* opts,
                             slw_cost_table** out);

/* Build a table from raw samples, host int64 ns [nb][nc][repeats] (e.g. an analytic model). */
int slw_cost_table_from_samples(const int32_t* c_grid, int32_t nc, const int32_t* b_grid,
                                int32_t nb, const int64_t* samples, int32_t repeats,
                                slw_cost_table** out);
/* The same with a context axis: samples [np][nb][nc][repeats], p_grid as for the _ctx profiler. */
int slw_cost_table_from_samples_ctx(const int32_t* c_grid, int32_t nc, const int32_t* b_grid, int32_t nb,
                                    const int32_t* p_grid, int32_t np, const int64_t* samples, int32_t repeats,
                                    slw_cost_table** out);
/*
 * A table holding the simulator's analytic cost model (Sec. 4.1) at every
 * grid point, one sample each:
 *   T(n, c) = 0.35 + 1[n>0](0.90 + 0.055 n) + 1[c>0](0.40 + 0.006 c) ms.
 * Grids as for slw_cost_table_from_samples.
 */
int slw_cost_table_analytic(const int32_t* c_grid, int32_t nc, const int32_t* b_grid, int32_t nb,
                            slw_cost_table** out);
void slw_cost_table_free(slw_cost_table* t);
int slw_cost_table_dims(const slw_cost_table* t, int32_t* nc, int32_t* nb, int32_t* repeats);
int slw_cost_table_grids(const slw_cost_table* t, int32_t* c_grid, int32_t* b_grid);
/* Context points of the table into p_grid (cap entries; may be NULL); *np = 0 without a context axis. */
int slw_cost_table_prefixes(const slw_cost_table* t, int32_t* p_grid, int32_t cap, int32_t* np);

/*
 * Copy a table view to host int64:
 *   SLW_TABLE_SAMPLES [nb][nc][repeats] raw ns; SLW_TABLE_P50 / SLW_TABLE_P99 [nb][nc]
 *   nearest-rank percentiles sorted[ceil(k*q)-1]; SLW_TABLE_THAT [nb][nc] the P99 with
 *   a running maximum along c (the table the controller reads).  Tables with a
 *   context axis have a leading [np] dimension.
 */
#define SLW_TABLE_SAMPLES 0
#define SLW_TABLE_P50 1
#define SLW_TABLE_P99 2
#define SLW_TABLE_THAT 3
int slw_cost_table_values(const slw_cost_table* t, int32_t which, int64_t* out, size_t cap);

/*
 * Predicted time T_hat(n, c) in ns.  n rounds up to the next b_grid point
 * (SLW_ERANGE above the last); c = 0 reads column 0; 0 < c <= c_1 reads c_1;
 * c_j < c <= c_{j+1} interpolates T_hat_j + ceil((T_hat_{j+1}-T_hat_j)(c-c_j)/(c_{j+1}-c_j));
 * c above the last grid point is SLW_ERANGE.
 */
int slw_cost_table_lookup(const slw_cost_table* t, int32_t n, int32_t c, int64_t* t_ns);
/*
 * The same at the cached context `prefix` (tokens of the chunk's sequence
 * cached before the chunk): the plane of the first context point >= prefix
 * (SLW_ERANGE above the last).  Tables without a context axis ignore prefix;
 * slw_cost_table_lookup is this with prefix 0.
 */
int slw_cost_table_lookup_ctx(const slw_cost_table* t, int32_t prefix, int32_t n, int32_t c, int64_t* t_ns);
/* Raw P99 decreases along c before the running maximum: count and largest drop (ns). */
int slw_cost_table_monotone(const slw_cost_table* t, int32_t* violations, int64_t* worst_ns);
/* Text save / load of grids and raw samples (percentiles are recomputed on load). */
int slw_cost_table_save(const slw_cost_table* t, const char* path);
int slw_cost_table_load(const char* path, slw_cost_table** out);

/*
 * Read `bytes` of the device buffer `buf` on `stream` (asynchronous): the
 * last-level cache sweep the profiler runs before every timed repeat (it
 * evicts cached weights and K/V without leaving dirty lines behind; only
 * the buffer's first word may be overwritten), for callers that time
 * iterations from a cold cache themselves.  buf is 16-byte aligned.
 */
int slw_flush_cache(void* buf, size_t bytes, void* stream);

/*
 * Fill device bf16 dst[0 .. n-1] with mean + std * z_i (asynchronous on
 * `stream`): seeded synthetic weights for stacks too large to draw on the
 * host, not a step of the iteration.  z is the standard-normal stream of
 * the counter-based Philox4x32-10 generator (Salmon et al., SC 2011) keyed
 * by `seed`: draw t (counter (t mod 2^32, t div 2^32, 0, 0)) gives words
 * w0..w3, and elements 4t .. 4t+3 are Box-Muller pairs of the 24-bit
 * uniforms u = ((w0 >> 8) + 1/2) 2^-24, v = (w1 >> 8) 2^-24 (then w2, w3):
 * sqrt(-2 ln u) cos(2 pi v), sqrt(-2 ln u) sin(2 pi v), rounded to bf16.
 */
int slw_fill_normal(void* dst, size_t n, uint64_t seed, float mean, float std, void* stream);

/*
 * The GEMM plan an iteration uses for a projection out[m][n] = A[m][k] W^T
 * (host only, touches no GPU), for callers and tests that need to know which
 * kernel variant a row count reaches.  out[0..5]: tile configuration (99:
 * the weight-streaming kernel for m <= 32; 98: the narrow kernel for
 * m <= 24, k split over the waves of a work-group), tile rows BM, tile columns BN,
 * k split factor (1: none), stream-K work-groups (0: not used), whole tiles
 * run before them.  m >= 1; n a multiple of 128 and k of 64, else SLW_EINVAL.
 */
int slw_gemm_plan(int32_t m, int32_t n, int32_t k, int32_t out[6]);

/*
 * The attention work lists an iteration would build (host only, touches no
 * GPU), for B decodes with context_lens[b] cached tokens each and n_prefill
 * prompts, prompt i running chunk_lens[i] rows after prefix_lens[i] cached
 * tokens, under cfg.  out[0..11]:
 *   decode attention: work items, wave slots per kv head, largest and
 *     smallest number of keys a slot takes;
 *   chunk attention: query tiles, work items, work-groups per kv head,
 *     1 when every work-group takes whole query tiles (nothing to merge),
 *     largest and smallest number of 64-key tiles a work-group takes, 64-key
 *     tiles in all;
 *   out[11] = 0.
 * The same invariants the executor checks on every iteration are checked
 * here (every item list tiles its keys exactly, caps respected).
 * SLW_EINVAL for a bad cfg, negative sizes, prompts beyond max_pos or more
 * than SLW_MAX_PREFILLS prompts.
 */
int slw_attention_plan(const slw_model_cfg* cfg, int32_t B, const int32_t* context_lens, int32_t n_prefill,
                       const int32_t* prefix_lens, const int32_t* chunk_lens, int64_t out[12]);

/* ------------------------------------------------------------------------ */
/* Controller (Eq. 1 solved by bisection as Alg. 1 does; margin of Sec. 3.3) */
/* ------------------------------------------------------------------------ */

/*
 * Largest chunk c <= min(c_max, remaining, last grid C) with
 * T_hat(n_active, c) + margin_ns <= min_i deadlines_ns[i] - now_ns.
 *   deadlines_ns  host [n_active] absolute next-token deadlines d_i = l_i + D_i
 *   remaining     remaining prompt tokens of the oldest pending prefill (<= 0: none)
 * remaining <= 0 gives 0 (NO_PENDING); n_active == 0 gives the cap (NO_ACTIVE);
 * when no chunk fits the result is 0 (a decode-only iteration) and
 * DECODE_INFEASIBLE tells whether decode-only itself misses the budget.
 * n_active above the last b_grid point is SLW_ERANGE with *chunk = 0.
 * n_lookups (may be NULL) receives the number of table lookups made.
 * Pure, no allocation, thread-safe.
 */
int slw_select_chunk(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active,
                     int64_t now_ns, int32_t remaining, int32_t c_max, int64_t margin_ns,
                     int32_t* chunk, uint32_t* flags, int32_t* n_lookups);
/*
 * Alg. 1 priced at the cached context of the chunk's sequence: as
 * slw_select_chunk with every lookup made by slw_cost_table_lookup_ctx at
 * `prefix` (a prefix above the context grid is SLW_ERANGE once a lookup is
 * needed).  slw_select_chunk is this with prefix 0.
 */
int slw_select_chunk_ctx(const slw_cost_table* t, const int64_t* deadlines_ns, int32_t n_active,
                         int64_t now_ns, int32_t prefix, int32_t remaining, int32_t c_max, int64_t margin_ns,
                         int32_t* chunk, uint32_t* flags, int32_t* n_lookups);

/* ------------------------------------------------------------------------ */
/* Serving loop (Sec. 3.1 deadline model; Sec. 4.1 iteration semantics;     */
/* Sec. 4.3 oldest-first queueing shared by every policy)                    */
/* ------------------------------------------------------------------------ */

/* One request of a trace (host memory). */
typedef struct slw_request {
    int64_t id;          /* distinct; the request's KV sequence id while it lives     */
    int64_t arrival_ns;  /* arrival time on the trace clock (>= 0)                    */
    int32_t prompt_len;  /* prompt tokens, >= 1                                       */
    int32_t output_len;  /* output tokens, >= 1; the first one comes from the prefill */
} slw_request;

/*
 * Optional per-request objectives (Sec. 3.5), parallel to the request array.
 * A chunk is admissible when T_hat + delta_i <= d_i - s_t for every active
 * request i, with d_i = l_i + D_i: the loop runs Alg. 1 on the deadlines
 * d_i - (delta_i - opts->margin_ns) with margin opts->margin_ns.
 */
typedef struct slw_request_slo {
    int64_t tpot_ns;     /* D_i (> 0), or 0 for opts->tpot_ns                       */
    int64_t margin_ns;   /* delta_i of the request's class (>= 0), or < 0 for opts  */
    int64_t ttft_ns;     /* TTFT objective for SLW_QUEUE_EDF (> 0), or 0 for none   */
} slw_request_slo;

#define SLW_POLICY_SLOWEAVE 0 /* Alg. 1 over opts->table with margin and cap       */
#define SLW_POLICY_FIXED 1    /* chunks of opts->fixed_chunk tokens                */

#define SLW_EXEC_GPU 0        /* run each iteration with slw_mixed_iteration        */
#define SLW_EXEC_ANALYTIC 1   /* advance a virtual clock by the Sec. 4.1 cost model */
#define SLW_EXEC_TABLE 2      /* advance a virtual clock by opts->exec_table         */

/* flags of an iteration record besides those of slw_select_chunk */
#define SLW_SERVE_KV_WAIT 0x100u      /* the oldest prompt waits for KV blocks      */
#define SLW_SERVE_DECODE_CAP 0x200u   /* the oldest prompt waits: decode batch full */
#define SLW_SERVE_UNPRICED 0x400u     /* decode batch above the table: decode-only  */
#define SLW_SERVE_AGED 0x800u         /* chunk forced by the aging threshold         */
#define SLW_SERVE_FALLBACK 0x1000u    /* decode-only: residual P99 above the margin  */

/* Queue disciplines (Sec. 3.4): which pending prompt is served first.  Ties
 * go to the older request (arrival, then id). */
#define SLW_QUEUE_OLDEST 0   /* earliest arrival                                    */
#define SLW_QUEUE_SRPT 1     /* fewest remaining prompt tokens                      */
#define SLW_QUEUE_EDF 2      /* earliest arrival + TTFT objective (none: last)      */

typedef struct slw_serve_opts {
    int32_t policy;          /* SLW_POLICY_*                                            */
    int32_t fixed_chunk;     /* SLW_POLICY_FIXED: tokens per chunk (>= 1)               */
    int32_t c_max;           /* SLW_POLICY_SLOWEAVE: chunk cap (>= 1)                   */
    int32_t max_decode;      /* decode-batch cap (>= 1)                                 */
    int64_t tpot_ns;         /* D: next-token deadline d_i = l_i + D                    */
    int64_t margin_ns;       /* delta of Sec. 3.3 (>= 0)                                */
    const slw_cost_table* table; /* SLOWeave's predictor T_hat (required for it)        */
    int32_t executor;        /* SLW_EXEC_*                                              */
    int32_t skip_idle;       /* GPU: 1 = jump the clock over idle gaps, 0 = wait        */
    /* SLW_EXEC_GPU only (device memory, as for slw_mixed_iteration): */
    const void* x_in;        /* bf16 [max_rows][d] input rows                           */
    void* x_out;             /* bf16 [max_rows][d]                                      */
    int32_t max_rows;        /* rows x_in/x_out hold: >= chunk cap + max_decode         */
    void* ws;                /* workspace for (chunk cap, max_decode)                   */
    size_t ws_bytes;
    void* stream;
    /* Telemetry margin (Sec. 3.3 proposes a margin taken from a high
     * percentile of observed prediction errors; Sec. 5.1 feeds observed
     * durations back to the controller).  After every
     * iteration that ran a chunk priced by `table`, the relative residual
     * floor((observed - predicted) * 1e6 / predicted) ppm enters a window of
     * the last residual_window such values; each SLOWeave decision then adds
     * ceil(q * T_hat(n, c) / 1e6) to the prediction, q = max(0, nearest-rank
     * P99 of the window).  0 = off. */
    int32_t residual_window;
    const slw_cost_table* exec_table;  /* SLW_EXEC_TABLE: the iteration times */
    /* Policy variants (Sec. 3.3-3.5).  Zero-initialised fields leave the
     * loop as described above. */
    const slw_request_slo* slo; /* host [n] per-request objectives, or NULL            */
    int32_t queue;           /* SLW_QUEUE_*                                             */
    /* Admission control: a request that becomes eligible is refused when
     * T_hat(n, 0) + delta_i > D_i * admit_ppm / 1e6 (table lookup at prefix 0),
     * n counting the active decodes, the admitted pending prompts and the
     * request; also refused when n is beyond the table.  A refused request
     * emits no token: its token_ns entries are -1.  0 = off; needs table. */
    int32_t admit_ppm;
    /* Aging (SLOWeave): when Alg. 1 gives no chunk to a head that may run and
     * that has waited aging_ns since it became eligible or last ran a chunk,
     * min(aging_chunk, remaining, c_max) tokens run anyway (SLW_SERVE_AGED): a
     * bounded deadline violation recorded as such.  0 = off. */
    int64_t aging_ns;
    int32_t aging_chunk;
    /* Prefill batching by first fit (SLOWeave; at most SLW_MAX_PREFILLS
     * prompts on the GPU executor): when the head's chunk finishes
     * its prompt, the next pending prompts in queue order join while the
     * decode cap allows (counting prompts that finish earlier in the
     * iteration) and, on the GPU, while the KV pool can hold each prompt
     * that starts to its last token, up to max_prefills prompts, each with the largest chunk c
     * for which T_hat(n, S + c) still meets the budget, S being the tokens
     * already placed; a prompt that does not finish ends the list.  The
     * iteration is priced at the total.  0 or 1 = one prompt. */
    int32_t max_prefills;
    /* Telemetry fallback (Sec. 5.1: the scheduler falls back to decode-only
     * execution when telemetry residuals exceed the configured margin;
     * Table 1: telemetry records fallback events).  Every iteration whose
     * time `table` predicts leaves observed - predicted (ns) in a window of
     * the last fallback_window such values; while the window's nearest-rank
     * P99 exceeds margin_ns, a SLOWeave decision with a prompt to serve and
     * active decodes runs no chunk and its record carries SLW_SERVE_FALLBACK
     * (with no active decode there is no deadline to protect).  Decode-only
     * iterations keep filling the window, so chunks return once the observed
     * residuals are back within the margin.  0 = off. */
    int32_t fallback_window;
    /* Progress: after every log_every-th iteration the loop writes one line
     * to stderr (iterations so far, trace clock, requests done), so that a
     * long run shows where it is.  0 = silent. */
    int32_t log_every;
} slw_serve_opts;

/* One iteration of a serving run (host memory). */
typedef struct slw_iteration_record {
    int64_t start_ns;     /* trace clock before the chunk decision                      */
    int64_t end_ns;       /* trace clock once the iteration's work has completed        */
    int64_t budget_ns;    /* earliest next-token deadline minus start_ns (0: no decode) */
    int64_t decide_ns;    /* host nanoseconds spent choosing the chunk                  */
    int64_t predicted_ns; /* T_hat(n_decode, chunk) from opts->table, -1 without one    */
    int64_t prefill_id;   /* request the chunk belongs to, -1 when chunk == 0           */
    int32_t chunk;        /* prefill tokens run                                          */
    int32_t n_decode;     /* decode tokens run                                           */
    int32_t remaining;    /* prompt tokens of the oldest eligible prompt before the chunk
                             (0 when none may run)                                       */
    uint32_t flags;       /* SLW_FLAG_* of the decision | SLW_SERVE_*                    */
    int64_t rel_margin_ppm; /* telemetry margin q used by the decision (0 when off)       */
    int32_t n_prefill;    /* prompts served (chunk is their total; prefill_id the first)  */
    int32_t reserved;
    int64_t resid_p99_ns; /* fallback window's P99 tested by the decision (0 when off, when
                             the window is empty, or with no prompt to serve or no decode) */
} slw_iteration_record;

/*
 * Serve a trace to completion (synchronous).  Each iteration decodes one
 * token for every active request (decode rows in ascending id order) and
 * runs at most one prefill chunk of the oldest eligible prompt (by arrival,
 * then id; opts->queue and opts->max_prefills change which and how many
 * prompts); requests that arrive during an iteration become eligible when
 * it ends; the first output token is emitted by the iteration that finishes
 * the prompt, which also sets l_i; a prompt may start only while fewer than
 * max_decode requests decode and (GPU) while the pool can hold every
 * admitted request to its last token.  With no eligible work the clock
 * moves to the next arrival (SLW_EXEC_ANALYTIC, or skip_idle) or waits for
 * it.  The table executor advances the clock by exec_table's T_hat(n, c)
 * (a stand-in for hardware whose cost differs from the controller's table).
 * With a context axis in the table, decisions and predictions are priced
 * at the cached prefix of the first prompt the iteration serves (0 with none).
 * The GPU executor synchronises `stream` after every iteration, creates
 * a KV sequence per request when its prompt starts and frees it when its
 * last token is out; ctx may be NULL with SLW_EXEC_ANALYTIC.
 *   reqs       host [n], any order, distinct ids
 *   token_ns   host [sum of output_len]: request k's tokens at offset
 *              sum_{j<k} output_len[j], each the trace-clock time it was emitted
 *   iters      host [iter_cap] iteration records; *n_iters receives the count
 * SLW_ERANGE if the run needs more than iter_cap iterations or token_cap is
 * short; SLW_ENOMEM if one request alone can never fit the KV pool.
 */
int slw_serve(slw_ctx* ctx, const slw_request* reqs, int32_t n, const slw_serve_opts* opts,
              int64_t* token_ns, int64_t token_cap, slw_iteration_record* iters, int64_t iter_cap,
              int64_t* n_iters);

#ifdef __cplusplus
}
#endif

#endif /* SLOWEAVE_H */

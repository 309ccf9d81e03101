// Host-side launch interface of the gfx950 kernels (internal to libsloweave).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace slw {

// y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g over rows of d values; x is bf16
// or (x_f32) fp32, y is bf16.
void launch_rmsnorm(const void* x, bool x_f32, const void* g, void* y, int rows, int d, float eps,
                    hipStream_t s);


// GEMM out = A W^T with an epilogue:
//   EPI_RESID_F32OUT  out fp32 = acc + resid (bf16)
//   EPI_RESID_F32IN   out bf16 = acc + resid (fp32)
//   EPI_SWIGLU        W holds gate rows then up rows (n = 2f); out bf16 [m][f] = silu(gate) * up
//   EPI_QKV           W is the fused q/k/v projection; out bf16 [m][n] holds q and k rotated by
//                     RoPE and v; k and v are also appended to the paged pools at slot[r]
enum GemmEpilogue { EPI_RESID_F32OUT = 0, EPI_RESID_F32IN = 1, EPI_SWIGLU = 2, EPI_QKV = 3 };
struct GemmArgs {
    const void* a;      // bf16 [m][k], row stride lda
    const void* w;      // bf16 [n][k]
    void* out;          // [m][n_out], row stride ldo
    const void* resid;  // [m][n_out], row stride ldo
    int m, n, k;        // n counts W rows
    int lda, ldo;
    int epi;
    // EPI_QKV only
    const float2* rope_cs;  // [m][hd/2]
    const int32_t* slot;    // [m]
    void* k_pool;           // this layer's pages
    void* v_pool;
    int hq, hkv, hd;
};
struct GemmPlan {
    int cfg;      // tile configuration index (kSkinnyCfg: the weight-streaming kernel)
    int bm, bn;
    int splits;   // split-K factor across work-groups (1: fused epilogue)
    size_t partial_bytes;
    int ks;     // weight-streaming kernel (m <= 32): k slices per work-group
    int sk_workers = 0;  // stream-K: work-groups sharing the k steps of the last tiles (0: off)
    int dp_tiles = 0;    // stream-K: tiles run whole before them
};
// CUs the stream-K schedule spreads its last round over (MI355X).
constexpr int kStreamKCus = 256;
constexpr int kSkinnyCfg = 99;
constexpr int kNarrowCfg = 98;  // the narrow kernel (m <= 32, k split inside the work-group)
GemmPlan plan_gemm(int m, int n, int k);
// The plan for a given tile configuration (split-K chosen by tile count).
GemmPlan plan_with_cfg(int cfg, int m, int n, int k);
// The configuration with a stream-K schedule: whole tiles for all rounds but
// the last full one, whose tiles and the remainder share their k steps
// equally over one round of work-groups (plain tiles when rounds are whole).
GemmPlan plan_stream_k(int cfg, int m, int n, int k);
// Whether the plan's tiles divide n and k.
bool gemm_shape_ok(const GemmPlan& p, int n, int k);
// Enqueue the GEMM; `partial` must hold plan.partial_bytes when plan.splits > 1.
void launch_gemm(const GemmArgs& g, const GemmPlan& plan, void* partial, hipStream_t s);

// Causal chunk-vs-prefix attention over the prefill sequences' pages.
// A query tile holds up to 256 / group consecutive chunk rows of one prefill
// sequence; a work-group covers 256 (position, head) rows of one kv head: the
// tile's positions times the group's q heads.  Work item i covers query tile
// item_qt[i] against keys [item_kb[i], item_ke[i]); when a tile's keys are
// split over several items, partials are merged afterwards.
struct ChunkAttnArgs {
    const void* qkv;       // bf16 rows 0..c-1 (q after RoPE), row stride ld_qkv
    void* out;             // bf16 [c][hq * hd]
    const void* k_pool;    // this layer
    const void* v_pool;
    const int32_t* bt;     // block tables of the prefill sequences, one after the other
    const int32_t* qt_row0;   // [n_qt] first chunk row of each query tile
    const int32_t* qt_rows;   // [n_qt] rows of the tile (<= 256 / group)
    const int32_t* qt_pos0;   // [n_qt] sequence position of the tile's first row
    const int32_t* qt_bt;     // [n_qt] offset of the tile's sequence's block table in bt
    const int32_t* item_qt;   // [n_items]
    const int32_t* item_kb;   // [n_items] multiple of 64
    const int32_t* item_ke;   // [n_items]
    const int32_t* qt_off;    // [n_qt + 1] first item of each query tile
    const int32_t* slot_off;  // [n_slots + 1] first entry of each work-group in slot_items (per kv head)
    const int32_t* slot_items; // [n_items] the items of each work-group, in the order it takes them
    float* part_o;            // [n_items][hkv][256][hd]   (items of split query tiles)
    float* part_ml;           // [n_items][hkv][256][2]
    int c, hq, hkv, hd, ld_qkv;
    int n_qt, n_items, n_slots;
    int split;                // some query tile has several items: the merge kernel runs
};
// Query positions per work-group for a group size (rows / group).
inline int chunk_tile_positions(int group) { return 256 / group; }
void launch_chunk_attention(const ChunkAttnArgs& a, hipStream_t s);

// Split-K paged decode attention plus merge.
struct DecodeAttnArgs {
    const void* q;           // bf16 decode rows (q after RoPE), row stride ld_q
    void* out;               // bf16 [b][hq * hd]
    const void* k_pool;
    const void* v_pool;
    const int32_t* kv_len;   // [b] keys per decode (context + 1)
    const int32_t* bt_off;   // [b + 1] offsets into bt
    const int32_t* bt;       // concatenated block tables
    const int32_t* work_b;   // [n_work] decode of each work item
    const int32_t* work_kb;  // [n_work] first key of the item (a multiple of 64)
    const int32_t* work_ke;  // [n_work] key past its last
    const int32_t* work_off; // [b + 1] first work item of each decode
    const int32_t* slot_off; // [n_slots + 1] first work item of each wave (per kv head)
    float* part_o;           // [n_work][hq][hd]
    float* part_ml;          // [n_work][hq][2]
    int b, n_work, n_slots, hq, hkv, hd, ld_q;
};
void launch_decode_attention_split(const DecodeAttnArgs& a, hipStream_t s);
// Both attentions of a layer in one launch (chunk work-groups first, decode
// waves after them); either part may be empty.
void launch_attention(const ChunkAttnArgs& ca, const DecodeAttnArgs& da, hipStream_t s);
// Combine the partials of both attentions in one launch: chunk rows of
// query tiles split over several items (ca may be null or unsplit) and every
// decode (da may be null or have b = 0).
void launch_attention_merge(const ChunkAttnArgs* ca, const DecodeAttnArgs* da, hipStream_t s);

// One kernel: copy `words` 32-bit words from coherent, mapped host memory
// (its device address; both pointers 16-byte aligned) to device memory, and
// fill the RoPE table: cs[r][i] = (cos, sin) of pos_host[r] * theta^(-2i/hd),
// i < hd/2, formed in double (pos_host lies in that host memory).
void launch_iteration_setup(void* dst, const void* src, size_t words, const int32_t* pos_host, float2* cs,
                            int rows, int hd, double theta, hipStream_t s);

// dst[i] = bf16(mean + std z_i), z the standard normals of the Philox4x32-10
// stream keyed by seed (element i from draw i / 4 by Box-Muller).
void launch_fill_normal(void* dst, size_t n, uint64_t seed, float mean, float std, hipStream_t s);

// Read `bytes` of device memory (last-level cache flush that leaves no dirty
// lines); the buffer is written only if a thread's xor of its words equals key.
void launch_cache_sweep(void* p, size_t bytes, uint32_t key, hipStream_t s);

}  // namespace slw

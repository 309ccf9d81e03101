// Host-side launch interface of the gfx950 kernels (internal to libsloweave).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace slw {

// y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g, rows of d bf16 values.
void launch_rmsnorm(const void* x, const void* g, void* y, int rows, int d, float eps,
                    hipStream_t s);

// Rotate q and k of every row of qkv in place (rotate-half RoPE at pos[r]) and
// append k (rotated) and v to the paged pools at slot[r].
struct RopeAppendArgs {
    void* qkv;             // bf16 [rows][(hq + 2 hkv) * hd]
    const int32_t* pos;    // [rows]
    const int32_t* slot;   // [rows]
    void* k_pool;          // bf16 pages of this layer
    void* v_pool;
    int rows, hq, hkv, hd;
    double theta;
};
void launch_rope_append(const RopeAppendArgs& a, hipStream_t s);

// GEMM out = A W^T with an epilogue.
enum GemmEpilogue { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };
struct GemmArgs {
    const void* a;      // bf16 [m][k], row stride lda
    const void* w;      // bf16 [n][k] (EPI_SWIGLU: [2 f][k], gate rows then up rows)
    void* out;          // bf16 [m][n_out], row stride ldo
    const void* resid;  // bf16 [m][n_out], row stride ldo (EPI_RESID)
    int m, n, k;        // n counts W rows (2 f for EPI_SWIGLU)
    int lda, ldo;
    int epi;
};
struct GemmPlan {
    int cfg;      // tile configuration index
    int bm, bn;
    int splits;   // split-K factor (1: fused epilogue)
    size_t partial_bytes;
};
GemmPlan plan_gemm(int m, int n, int k);
// Enqueue the GEMM; `partial` must hold plan.partial_bytes when plan.splits > 1.
void launch_gemm(const GemmArgs& g, const GemmPlan& plan, void* partial, hipStream_t s);

// Causal chunk-vs-prefix attention over the prefill sequence's pages.
struct ChunkAttnArgs {
    const void* qkv;       // bf16 rows 0..c-1 (q after RoPE), row stride ld_qkv
    void* out;             // bf16 [c][hq * hd]
    const void* k_pool;    // this layer
    const void* v_pool;
    const int32_t* bt;     // block table of the prefill sequence
    int c, prefix, hq, hkv, hd, ld_qkv;
};
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
    const int32_t* work_s;   // [n_work] split index of each work item
    const int32_t* work_off; // [b + 1] first work item of each decode
    float* part_o;           // [n_work][hq][hd]
    float* part_ml;          // [n_work][hq][2]
    int b, n_work, split_tokens, hq, hkv, hd, ld_q;
};
void launch_decode_attention(const DecodeAttnArgs& a, hipStream_t s);

// Fill `bytes` of device memory with a byte pattern (last-level cache flush).
void launch_fill(void* p, size_t bytes, uint32_t pattern, hipStream_t s);

}  // namespace slw

// bf16 GEMM out = A W^T on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// A [m][k] and W [n][k] are both k-contiguous.  A work-group of four waves
// computes a BM x BN tile; k advances in steps of 64 through a double-buffered
// LDS tile (one barrier per step, next tile prefetched into registers while
// the current one feeds the matrix cores).  LDS rows are 128 bytes; the
// 16-byte chunk c of row r is stored at c ^ ((r >> 1) & 7) so that the
// 32 rows read by one MFMA operand load hit distinct banks.
//
// Epilogues: plain store, residual add, and SwiGLU.  For SwiGLU the B tile
// interleaves 32-row blocks of gate and up rows, so each wave holds the gate
// and up accumulators of the same output column in the same lane and writes
// silu(gate) * up directly.  Small problems split k across work-groups; the
// fp32 partial sums are then reduced by a second kernel that applies the
// epilogue.
#include <math.h>

#include "device.h"
#include "kernels.h"

namespace slw {
namespace {

constexpr int BK = 64;
constexpr int kThreads = 256;

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// W row feeding B-tile row r of the tile starting at B column n0.
template <int EPI>
__device__ __forceinline__ int w_row(int n0, int r, int n) {
    if (EPI == EPI_SWIGLU) {
        const int sub = r >> 5, f = n >> 1;
        const int col = (n0 >> 1) + (sub >> 1) * 32 + (r & 31);
        return (sub & 1) ? f + col : col;
    }
    return n0 + r;
}

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

template <int BM, int BN, int WM, int WN, int EPI, bool SPLIT>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs g, float* __restrict__ partial,
                                                        int k_per_split) {
    constexpr int WAVES_N = BN / WN;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int A_LOADS = BM * 8 / kThreads;
    constexpr int B_LOADS = BN * 8 / kThreads;
    static_assert((BM / WM) * (BN / WN) == 4, "four waves");
    static_assert(A_LOADS >= 1 && B_LOADS >= 1, "tile too small");

    __shared__ __attribute__((aligned(16))) bf16 As[2][BM * BK];
    __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * BK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
    const int kb = blockIdx.z * k_per_split;
    const int nk = k_per_split / BK;

    const bf16* A = static_cast<const bf16*>(g.a);
    const bf16* W = static_cast<const bf16*>(g.w);

    // per-thread global source pointers (row fixed for the whole k loop)
    const bf16* a_src[A_LOADS];
    bool a_ok[A_LOADS];
    int a_lds[A_LOADS];
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
        const int idx = tid + i * kThreads, row = idx >> 3, ch = idx & 7;
        a_ok[i] = (m0 + row) < g.m;
        a_src[i] = A + static_cast<size_t>(a_ok[i] ? m0 + row : 0) * g.lda + kb + ch * 8;
        a_lds[i] = row * BK + swz(row, ch) * 8;
    }
    const bf16* b_src[B_LOADS];
    int b_lds[B_LOADS];
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
        const int idx = tid + i * kThreads, row = idx >> 3, ch = idx & 7;
        b_src[i] = W + static_cast<size_t>(w_row<EPI>(n0, row, g.n)) * g.k + kb + ch * 8;
        b_lds[i] = row * BK + swz(row, ch) * 8;
    }

    bf16x8 ra[A_LOADS], rb[B_LOADS];
    const bf16x8 zero8 = {};
    auto load_tile = [&](int kt) {
        const int off = kt * BK;
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            ra[i] = a_ok[i] ? *reinterpret_cast<const bf16x8*>(a_src[i] + off) : zero8;
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) rb[i] = *reinterpret_cast<const bf16x8*>(b_src[i] + off);
    };
    auto store_tile = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) *reinterpret_cast<bf16x8*>(&As[buf][a_lds[i]]) = ra[i];
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) *reinterpret_cast<bf16x8*>(&Bs[buf][b_lds[i]]) = rb[i];
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

    // LDS element offsets of this lane's operand rows
    int a_row[TM], b_row[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) a_row[i] = wm * WM + i * 32 + (lane & 31);
#pragma unroll
    for (int j = 0; j < TN; ++j) b_row[j] = wn * WN + j * 32 + (lane & 31);
    const int kg = lane >> 5;

    load_tile(0);
    store_tile(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_tile(kt + 1);
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            bf16x8 fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = *reinterpret_cast<const bf16x8*>(
                    &As[buf][a_row[i] * BK + swz(a_row[i], 2 * s + kg) * 8]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[j] = *reinterpret_cast<const bf16x8*>(
                    &Bs[buf][b_row[j] * BK + swz(b_row[j], 2 * s + kg) * 8]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(fa[i], fb[j], acc[i][j]);
        }
        if (kt + 1 < nk) store_tile(buf ^ 1);
        __syncthreads();
    }

    // epilogue
    const int rbase = m0 + wm * WM + 4 * (lane >> 5);
    if (SPLIT) {
        float* P = partial + static_cast<size_t>(blockIdx.z) * g.m * g.n;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = n0 + wn * WN + j * 32 + (lane & 31);
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
                    if (row < g.m) P[static_cast<size_t>(row) * g.n + col] = acc[i][j][e];
                }
            }
        return;
    }
    bf16* out = static_cast<bf16*>(g.out);
    const bf16* res = static_cast<const bf16*>(g.resid);
    if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int p = 0; p < TN / 2; ++p) {
                const int col = ((n0 + wn * WN) >> 1) + p * 32 + (lane & 31);
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
                    if (row < g.m)
                        out[static_cast<size_t>(row) * g.ldo + col] =
                            f2bf(silu(acc[i][2 * p][e]) * acc[i][2 * p + 1][e]);
                }
            }
        return;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = n0 + wn * WN + j * 32 + (lane & 31);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
                if (row < g.m) {
                    float v = acc[i][j][e];
                    const size_t o = static_cast<size_t>(row) * g.ldo + col;
                    if (EPI == EPI_RESID) v += bf2f(res[o]);
                    out[o] = f2bf(v);
                }
            }
        }
}

// Sum split-K partials [splits][m][n] and apply the epilogue; 4 outputs per thread.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs g, const float* __restrict__ part,
                                                            int splits) {
    const int n_out = (EPI == EPI_SWIGLU) ? g.n / 2 : g.n;
    const int per_row = n_out / 4;
    const size_t idx = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
    if (idx >= static_cast<size_t>(g.m) * per_row) return;
    const int row = static_cast<int>(idx / per_row);
    const int c4 = static_cast<int>(idx % per_row) * 4;
    const size_t slab = static_cast<size_t>(g.m) * g.n;
    bf16* out = static_cast<bf16*>(g.out) + static_cast<size_t>(row) * g.ldo + c4;
    if (EPI == EPI_SWIGLU) {
        const int gc = (c4 >> 5) * 64 + (c4 & 31);  // gate column in B order; up is +32
        f32x4 gs = {}, us = {};
        for (int z = 0; z < splits; ++z) {
            const float* p = part + z * slab + static_cast<size_t>(row) * g.n + gc;
            gs += *reinterpret_cast<const f32x4*>(p);
            us += *reinterpret_cast<const f32x4*>(p + 32);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = f2bf(silu(gs[e]) * us[e]);
        return;
    }
    f32x4 s = {};
    for (int z = 0; z < splits; ++z)
        s += *reinterpret_cast<const f32x4*>(part + z * slab + static_cast<size_t>(row) * g.n + c4);
    if (EPI == EPI_RESID) {
        const bf16* r = static_cast<const bf16*>(g.resid) + static_cast<size_t>(row) * g.ldo + c4;
#pragma unroll
        for (int e = 0; e < 4; ++e) s[e] += bf2f(r[e]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) out[e] = f2bf(s[e]);
}

struct TileCfg {
    int bm, bn;
};
constexpr TileCfg kCfgs[3] = {{128, 128}, {64, 128}, {32, 256}};

template <int BM, int BN, int WM, int WN>
void launch_cfg(const GemmArgs& g, const GemmPlan& p, void* partial, hipStream_t s) {
    dim3 grid(g.n / BN, (g.m + BM - 1) / BM, p.splits);
    const int kps = g.k / p.splits;
    float* part = static_cast<float*>(partial);
    if (p.splits > 1) {
        switch (g.epi) {
            case EPI_STORE: gemm_kernel<BM, BN, WM, WN, EPI_STORE, true><<<grid, kThreads, 0, s>>>(g, part, kps); break;
            case EPI_RESID: gemm_kernel<BM, BN, WM, WN, EPI_RESID, true><<<grid, kThreads, 0, s>>>(g, part, kps); break;
            default: gemm_kernel<BM, BN, WM, WN, EPI_SWIGLU, true><<<grid, kThreads, 0, s>>>(g, part, kps); break;
        }
        const int n_out = g.epi == EPI_SWIGLU ? g.n / 2 : g.n;
        const size_t work = static_cast<size_t>(g.m) * (n_out / 4);
        const int blocks = static_cast<int>((work + 255) / 256);
        switch (g.epi) {
            case EPI_STORE: splitk_reduce_kernel<EPI_STORE><<<blocks, 256, 0, s>>>(g, part, p.splits); break;
            case EPI_RESID: splitk_reduce_kernel<EPI_RESID><<<blocks, 256, 0, s>>>(g, part, p.splits); break;
            default: splitk_reduce_kernel<EPI_SWIGLU><<<blocks, 256, 0, s>>>(g, part, p.splits); break;
        }
        return;
    }
    switch (g.epi) {
        case EPI_STORE: gemm_kernel<BM, BN, WM, WN, EPI_STORE, false><<<grid, kThreads, 0, s>>>(g, nullptr, kps); break;
        case EPI_RESID: gemm_kernel<BM, BN, WM, WN, EPI_RESID, false><<<grid, kThreads, 0, s>>>(g, nullptr, kps); break;
        default: gemm_kernel<BM, BN, WM, WN, EPI_SWIGLU, false><<<grid, kThreads, 0, s>>>(g, nullptr, kps); break;
    }
}

}  // namespace

// Tile and split choice.  n must be a multiple of 128 and k of 64.
GemmPlan plan_gemm(int m, int n, int k) {
    GemmPlan p{};
    if (m <= 32 && n % 256 == 0) p.cfg = 2;
    else if (m <= 64) p.cfg = 1;
    else p.cfg = 0;
    p.bm = kCfgs[p.cfg].bm;
    p.bn = kCfgs[p.cfg].bn;
    const long tiles = static_cast<long>(n / p.bn) * ((m + p.bm - 1) / p.bm);
    int splits = 1;
    // Too few tiles to fill 256 compute units: split k (each split >= 512 deep).
    while (splits < 8 && tiles * splits < 384 && k % (2 * splits * BK) == 0 && k / (2 * splits) >= 512)
        splits *= 2;
    p.splits = splits;
    p.partial_bytes = splits > 1 ? static_cast<size_t>(splits) * m * n * sizeof(float) : 0;
    return p;
}

void launch_gemm(const GemmArgs& g, const GemmPlan& p, void* partial, hipStream_t s) {
    if (g.m <= 0) return;
    switch (p.cfg) {
        case 0: launch_cfg<128, 128, 64, 64>(g, p, partial, s); break;
        case 1: launch_cfg<64, 128, 32, 64>(g, p, partial, s); break;
        default: launch_cfg<32, 256, 32, 64>(g, p, partial, s); break;
    }
}

}  // namespace slw
